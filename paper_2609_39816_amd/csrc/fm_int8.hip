// The integer path of libfm for CDNA4 (gfx950): integer codes at a
// quantization specification (Sec. 2.2; App. D), the classical int8 operator
// and the certified fast realization of Sec. 4.2 (Prop. 1).
//
//  i8_quantize_kernel  codes x / d rounded to nearest even, d = max|x| / b,
//                      one scale per row and group of g along the inner
//                      dimension (B is quantized through its transpose).
//  i8_form_dot_kernel  block sums of codes for every call of the fast
//                      realization (exact integers; a flag records any that
//                      leaves int8), on v_dot4 for up to 16 blocks;
//                      i8_form_kernel for larger grids.
//  i8_gemm_kernel      grouped int8 products on the matrix cores
//                      (v_mfma_i32_16x16x64_i8, exact int32 sums), each
//                      group's integer product rescaled as (P dA) dB and
//                      added in fp32 in ascending group order.  Classical:
//                      the operand rows are the codes.  Fast: every output
//                      block C_c of the scheme is one such product whose
//                      inner dimension runs through the segments
//                      (w_rc T_r, S_r) of the products it combines, per call:
//                      C_c = sum_r w_rc T_r S_r = [T_r ...] [w_rc S_r ...]^T,
//                      exact in int32 under the certificate.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <utility>
#include <vector>

#include "fm_device.h"
#include "fm_lds_ring.h"

namespace fm {
namespace {
using namespace dev;
using namespace ring;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ quantizer
// One wave per (row, group): lane l holds entries l, l + 64, ... of the
// group (g a multiple of 64, at most 512).
__global__ __launch_bounds__(kThreads) void i8_quantize_kernel(const float* __restrict__ X,
                                                               int rows, int K, int g, int b,
                                                               int8_t* __restrict__ codes,
                                                               float* __restrict__ d,
                                                               uint32_t* flag) {
  const int lane = threadIdx.x & 63;
  const long long w = (long long)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int ng = K / g;
  if (w >= (long long)rows * ng) return;
  const int t = (int)(w / ng), gi = (int)(w - (long long)t * ng);
  const float* x = X + (size_t)t * K + (size_t)gi * g;
  const int per = g / 64;
  float v[8];
  uint32_t m = 0u;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (e < per) {
      v[e] = x[lane + 64 * e];
      m = max(m, __float_as_uint(v[e]) & 0x7fffffffu);
    }
  m = wave_max_u32(m);
  if (m >= 0x7f800000u) {  // Inf or NaN in the group
    if (lane == 0 && flag) atomicOr(flag, 1u);
  }
  const float amax = __uint_as_float(m);
  const float s = amax == 0.0f ? 1.0f : __fdiv_rn(amax, (float)b);
  if (lane == 0) d[(size_t)gi * rows + t] = s;
  int8_t* c = codes + (size_t)t * K + (size_t)gi * g;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (e < per) c[lane + 64 * e] = (int8_t)(int)__builtin_rintf(__fdiv_rn(v[e], s));
}

// --------------------------------------------------- fast: block sums
// X: rows x K codes (A, or B's transpose); for every call kappa (gk blocks of
// inner length h, consecutive along K) and product r:
//   out[kappa][r][x][y] = sum_{p,q} coef[r][p*gk + q] * X[p*br + x][kappa*gk*h + q*h + y]
// for x < br = rows / gp, y < h; with neg, outn holds the negation.  coef is
// int8 with a row stride of `stride` bytes (zero beyond the gp*gk blocks).
// The sums are exact in int32; any outside [-127, 127] sets bit 2 of *flag
// (the certificate rules it out for codes within the bound).

// Bytewise two's-complement negation of four packed int8 (no carries between
// bytes: the low seven bits of ~x + 1 never carry past bit 7).
__device__ __forceinline__ uint32_t neg_bytes(uint32_t x) {
  const uint32_t n = ~x;
  return ((n & 0x7f7f7f7fu) + 0x01010101u) ^ (n & 0x80808080u);
}

__device__ __forceinline__ uint32_t byte_of(uint32_t x, int j) { return (x >> (8 * j)) & 0xffu; }

__device__ __forceinline__ uint32_t dword_of(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

// Up to 4 * NG blocks (NG packed dwords of coefficients per product): one
// thread per (call, row x, 16 consecutive y) and grid row per group of rg
// products.  The thread loads
// each block's 16 bytes once, transposes them so that one dword holds four
// blocks' codes at one position, and forms every product of its group with
// v_dot4 (four int8 products summed exactly into int32) against the packed
// coefficient dwords, which are wave-uniform.
template <int NG, bool CORR>
__global__ __launch_bounds__(kThreads) void i8_form_dot_kernel(
    const int8_t* __restrict__ X, int rows, int K, int gp, int gk, int h, int R, int rg,
    const int8_t* __restrict__ coef, int stride, int8_t* __restrict__ out,
    int8_t* __restrict__ outn, int8_t* __restrict__ outR, int8_t* __restrict__ outnR, int qmax,
    uint32_t* flag) {
  const int br = rows / gp;
  const int hc = h / 16;
  const int ncall = K / (gk * h);
  const int rgi = blockIdx.y;  // product group: wave-uniform, so coefficients load as scalars
  const long long id = (long long)blockIdx.x * kThreads + threadIdx.x;
  const long long per_call = (long long)br * hc;
  if (id >= per_call * ncall) return;
  const int kap = (int)(id / per_call);
  const int rem = (int)(id - kap * per_call);
  const int x = rem / hc, y0 = (rem - (rem / hc) * hc) * 16;
  const int nb = gp * gk;
  // t[w][G][j]: byte i is block 4G+i's code at position y0 + 4w + j
  uint32_t t[4][NG][4];
#pragma unroll
  for (int G = 0; G < NG; ++G) {
    uint4 v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int bi = 4 * G + i;
      if (bi < nb) {
        const int p = bi / gk, q = bi - (bi / gk) * gk;
        v[i] = *reinterpret_cast<const uint4*>(X + (size_t)(p * br + x) * K +
                                               (size_t)kap * gk * h + q * h + y0);
      } else {
        v[i] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t d[4] = {dword_of(v[0], w), dword_of(v[1], w), dword_of(v[2], w),
                             dword_of(v[3], w)};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        t[w][G][j] = byte_of(d[0], j) | (byte_of(d[1], j) << 8) | (byte_of(d[2], j) << 16) |
                     (byte_of(d[3], j) << 24);
    }
  }
  const auto cf = ro(reinterpret_cast<const int32_t*>(coef));
  const int sw = stride / 4;
  // plain: max of s + 127 over the sums, unsigned (> 254 leaves int8);
  // corrected: max |q| over the split parts (> qmax leaves the certificate)
  uint32_t worst = 0u;
  const int r0 = rgi * rg, r1 = min(R, r0 + rg);
  for (int r = r0; r < r1; ++r) {
    int c[NG];
#pragma unroll
    for (int G = 0; G < NG; ++G) c[G] = cf[(size_t)r * sw + G];
    uint32_t o[4], oq[4], on[4], onq[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t packed = 0u, pq = 0u, pn = 0u, pnq = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int s = 0;
#pragma unroll
        for (int G = 0; G < NG; ++G) s = __builtin_amdgcn_sdot4((int)t[w][G][j], c[G], s, false);
        if constexpr (CORR) {
          // eq. (2): s = s0 + 256 q, q = floor((s + 128) / 256), s0 in [-128, 127];
          // the negation is split on its own (-s0 may be 128)
          const int q = (s + 128) >> 8, s0 = s - (q << 8);
          const int qn = (128 - s) >> 8, s0n = -s - (qn << 8);
          worst = max(worst, (uint32_t)max(abs(q), abs(qn)));
          packed |= ((uint32_t)s0 & 0xffu) << (8 * j);
          pq |= ((uint32_t)q & 0xffu) << (8 * j);
          pn |= ((uint32_t)s0n & 0xffu) << (8 * j);
          pnq |= ((uint32_t)qn & 0xffu) << (8 * j);
        } else {
          worst = max(worst, (uint32_t)(s + 127));
          packed |= ((uint32_t)s & 0xffu) << (8 * j);
        }
      }
      o[w] = packed;
      oq[w] = pq;
      on[w] = pn;
      onq[w] = pnq;
    }
    const size_t off = (((size_t)kap * R + r) * br + x) * h + y0;
    *reinterpret_cast<uint4*>(out + off) = make_uint4(o[0], o[1], o[2], o[3]);
    if constexpr (CORR) {
      *reinterpret_cast<uint4*>(outR + off) = make_uint4(oq[0], oq[1], oq[2], oq[3]);
      if (outn) {
        *reinterpret_cast<uint4*>(outn + off) = make_uint4(on[0], on[1], on[2], on[3]);
        *reinterpret_cast<uint4*>(outnR + off) = make_uint4(onq[0], onq[1], onq[2], onq[3]);
      }
    } else if (outn) {
      *reinterpret_cast<uint4*>(outn + off) =
          make_uint4(neg_bytes(o[0]), neg_bytes(o[1]), neg_bytes(o[2]), neg_bytes(o[3]));
    }
  }
  const bool bad = CORR ? worst > (uint32_t)qmax : worst > 254u;
  if (bad && flag) atomicOr(flag, 2u);
}

// Any number of blocks: one thread per (call, x, four consecutive y) and all
// products, each block's four codes loaded per nonzero coefficient.
__global__ __launch_bounds__(kThreads) void i8_form_kernel(const int8_t* __restrict__ X, int rows,
                                                           int K, int gp, int gk, int h, int R,
                                                           const int8_t* __restrict__ coef,
                                                           int stride, int8_t* __restrict__ out,
                                                           int8_t* __restrict__ outn,
                                                           uint32_t* flag) {
  const int br = rows / gp;
  const int hq = h / 4;
  const int ncall = K / (gk * h);
  const long long id = (long long)blockIdx.x * kThreads + threadIdx.x;
  if (id >= (long long)ncall * br * hq) return;
  const int kap = (int)(id / ((long long)br * hq));
  const int rem = (int)(id - (long long)kap * br * hq);
  const int x = rem / hq, y0 = (rem - (rem / hq) * hq) * 4;
  const auto cf = ro(coef);
  bool bad = false;
  for (int r = 0; r < R; ++r) {
    int s0 = 0, s1 = 0, s2 = 0, s3 = 0;
    for (int p = 0; p < gp; ++p)
      for (int q = 0; q < gk; ++q) {
        const int c = cf[(size_t)r * stride + p * gk + q];
        if (c == 0) continue;
        const char4 v = *reinterpret_cast<const char4*>(
            X + (size_t)(p * br + x) * K + (size_t)kap * gk * h + q * h + y0);
        s0 += c * v.x;
        s1 += c * v.y;
        s2 += c * v.z;
        s3 += c * v.w;
      }
    bad |= s0 < -127 || s0 > 127 || s1 < -127 || s1 > 127 || s2 < -127 || s2 > 127 ||
           s3 < -127 || s3 > 127;
    const size_t o = (((size_t)kap * R + r) * br + x) * h + y0;
    *reinterpret_cast<char4*>(out + o) = make_char4((char)s0, (char)s1, (char)s2, (char)s3);
    if (outn)
      *reinterpret_cast<char4*>(outn + o) = make_char4((char)-s0, (char)-s1, (char)-s2, (char)-s3);
  }
  if (bad && flag) atomicOr(flag, 2u);
}

// ----------------------------------------------------- grouped int8 GEMM
struct I8Args {
  const int8_t* A;      // classical: M x K codes; fast: T[call][R][Mb][h]
  const int8_t* B;      // classical: N x K codes (B^T); fast: S[call][R][Nb][h] (transposed)
  const int8_t* Bn;     // fast: -S, same layout
  const int8_t* zero;   // fast: at least 128 zero bytes (padding segments)
  const float* dA;      // [K/g][M]
  const float* dB;      // [K/g][N]
  float* out;           // M x N
  const int32_t* segs;  // fast: segments per block, r | (w < 0) << 16; r = 0xffff: padding
  const int32_t* seg_off;  // fast: gm * gn + 1 offsets into segs
  const int32_t* order;    // fast: the tiles of every workgroup, consecutively
  const int32_t* order_off;  // fast: gridDim.x + 1 offsets into order
  // corrected fast path (eq. (2)): the split parts q of the block sums (the
  // remainders s0 are A, B, Bn above), and per block the K steps of a call
  // where the cross terms and the remainder products begin
  const int8_t* AR;
  const int8_t* BR;
  const int8_t* BnR;
  const int32_t* phase;  // [gm * gn][2]
  int M, N, K, g;
  int gm, gn, Mb, Nb, tiles_m, tiles_n, total;
  int R, calls_per_group;
};

constexpr int SCALE_BYTES = 2048;            // per stage: dA (1 KB) + dB (1 KB slot)
constexpr int I8STAGE = DSTAGE + SCALE_BYTES;
constexpr int MAX_SEGS = 1024;

// Position of a workgroup in its work: the slot of its tile list (fast) or
// the tile itself (classical), the tile's geometry and K-step count per
// call, and the step (group gi, call kc within the group, step st within the
// call).  All wave-uniform; advanced incrementally so that no step divides.
struct I8Cursor {
  int slot, ib, jb, m0, n0, spc, sb, gi, kc, st, p1, p0;
};

// H: the block inner length h of the fast realization (0: classical).
// CORR: the overflow correction (eq. (2)).  A call's segments then come in
// three phases, R_A R_B, then R_A B0 and A0 R_B, then A0 B0, and the int32
// accumulator is multiplied by 256 as each of the last two begins (Horner's
// rule: ((R_A R_B) 256 + cross terms) 256 + A0 B0), so one accumulator holds
// the exact product; a group is one call.
template <int H, bool CORR>
__global__ __launch_bounds__(DNT) void i8_gemm_kernel(I8Args a) {
  constexpr bool FAST = H > 0;
  static_assert(!FAST || (H >= 16 && H <= GK && GK % H == 0), "block inner length");
  static_assert(FAST || !CORR, "the correction belongs to the fast path");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[DNS * I8STAGE];
  __shared__ int32_t seg_lds[FAST ? MAX_SEGS : 1];
  __shared__ int32_t off_lds[FAST ? 65 : 1];
  __shared__ int32_t ph_lds[CORR ? 128 : 1];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q = lane >> 4, l16 = lane & 15;
  const int tiles_blk = a.tiles_m * a.tiles_n;
  const int ng = a.K / a.g;
  const int cpg = FAST ? a.calls_per_group : 1;
  if constexpr (FAST) {
    const int nb = a.gm * a.gn;
    for (int i = tid; i <= nb; i += DNT) off_lds[i] = ro(a.seg_off)[i];
    const int ns = ro(a.seg_off)[nb];
    for (int i = tid; i < ns; i += DNT) seg_lds[i] = ro(a.segs)[i];
    if constexpr (CORR)
      for (int i = tid; i < 2 * nb; i += DNT) ph_lds[i] = ro(a.phase)[i];
    __syncthreads();
  }
  const bool vec_store = (a.Nb & 3) == 0 && (a.N & 3) == 0;

  // the workgroup's tiles: fast, its list; classical, a stride through the
  // tiles, consecutive ones on one XCD
  int slot0, slot_end, slot_step;
  if constexpr (FAST) {
    slot0 = ro(a.order_off)[blockIdx.x];
    slot_end = ro(a.order_off)[blockIdx.x + 1];
    slot_step = 1;
  } else {
    const int G = gridDim.x;
    const bool xcd_split = (G & 7) == 0 && (a.total & 7) == 0;
    slot0 = xcd_split ? (blockIdx.x & 7) * (a.total >> 3) + (blockIdx.x >> 3) : blockIdx.x;
    slot_step = xcd_split ? (G >> 3) : G;
    slot_end = xcd_split ? ((blockIdx.x & 7) + 1) * (a.total >> 3) : a.total;
  }
  if (slot0 >= slot_end) return;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;

  // classical tiles have one block (ib = jb = 0), one call per group and
  // g / GK steps per call: those fields stay constant and fold away
  const int spc_cl = a.g / GK;
  auto spc_of = [&](const I8Cursor& u) { return FAST ? u.spc : spc_cl; };
  auto enter = [&](I8Cursor& u) {  // u.slot valid: load the tile's geometry
    const int tile = FAST ? ro(a.order)[u.slot] : u.slot;
    const int c = tile / tiles_blk;
    const int tt = tile - c * tiles_blk;
    const int tmi = tt / a.tiles_n;
    u.m0 = tmi * DBM;
    u.n0 = (tt - tmi * a.tiles_n) * DBN;
    if constexpr (FAST) {
      u.ib = c / a.gn;
      u.jb = c - u.ib * a.gn;
      u.sb = off_lds[c];
      u.spc = (off_lds[c + 1] - u.sb) * H / GK;
    } else {
      u.ib = u.jb = u.sb = u.spc = 0;
    }
    if constexpr (CORR) {
      u.p1 = ph_lds[2 * c];
      u.p0 = ph_lds[2 * c + 1];
    } else {
      u.p1 = u.p0 = -1;
    }
    u.gi = u.kc = u.st = 0;
  };
  auto advance = [&](I8Cursor& u) {
    if (++u.st < spc_of(u)) return;
    u.st = 0;
    if constexpr (FAST) {
      if (++u.kc < cpg) return;
      u.kc = 0;
    }
    if (++u.gi < ng) return;
    u.slot += slot_step;
    if (u.slot < slot_end) enter(u);
  };

  auto issue = [&](const I8Cursor& u, int buf) {
    // row r of the stage (wave-load j, lane) takes 16-byte chunk
    // (lane & 7) ^ swz(r) = (lane & 7) ^ (lane >> 3) ^ (j & 1)
    const int ch_even = (lane & 7) ^ (lane >> 3);
    [[maybe_unused]] int e_even = 0, e_odd = 0;
    [[maybe_unused]] int kap = 0;
    if constexpr (FAST) {
      kap = u.gi * cpg + u.kc;
      const int sbase = u.sb + u.st * (GK / H);
      e_even = seg_lds[sbase + (ch_even * 16) / H];
      e_odd = H >= 32 ? e_even : seg_lds[sbase + ((ch_even ^ 1) * 16) / H];
    }
#pragma unroll
    for (int j = 0; j < DLOADS; ++j) {
      const int r0 = (wave * DLOADS + j) * 8;  // first of the 8 rows this wave-load fills
      const int r = r0 + (lane >> 3);
      const int ch = ch_even ^ (j & 1);
      const uint8_t* src;
      if constexpr (FAST) {
        const int e = (j & 1) ? e_odd : e_even;
        const int pr = e & 0xffff;
        const int oin = (ch * 16) % H;
        if (r0 < DBM) {
          int row = u.m0 + r;
          row = row < a.Mb ? row : 0;
          const int8_t* T = CORR && ((e >> 17) & 1) ? a.AR : a.A;
          src = pr == 0xffff ? (const uint8_t*)a.zero
                             : (const uint8_t*)T + (((size_t)kap * a.R + pr) * a.Mb + row) * H + oin;
        } else {
          int col = u.n0 + r - DBM;
          col = col < a.Nb ? col : 0;
          const bool neg = (e >> 16) & 1;
          const int8_t* S = CORR && ((e >> 18) & 1) ? (neg ? a.BnR : a.BR) : (neg ? a.Bn : a.B);
          src = pr == 0xffff ? (const uint8_t*)a.zero
                             : (const uint8_t*)S + (((size_t)kap * a.R + pr) * a.Nb + col) * H + oin;
        }
      } else {
        const size_t k0 = (size_t)u.gi * a.g + (size_t)u.st * GK + ch * 16;
        if (r0 < DBM) {
          int row = u.m0 + r;
          row = row < a.M ? row : 0;
          src = (const uint8_t*)a.A + (size_t)row * a.K + k0;
        } else {
          int col = u.n0 + r - DBM;
          col = col < a.N ? col : 0;
          src = (const uint8_t*)a.B + (size_t)col * a.K + k0;
        }
      }
      dma16(src, lds_base + (uint32_t)(buf * I8STAGE + r0 * GK));
    }
    // the group's scales ride with its last step: wave 0 loads dA for the
    // tile's 256 rows, wave 1 dB for its 128 columns (lanes 32-63 repeat
    // lanes 0-31); 4 rows or columns per lane, all in or all out of range
    if (u.st == spc_of(u) - 1 && (!FAST || u.kc == cpg - 1) && wave < 2) {
      const float* src;
      if (wave == 0) {
        const int row = u.m0 + 4 * lane;
        src = a.dA + (size_t)u.gi * a.M + (size_t)u.ib * a.Mb + (row < a.Mb ? row : 0);
      } else {
        const int col = u.n0 + 4 * (lane & 31);
        src = a.dB + (size_t)u.gi * a.N + (size_t)u.jb * a.Nb + (col < a.Nb ? col : 0);
      }
      dma16(src, lds_base + (uint32_t)(buf * I8STAGE + DSTAGE + wave * 1024));
    }
  };
  uint4 fa[2][4], fb[2][4];
  auto read_half = [&](int hh, int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = wm * 64 + i * 16 + l16;
      fa[hh][i] = *reinterpret_cast<const uint4*>(lds + buf * I8STAGE + row * GK +
                                                  (((2 * q + hh) ^ swz(row)) << 4));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = DBM + wn * 64 + j * 16 + l16;
      fb[hh][j] = *reinterpret_cast<const uint4*>(lds + buf * I8STAGE + row * GK +
                                                  (((2 * q + hh) ^ swz(row)) << 4));
    }
  };
  // acc[i][j]: the group's integer product, transposed 16 x 16 tiles: element
  // (4q+v, l16) is output row i*16 + l16, column j*16 + 4q + v of the wave's
  // 64 x 64 block; ofl: the fp32 sum over the groups so far
  v4i acc[4][4];
  v4f ofl[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[i][j] = (v4i){0, 0, 0, 0};
      ofl[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
    }
  auto compute_half = [&](int hh) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
            (v4i){(int)fb[hh][j].x, (int)fb[hh][j].y, (int)fb[hh][j].z, (int)fb[hh][j].w},
            (v4i){(int)fa[hh][i].x, (int)fa[hh][i].y, (int)fa[hh][i].z, (int)fa[hh][i].w},
            acc[i][j], 0, 0, 0);
  };
  float sa[4];
  float4 sb[4];
  auto read_scales = [&](int buf) {
    const float* sA = reinterpret_cast<const float*>(lds + buf * I8STAGE + DSTAGE);
    const float* sB = reinterpret_cast<const float*>(lds + buf * I8STAGE + DSTAGE + 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) sa[i] = sA[wm * 64 + i * 16 + l16];
#pragma unroll
    for (int j = 0; j < 4; ++j) sb[j] = *reinterpret_cast<const float4*>(sB + wn * 64 + j * 16 + 4 * q);
  };
  // out += (fl(P) * dA) * dB, each an fp32 operation, then the group restarts
  auto rescale = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float s4[4] = {sb[j].x, sb[j].y, sb[j].z, sb[j].w};
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float p = (float)acc[i][j][v];
          p = p * sa[i];
          p = p * s4[v];
          ofl[i][j][v] = ofl[i][j][v] + p;
        }
        acc[i][j] = (v4i){0, 0, 0, 0};
      }
  };
  auto epilogue = [&](const I8Cursor& u) -> int {  // returns the number of stores counted
    const int r_base = u.m0 + wm * 64 + l16, c_base = u.n0 + wn * 64 + 4 * q;
    float* Ob = a.out + (size_t)u.ib * a.Mb * a.N + (size_t)u.jb * a.Nb;
    int counted = 0;
    if (vec_store && u.m0 + DBM <= a.Mb && u.n0 + DBN <= a.Nb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float* prow = Ob + (size_t)(r_base + i * 16) * a.N + c_base;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<float4*>(prow + j * 16) =
              make_float4(ofl[i][j][0], ofl[i][j][1], ofl[i][j][2], ofl[i][j][3]);
      }
      counted = DSTORES;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = r_base + i * 16;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int col = c_base + j * 16 + v;
            if (row < a.Mb && col < a.Nb) Ob[(size_t)row * a.N + col] = ofl[i][j][v];
          }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) ofl[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
    return counted;
  };

  // K steps s_0, s_1, ... (cursors u0..u3) in LDS buffer s mod 3, as in the
  // block-product kernel; a group ends with the last step of its last call
  I8Cursor u0;
  u0.slot = slot0;
  enter(u0);
  I8Cursor u1 = u0;
  advance(u1);
  I8Cursor u2 = u1;
  advance(u2);
  I8Cursor u3 = u2;
  advance(u3);
  issue(u0, 0);
  int after1 = 0;
  if (u1.slot < slot_end) issue(u1, 1);
  if (u2.slot < slot_end) {
    issue(u2, 2);
    after1 = DLOADS;
  }
  wait_vm(u1.slot < slot_end ? after1 + DLOADS : 0);
  FM_COMPILER_FENCE();
  __builtin_amdgcn_s_barrier();
  FM_COMPILER_FENCE();
  read_half(0, 0);
  int cb = 0;
  while (true) {
    const bool group_end = u0.st == spc_of(u0) - 1 && (!FAST || u0.kc == cpg - 1);
    const bool tile_end = group_end && u0.gi == ng - 1;
    read_half(1, cb);
    if (group_end) read_scales(cb);
    if (CORR && (u0.st == u0.p1 || u0.st == u0.p0)) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = acc[i][j] << 8;
    }
    compute_half(0);
    wait_vm(after1);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of stage cb are done
    FM_COMPILER_FENCE();
    __builtin_amdgcn_s_barrier();
    FM_COMPILER_FENCE();
    const int nb = cb == 2 ? 0 : cb + 1;
    int after2 = 0;
    if (u3.slot < slot_end) {
      issue(u3, cb);
      after2 = DLOADS;
    }
    FM_COMPILER_FENCE();
    const bool more = u1.slot < slot_end;
    if (more) read_half(0, nb);
    compute_half(1);
    if (group_end) rescale();
    if (tile_end) after2 += epilogue(u0);
    FM_COMPILER_FENCE();
    if (!more) break;
    u0 = u1;
    u1 = u2;
    u2 = u3;
    advance(u3);
    after1 = after2;
    cb = nb;
  }
}

}  // namespace

int launch_i8_quantize(const float* X, int rows, int K, int g, int b, int8_t* codes, float* d,
                       uint32_t* flag, hipStream_t st) {
  const long long waves = (long long)rows * (K / g);
  const long long blocks = (waves + kThreads / 64 - 1) / (kThreads / 64);
  if (blocks > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many groups");
  i8_quantize_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(X, rows, K, g, b, codes, d, flag);
  return launched("i8_quantize_kernel");
}

int launch_i8_form(const int8_t* X, int rows, int K, int gp, int gk, int h, int R,
                   const int8_t* coef, int stride, int8_t* out, int8_t* outn, int8_t* outR,
                   int8_t* outnR, int qmax, uint32_t* flag, hipStream_t st) {
  const int nb = gp * gk;
  const int ng = (nb + 3) / 4;
  const bool corr = outR != nullptr;
  if (h % 16 || stride < 4 * ng || stride % 4) return fail(FM_E_ARG, "block-sum layout");
  if (corr && (ng > 4 || (outn && !outnR))) return fail(FM_E_ARG, "corrected block sums");
  if (ng <= 4) {
    const int nrg = (R + 7) / 8, rg = (R + nrg - 1) / nrg;
    const long long n = (long long)(K / (gk * h)) * (rows / gp) * (h / 16);
    const long long blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 0x7fffffffLL || nrg > 65535) return fail(FM_E_SHAPE, "too many block sums");
    const dim3 grid((unsigned)blocks, (unsigned)nrg);
#define FM_FORM_DOT(NG, C)                                                                    \
  i8_form_dot_kernel<NG, C><<<grid, kThreads, 0, st>>>(X, rows, K, gp, gk, h, R, rg, coef,   \
                                                       stride, out, outn, outR, outnR, qmax, \
                                                       flag)
    switch (ng * 2 + (corr ? 1 : 0)) {
      case 2: FM_FORM_DOT(1, false); break;
      case 3: FM_FORM_DOT(1, true); break;
      case 4: FM_FORM_DOT(2, false); break;
      case 5: FM_FORM_DOT(2, true); break;
      case 6: FM_FORM_DOT(3, false); break;
      case 7: FM_FORM_DOT(3, true); break;
      case 8: FM_FORM_DOT(4, false); break;
      default: FM_FORM_DOT(4, true); break;
    }
#undef FM_FORM_DOT
    return launched("i8_form_dot_kernel");
  }
  const long long n = (long long)(K / (gk * h)) * (rows / gp) * (h / 4);
  const long long blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many block sums");
  i8_form_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(X, rows, K, gp, gk, h, R, coef, stride,
                                                        out, outn, flag);
  return launched("i8_form_kernel");
}

long long i8_fast_tiles(int gm, int gn, int Mb, int Nb) {
  return (long long)gm * gn * ((Mb + DBM - 1) / DBM) * ((Nb + DBN - 1) / DBN);
}

// Longest-first assignment of the fast kernel's tiles to its workgroups: the
// tiles of block c cost block_steps[c] K steps plus two for the epilogue;
// in descending cost (ascending tile among equals) each goes to the least
// loaded of min(tiles, 256) workgroups (lowest first among equals).  The
// workgroups are numbered so that consecutive ones share an XCD (the
// hardware deals workgroup w to XCD w mod 8), which keeps a block's tiles,
// and the block sums they read, in one L2.
int i8_fast_schedule(int gm, int gn, int Mb, int Nb, const std::vector<int>& block_steps,
                     std::vector<int32_t>& order, std::vector<int32_t>& off) {
  const int tiles_m = (Mb + DBM - 1) / DBM, tiles_n = (Nb + DBN - 1) / DBN;
  const int per_blk = tiles_m * tiles_n;
  const int total = gm * gn * per_blk;
  const int grid = std::min(total, 256);
  std::vector<int> tiles(total);
  for (int t = 0; t < total; ++t) tiles[t] = t;
  auto cost = [&](int t) { return (long long)block_steps[t / per_blk] + 2; };
  std::stable_sort(tiles.begin(), tiles.end(), [&](int x, int y) { return cost(x) > cost(y); });
  const int per_xcd = grid % 8 == 0 ? grid / 8 : grid;
  auto physical = [&](int v) { return grid % 8 == 0 ? 8 * (v % per_xcd) + v / per_xcd : v; };
  std::vector<long long> load(grid, 0);
  std::vector<std::vector<int32_t>> lists(grid);
  // (load, virtual index) min-heap
  std::vector<std::pair<long long, int>> heap;
  for (int v = 0; v < grid; ++v) heap.emplace_back(0, v);
  auto later = [](const std::pair<long long, int>& x, const std::pair<long long, int>& y) {
    return x > y;
  };
  std::make_heap(heap.begin(), heap.end(), later);
  for (int t : tiles) {
    std::pop_heap(heap.begin(), heap.end(), later);
    auto& top = heap.back();
    lists[physical(top.second)].push_back(t);
    top.first += cost(t);
    std::push_heap(heap.begin(), heap.end(), later);
  }
  order.clear();
  off.assign(1, 0);
  for (int w = 0; w < grid; ++w) {
    order.insert(order.end(), lists[w].begin(), lists[w].end());
    off.push_back((int32_t)order.size());
  }
  return grid;
}

int launch_i8_gemm(bool fast, const int8_t* A, const int8_t* B, const int8_t* Bn,
                   const int8_t* zero, const float* dA, const float* dB, float* out,
                   const int32_t* segs, const int32_t* seg_off, int nsegs, const int32_t* order,
                   const int32_t* order_off, int grid, int M, int N, int K, int g, int gm, int gn,
                   int R, int h, int calls_per_group, const int8_t* AR, const int8_t* BR,
                   const int8_t* BnR, const int32_t* phase, hipStream_t st) {
  I8Args a{};
  a.A = A;
  a.B = B;
  a.Bn = Bn;
  a.zero = zero;
  a.dA = dA;
  a.dB = dB;
  a.out = out;
  a.segs = segs;
  a.seg_off = seg_off;
  a.order = order;
  a.order_off = order_off;
  a.AR = AR;
  a.BR = BR;
  a.BnR = BnR;
  a.phase = phase;
  a.M = M;
  a.N = N;
  a.K = K;
  a.g = g;
  a.gm = fast ? gm : 1;
  a.gn = fast ? gn : 1;
  a.Mb = M / a.gm;
  a.Nb = N / a.gn;
  a.tiles_m = (a.Mb + DBM - 1) / DBM;
  a.tiles_n = (a.Nb + DBN - 1) / DBN;
  const long long total = (long long)a.gm * a.gn * a.tiles_m * a.tiles_n;
  if (total > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many tiles");
  if (fast && (nsegs > MAX_SEGS || a.gm * a.gn > 64))
    return fail(FM_E_UNSUPPORTED, "scheme too large for the fast integer kernel");
  a.total = (int)total;
  a.R = R;
  a.calls_per_group = calls_per_group;
  if (!fast) {
    i8_gemm_kernel<0, false><<<(int)std::min<long long>(total, 256), DNT, 0, st>>>(a);
    return launched("i8_gemm_kernel");
  }
  if (!order || !order_off || grid < 1 || grid > total) return fail(FM_E_ARG, "tile schedule");
  const bool corr = phase != nullptr;
  if (corr && (!AR || !BR || !BnR || calls_per_group != 1))
    return fail(FM_E_ARG, "corrected products need the split parts and one call per group");
  switch (h * 2 + (corr ? 1 : 0)) {
    case 32: i8_gemm_kernel<16, false><<<grid, DNT, 0, st>>>(a); break;
    case 33: i8_gemm_kernel<16, true><<<grid, DNT, 0, st>>>(a); break;
    case 64: i8_gemm_kernel<32, false><<<grid, DNT, 0, st>>>(a); break;
    case 65: i8_gemm_kernel<32, true><<<grid, DNT, 0, st>>>(a); break;
    case 128: i8_gemm_kernel<64, false><<<grid, DNT, 0, st>>>(a); break;
    case 129: i8_gemm_kernel<64, true><<<grid, DNT, 0, st>>>(a); break;
    case 256: i8_gemm_kernel<128, false><<<grid, DNT, 0, st>>>(a); break;
    case 257: i8_gemm_kernel<128, true><<<grid, DNT, 0, st>>>(a); break;
    default: return fail(FM_E_ARG, "h must be 16, 32, 64 or 128");
  }
  return launched("i8_gemm_kernel");
}

}  // namespace fm
