// The integer path of libfm for CDNA4 (gfx950): integer codes at a
// quantization specification (Sec. 2.2; App. D), the classical int8 operator
// and the certified fast realization of Sec. 4.2 (Prop. 1).
//
//  i8_quantize_kernel  codes x / d rounded to nearest even, d = max|x| / b,
//                      one scale per row and group of g along the inner
//                      dimension (B is quantized through its transpose).
//  i8_form_kernel      block sums of codes for every call of the fast
//                      realization (exact integers; a flag records any that
//                      leaves int8).
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
// for x < br = rows / gp, y < h; with neg, outn holds the negation.  One
// thread per (kappa, x, four consecutive y) and all r.  The sums are exact
// in int32; any outside int8 sets *flag (the certificate rules it out for
// codes within the bound).
__global__ __launch_bounds__(kThreads) void i8_form_kernel(const int8_t* __restrict__ X, int rows,
                                                           int K, int gp, int gk, int h, int R,
                                                           const int8_t* __restrict__ coef,
                                                           int8_t* __restrict__ out,
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
        const int c = cf[(size_t)r * gp * gk + p * gk + q];
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
  int M, N, K, g;
  int gm, gn, Mb, Nb, tiles_m, tiles_n, total;
  int R, h, calls_per_group;
};

constexpr int SCALE_BYTES = 2048;            // per stage: dA (1 KB) + dB (1 KB slot)
constexpr int I8STAGE = DSTAGE + SCALE_BYTES;
constexpr int MAX_SEGS = 1024;

template <bool FAST>
__global__ __launch_bounds__(DNT) void i8_gemm_kernel(I8Args a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[DNS * I8STAGE];
  __shared__ int32_t seg_lds[FAST ? MAX_SEGS : 1];
  __shared__ int32_t off_lds[FAST ? 65 : 1];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q = lane >> 4, l16 = lane & 15;
  const int tiles_blk = a.tiles_m * a.tiles_n;
  const int ng = a.K / a.g;
  if constexpr (FAST) {
    const int nb = a.gm * a.gn;
    for (int i = tid; i <= nb; i += DNT) off_lds[i] = ro(a.seg_off)[i];
    const int ns = ro(a.seg_off)[nb];
    for (int i = tid; i < ns; i += DNT) seg_lds[i] = ro(a.segs)[i];
    __syncthreads();
  }
  // K steps per group for the block of a tile
  auto steps_per_group = [&](int c) -> int {
    if constexpr (FAST) return a.calls_per_group * (off_lds[c + 1] - off_lds[c]) * a.h / GK;
    else return a.g / GK;
  };
  const bool vec_store = (a.Nb & 3) == 0 && (a.N & 3) == 0;

  const int G = gridDim.x;
  const int total = a.total;
  const bool xcd_split = (G & 7) == 0 && (total & 7) == 0;
  const int t = xcd_split ? (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3) : blockIdx.x;
  const int tstep = xcd_split ? (G >> 3) : G;
  const int t_end = xcd_split ? ((blockIdx.x & 7) + 1) * (total >> 3) : total;
  if (t >= t_end) return;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;

  struct TileGeo {
    int c, ib, jb, m0, n0;
  };
  auto geo = [&](int tile) {
    TileGeo r;
    r.c = tile / tiles_blk;
    const int tt = tile - r.c * tiles_blk;
    r.ib = r.c / a.gn;
    r.jb = r.c - r.ib * a.gn;
    const int tmi = tt / a.tiles_n;
    r.m0 = tmi * DBM;
    r.n0 = (tt - tmi * a.tiles_n) * DBN;
    return r;
  };

  auto issue = [&](int tile, int kt, int buf) {
    const TileGeo tg = geo(tile);
    const int spg = steps_per_group(tg.c);
    const int gi = kt / spg, sg = kt - (kt / spg) * spg;
    int kap = 0, st = 0, sbase = 0;
    if constexpr (FAST) {
      const int spc = spg / a.calls_per_group;  // steps per call
      const int kc = sg / spc;
      st = sg - kc * spc;
      kap = gi * a.calls_per_group + kc;
      sbase = off_lds[tg.c] + st * (GK / a.h);
    }
#pragma unroll
    for (int j = 0; j < DLOADS; ++j) {
      const int r0 = (wave * DLOADS + j) * 8;  // first of the 8 rows this wave-load fills
      const int r = r0 + (lane >> 3);
      const int ch = (lane & 7) ^ swz(r);
      const uint8_t* src;
      if constexpr (FAST) {
        const int s = sbase + (ch * 16) / a.h;
        const int oin = (ch * 16) % a.h;
        const int e = seg_lds[s];
        const int pr = e & 0xffff;
        if (r0 < DBM) {
          int row = tg.m0 + r;
          row = row < a.Mb ? row : 0;
          src = pr == 0xffff ? (const uint8_t*)a.zero
                             : (const uint8_t*)a.A + (((size_t)kap * a.R + pr) * a.Mb + row) * a.h + oin;
        } else {
          int col = tg.n0 + r - DBM;
          col = col < a.Nb ? col : 0;
          const int8_t* S = (e >> 16) ? a.Bn : a.B;
          src = pr == 0xffff ? (const uint8_t*)a.zero
                             : (const uint8_t*)S + (((size_t)kap * a.R + pr) * a.Nb + col) * a.h + oin;
        }
      } else {
        if (r0 < DBM) {
          int row = tg.m0 + r;
          row = row < a.M ? row : 0;
          src = (const uint8_t*)a.A + (size_t)row * a.K + (size_t)kt * GK + ch * 16;
        } else {
          int col = tg.n0 + r - DBM;
          col = col < a.N ? col : 0;
          src = (const uint8_t*)a.B + (size_t)col * a.K + (size_t)kt * GK + ch * 16;
        }
      }
      dma16(src, lds_base + (uint32_t)(buf * I8STAGE + r0 * GK));
    }
    // the group's scales ride with its last step: wave 0 loads dA for the
    // tile's 256 rows, wave 1 dB for its 128 columns (lanes 32-63 repeat
    // lanes 0-31); 4 rows or columns per lane, all in or all out of range
    if (sg == spg - 1 && wave < 2) {
      const float* src;
      if (wave == 0) {
        const int row = tg.m0 + 4 * lane;
        src = a.dA + (size_t)gi * a.M + (size_t)tg.ib * a.Mb + (row < a.Mb ? row : 0);
      } else {
        const int col = tg.n0 + 4 * (lane & 31);
        src = a.dB + (size_t)gi * a.N + (size_t)tg.jb * a.Nb + (col < a.Nb ? col : 0);
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
  auto epilogue = [&](int tile) -> int {  // returns the number of stores counted
    const TileGeo tg = geo(tile);
    const int r_base = tg.m0 + wm * 64 + l16, c_base = tg.n0 + wn * 64 + 4 * q;
    float* Ob = a.out + (size_t)tg.ib * a.Mb * a.N + (size_t)tg.jb * a.Nb;
    int counted = 0;
    if (vec_store && tg.m0 + DBM <= a.Mb && tg.n0 + DBN <= a.Nb) {
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

  // (tile, K-step) pairs p_0, p_1, ... in LDS buffer s mod 3, as in the
  // block-product kernel; a group ends with the last K step of its span
  auto nsteps = [&](int tile) { return ng * steps_per_group(tile / tiles_blk); };
  auto advance = [&](int& tt, int& kk) {
    if (++kk == nsteps(tt)) {
      kk = 0;
      tt += tstep;
    }
  };
  int t1 = t, k1 = 0;
  advance(t1, k1);
  int t2 = t1, k2 = k1;
  advance(t2, k2);
  int t3 = t2, k3 = k2;
  advance(t3, k3);
  int ct = t, ck = 0;
  issue(ct, ck, 0);
  int after1 = 0;
  if (t1 < t_end) issue(t1, k1, 1);
  if (t2 < t_end) {
    issue(t2, k2, 2);
    after1 = DLOADS;
  }
  wait_vm(t1 < t_end ? after1 + DLOADS : 0);
  FM_COMPILER_FENCE();
  __builtin_amdgcn_s_barrier();
  FM_COMPILER_FENCE();
  read_half(0, 0);
  int cb = 0;
  while (true) {
    const int spg = steps_per_group(ct / tiles_blk);
    const bool group_end = (ck % spg) == spg - 1;
    read_half(1, cb);
    if (group_end) read_scales(cb);
    compute_half(0);
    wait_vm(after1);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of p_s are done
    FM_COMPILER_FENCE();
    __builtin_amdgcn_s_barrier();
    FM_COMPILER_FENCE();
    const int nb = cb == 2 ? 0 : cb + 1;
    int after2 = 0;
    if (t3 < t_end) {
      issue(t3, k3, cb);
      after2 = DLOADS;
    }
    FM_COMPILER_FENCE();
    const bool more = t1 < t_end;
    if (more) read_half(0, nb);
    compute_half(1);
    if (group_end) rescale();
    if (ck == nsteps(ct) - 1) after2 += epilogue(ct);
    FM_COMPILER_FENCE();
    if (!more) break;
    ct = t1;
    ck = k1;
    t1 = t2;
    k1 = k2;
    t2 = t3;
    k2 = k3;
    advance(t3, k3);
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
                   const int8_t* coef, int8_t* out, int8_t* outn, uint32_t* flag, hipStream_t st) {
  const long long n = (long long)(K / (gk * h)) * (rows / gp) * (h / 4);
  const long long blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many block sums");
  i8_form_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(X, rows, K, gp, gk, h, R, coef, out, outn,
                                                        flag);
  return launched("i8_form_kernel");
}

int launch_i8_gemm(bool fast, const int8_t* A, const int8_t* B, const int8_t* Bn,
                   const int8_t* zero, const float* dA, const float* dB, float* out,
                   const int32_t* segs, const int32_t* seg_off, int nsegs, int M, int N, int K,
                   int g, int gm, int gn, int R, int h, int calls_per_group, hipStream_t st) {
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
  a.h = h;
  a.calls_per_group = calls_per_group;
  const int grid = (int)std::min<long long>(total, 256);
  if (fast) i8_gemm_kernel<true><<<grid, DNT, 0, st>>>(a);
  else i8_gemm_kernel<false><<<grid, DNT, 0, st>>>(a);
  return launched("i8_gemm_kernel");
}

}  // namespace fm
