// Batched FP8 block products of libfm for CDNA4 (gfx950), wave64:
// M_r = (sum_k Tq_r[x,k] Sq_r[z,k]) * dT_r * dS_r for a batch of products
// (the block products of eq. (1); Sec. 2.1 and the FP8 schedule of App. B.1).
//
//  gemm_dma_kernel   persistent, 256 x 128 tiles, a 3-stage LDS ring filled
//                    by direct global-to-LDS loads; inner lengths that are
//                    multiples of 128.
//  gemm_tile_kernel  one 128 x 128 tile per workgroup, double-buffered LDS;
//                    any inner length that is a multiple of 16.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cstring>

#include "fm_device.h"
#include "fm_lds_ring.h"

namespace fm {
namespace {
using namespace dev;
using namespace ring;

// ------------------------------------------------------ FP8 block GEMM
// Workgroup tile 128 x 128, K step 128 bytes, 4 waves in 2 x 2, each wave
// 64 x 64 = 4 x 4 tiles of 16 x 16.  FP8 operands are staged through
// double-buffered LDS, rows of 128 bytes with the 16-byte chunk index
// XOR-swizzled by a function of the row so that the fragment reads (16 rows
// x one chunk per instruction) hit distinct banks.
//
// Lane (i, q) = (lane % 16, lane / 16) of a wave holds the 32 bytes
// [32q, 32q + 32) of row i of a 16-row fragment, for both operands, so every
// k of the step is paired with the same k of the other operand.
//
// Two arithmetics for the products:
//   ACC_BF16 (default): every FP8 value is widened exactly to bf16
//     (v_cvt_scalef32_pk_bf16_{fp8,bf8}, scale 1) and multiplied on the bf16
//     matrix cores, v_mfma_f32_16x16x32_bf16: exact products, fp32 sums.
//   ACC_FP8: v_mfma_scale_f32_16x16x128_f8f6f4 with unit scales, twice the
//     rate; its sums of small products beside large ones are truncated
//     (about 5e-5 relative on random FP8 data), so it is not the default.
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

constexpr int GT = 128;  // tile rows / cols

// Two FP8 codes (bytes 0-1 or 2-3 of w) -> two bf16 values, exactly.
template <int FMT, bool HI>
__device__ __forceinline__ v2bf widen2(int w) {
  if constexpr (FMT == FM_E4M3) return __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI);
  else return __builtin_amdgcn_cvt_scalef32_pk_bf16_bf8(w, 1.0f, HI);
}

// 8 FP8 codes (two dwords, little-endian byte order) -> 8 bf16 values
template <int FMT>
__device__ __forceinline__ v8bf widen8(int d0, int d1) {
  const v2bf a = widen2<FMT, false>(d0), b = widen2<FMT, true>(d0);
  const v2bf c = widen2<FMT, false>(d1), d = widen2<FMT, true>(d1);
  return (v8bf){a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// Scales of the epilogue: SC = 0 one scale per product (dT[b], dS[b]);
// SC = 1 one per row of Tq_b (dT[b * Mb + x]) and per row of Sq_b, i.e. per
// column of the product (dS[b * Nb + z]).  Either way M = (acc * dT) * dS.

// Non-persistent variant: one 128 x 128 tile per workgroup, 4 waves.
template <int FMT, int ACC, int SC>
__global__ __launch_bounds__(kThreads) void gemm_tile_kernel(const uint8_t* __restrict__ Tq,
                                                            const uint8_t* __restrict__ Sq,
                                                            const float* __restrict__ dT,
                                                            const float* __restrict__ dS,
                                                            float* __restrict__ Mout, int Mb,
                                                            int Nb, int Kb, int tiles_m,
                                                            int tiles_n, int total) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][GT * GK];
  // Workgroups are dispatched round-robin over the 8 XCDs; remap so that
  // each XCD works through a contiguous range of tiles (whole products),
  // keeping a product's operand panels in one L2.
  int w = blockIdx.x;
  if ((total & 7) == 0) w = (w & 7) * (total >> 3) + (w >> 3);
  const int tiles = tiles_m * tiles_n;
  const int b = w / tiles;
  const int t = w - b * tiles;
  const int tm = t / tiles_n, tn = t - (t / tiles_n) * tiles_n;
  const int m0 = tm * GT, n0 = tn * GT;
  const uint8_t* Ab = Tq + (size_t)b * Mb * Kb;
  const uint8_t* Bb = Sq + (size_t)b * Nb * Kb;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  uint4 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + kThreads * i;
      const int row = c >> 3, ch = c & 7;
      const int kk = k0 + ch * 16;
      ra[i] = make_uint4(0, 0, 0, 0);
      rb[i] = make_uint4(0, 0, 0, 0);
      if (kk < Kb) {
        if (m0 + row < Mb) ra[i] = *reinterpret_cast<const uint4*>(Ab + (size_t)(m0 + row) * Kb + kk);
        if (n0 + row < Nb) rb[i] = *reinterpret_cast<const uint4*>(Bb + (size_t)(n0 + row) * Kb + kk);
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + kThreads * i;
      const int row = c >> 3, ch = c & 7;
      const int o = row * GK + ((ch ^ swz(row)) << 4);
      *reinterpret_cast<uint4*>(&lds[buf][0][o]) = ra[i];
      *reinterpret_cast<uint4*>(&lds[buf][1][o]) = rb[i];
    }
  };

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  const int nk = (Kb + GK - 1) / GK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int q = lane >> 4, l16 = lane & 15;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * GK);
    v8i fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = wm * 64 + i * 16 + l16;
      const uint8_t* base = &lds[cur][0][row * GK];
      const uint4 lo = *reinterpret_cast<const uint4*>(base + (((2 * q) ^ swz(row)) << 4));
      const uint4 hi = *reinterpret_cast<const uint4*>(base + (((2 * q + 1) ^ swz(row)) << 4));
      fa[i] = (v8i){(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = wn * 64 + j * 16 + l16;
      const uint8_t* base = &lds[cur][1][row * GK];
      const uint4 lo = *reinterpret_cast<const uint4*>(base + (((2 * q) ^ swz(row)) << 4));
      const uint4 hi = *reinterpret_cast<const uint4*>(base + (((2 * q + 1) ^ swz(row)) << 4));
      fb[j] = (v8i){(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    }
    if constexpr (ACC == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fa[i], fb[j], acc[i][j], FMT,
                                                                       FMT, 0, 127, 0, 127);
    } else {
#pragma unroll
      for (int sub = 0; sub < 4; ++sub) {
        v8bf wa[4], wb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) wa[i] = widen8<FMT>(fa[i][2 * sub], fa[i][2 * sub + 1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) wb[j] = widen8<FMT>(fb[j][2 * sub], fb[j][2 * sub + 1]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[i], wb[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  float* Mo = Mout + (size_t)b * Mb * Nb;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + wn * 64 + j * 16 + l16;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm * 64 + i * 16 + 4 * q + v;
        if (row < Mb && col < Nb) {
          const float sT = SC ? dT[(size_t)b * Mb + row] : dT[b];
          const float sS = SC ? dS[(size_t)b * Nb + col] : dS[b];
          float m = acc[i][j][v] * sT;
          m = m * sS;
          Mo[(size_t)row * Nb + col] = m;
        }
      }
    }
}

// Pipelined persistent kernel (inner block length a multiple of 128):
// workgroup tile 256 x 128, 8 waves of 64 x 64 (4 x 2), K step 128 bytes, a
// ring of 3 LDS stages of 48 KB filled by direct global-to-LDS loads
// (global_load_lds_dwordx4: lane L of a wave writes the 16 bytes it fetched
// at M0 + 16 L, so the XOR swizzle is applied by choosing each lane's source
// chunk).  Each workgroup walks a flattened sequence of (tile, K-step) pairs
// with two pairs in flight while it computes a third, so the next tile's
// loads run under the current tile's epilogue.  Rows beyond the operand
// (ragged M or N) read row 0 instead: they only feed outputs never stored.
//
// The ring, its direct loads and their vmcnt accounting are in
// fm_lds_ring.h.  The products are accumulated transposed (operands swapped
// in the MFMA) so that each lane holds 4 consecutive output columns and the
// epilogue writes 16-byte stores.
template <int FMT, int ACC, int SC, bool OB = false>
__global__ __launch_bounds__(DNT) void gemm_dma_kernel(const uint8_t* __restrict__ Tq,
                                                       const uint8_t* __restrict__ Sq,
                                                       const float* __restrict__ dT,
                                                       const float* __restrict__ dS,
                                                       float* __restrict__ Mout, int Mb, int Nb,
                                                       int Kb, int tiles_m, int tiles_n, int total,
                                                       int tiled) {
  // SC = 2 (group scales): every K step is one group of 128; its scales ride
  // the ring in a 2 KB slot after the stage (dT of the tile's 256 rows, then
  // the tile's one dS)
  constexpr int STG = SC == 2 ? DSTAGE + 2048 : DSTAGE;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[DNS * STG];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q = lane >> 4, l16 = lane & 15;
  const int tiles = tiles_m * tiles_n;
  const int nk = Kb / GK;
  const bool vec_store = (Nb & 3) == 0;

  const int G = gridDim.x;
  // (XCD x takes tiles [x per, (x + 1) per), per = ceil(total / 8))
  const bool xcd_split = (G & 7) == 0;
  const int per = (total + 7) >> 3;
  const int t = xcd_split ? (blockIdx.x & 7) * per + (blockIdx.x >> 3) : blockIdx.x;
  const int tstep = xcd_split ? (G >> 3) : G;
  const int t_end = xcd_split ? min(total, ((blockIdx.x & 7) + 1) * per) : total;
  if (t >= t_end) return;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;

  auto issue = [&](int tile, int kt, int buf) {
    const int b = tile / tiles, tt = tile - b * tiles;
    const int tmi = tt / tiles_n;
    const int m0 = tmi * DBM, n0 = (tt - tmi * tiles_n) * DBN;
    const uint8_t* Ab = Tq + (size_t)b * Mb * Kb + (size_t)kt * GK;
    const uint8_t* Bb = Sq + (size_t)b * Nb * Kb + (size_t)kt * GK;
#pragma unroll
    for (int j = 0; j < DLOADS; ++j) {
      const int r0 = (wave * DLOADS + j) * 8;  // first of the 8 rows this wave-load fills
      const int r = r0 + (lane >> 3);
      const int ch = (lane & 7) ^ swz(r);
      const uint8_t* src;
      if (r0 < DBM) {  // uniform: a wave-load never straddles the A/B boundary
        int row = m0 + r;
        row = row < Mb ? row : 0;
        src = Ab + (size_t)row * Kb + ch * 16;
      } else {
        int row = n0 + r - DBM;
        row = row < Nb ? row : 0;
        src = Bb + (size_t)row * Kb + ch * 16;
      }
      dma16(src, lds_base + (uint32_t)(buf * STG + r0 * GK));
    }
    if constexpr (SC == 2) {
      // wave 0: dT[b][kt][m0 + 4 lane .. + 3] (Mb a multiple of 4); wave 1:
      // the 16-byte-aligned chunk holding dS[b][kt][n0 / 128] (the scale
      // arrays are padded to whole chunks)
      if (wave < 2) {
        const size_t grp = (size_t)b * nk + kt;
        const float* src;
        if (wave == 0) {
          const int row = m0 + 4 * lane;
          src = dT + grp * Mb + (row < Mb ? row : 0);
        } else {
          src = dS + ((grp * (Nb / 128) + n0 / 128) & ~(size_t)3);
        }
        dma16(src, lds_base + (uint32_t)(buf * STG + DSTAGE + wave * 1024));
      }
    }
  };
  // Half h of a K step: lane (l16, q) of fragment i holds bytes
  // [32q + 16h, 32q + 16h + 16) of its row, i.e. the k values of two 16x16x32
  // sub-steps (2h and 2h + 1).
  uint4 fa[2][4], fb[2][4];
  auto read_half = [&](int h, int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = wm * 64 + i * 16 + l16;
      fa[h][i] = *reinterpret_cast<const uint4*>(lds + buf * STG + row * GK +
                                                 (((2 * q + h) ^ swz(row)) << 4));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = DBM + wn * 64 + j * 16 + l16;
      fb[h][j] = *reinterpret_cast<const uint4*>(lds + buf * STG + row * GK +
                                                 (((2 * q + h) ^ swz(row)) << 4));
    }
  };

  v4f acc[4][4];
  v4f ofl[4][4];  // SC = 2: the fp32 sum over the groups so far
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
      ofl[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
    }
  // SC = 2: the step's scales, read from its ring slot before the barrier
  float gs[4];
  auto read_scales = [&](int buf, int tile, int kt) {
    const float* sA = reinterpret_cast<const float*>(lds + buf * STG + DSTAGE);
    const float* sB = reinterpret_cast<const float*>(lds + buf * STG + DSTAGE + 1024);
    const int b = tile / tiles, tt = tile - b * tiles;
    const int n0 = (tt - (tt / tiles_n) * tiles_n) * DBN;
    const float ds = sB[(((size_t)b * nk + kt) * (Nb / 128) + n0 / 128) & 3];
#pragma unroll
    for (int i = 0; i < 4; ++i) gs[i] = sA[wm * 64 + i * 16 + l16] * ds;
  };
  // out = fmaf(group sum, dT dS, out), then the next group starts from zero
  auto rescale = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int v = 0; v < 4; ++v) ofl[i][j][v] = __builtin_fmaf(acc[i][j][v], gs[i], ofl[i][j][v]);
        acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
      }
  };

  // acc[i][j] holds the transposed 16 x 16 product: element (4q+v, l16) is
  // output row i*16 + l16, column j*16 + 4q + v of the wave's 64 x 64 block
  auto compute_half = [&](int h) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      if constexpr (ACC == 1) {
        long xa[4], xb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          xa[i] = sub ? (long)(((unsigned long)(uint32_t)fa[h][i].w << 32) | (uint32_t)fa[h][i].z)
                      : (long)(((unsigned long)(uint32_t)fa[h][i].y << 32) | (uint32_t)fa[h][i].x);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          xb[j] = sub ? (long)(((unsigned long)(uint32_t)fb[h][j].w << 32) | (uint32_t)fb[h][j].z)
                      : (long)(((unsigned long)(uint32_t)fb[h][j].y << 32) | (uint32_t)fb[h][j].x);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if constexpr (FMT == FM_E4M3)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8(xb[j], xa[i], acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf8_bf8(xb[j], xa[i], acc[i][j], 0, 0, 0);
          }
      } else {
        v8bf wa[4], wb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          wa[i] = sub ? widen8<FMT>((int)fa[h][i].z, (int)fa[h][i].w) : widen8<FMT>((int)fa[h][i].x, (int)fa[h][i].y);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          wb[j] = sub ? widen8<FMT>((int)fb[h][j].z, (int)fb[h][j].w) : widen8<FMT>((int)fb[h][j].x, (int)fb[h][j].y);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wb[j], wa[i], acc[i][j], 0, 0, 0);
      }
    }
  };
  auto epilogue = [&](int tile) -> int {  // returns the number of stores counted
    const int b = tile / tiles, tt = tile - b * tiles;
    const int tmi = tt / tiles_n;
    const int m0 = tmi * DBM, n0 = (tt - tmi * tiles_n) * DBN;
    float* Mo = Mout + (size_t)b * Mb * Nb;
    const int r_base = m0 + wm * 64 + l16, c_base = n0 + wn * 64 + 4 * q;
    int counted = 0;
    if constexpr (SC == 2) {
      // products returned in bf16 (nearest even), held as fp32
      auto bf = [](float x) {
        const uint32_t u = __float_as_uint(x);
        return __uint_as_float((u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u);
      };
      // OB: stored as bf16 (the values' high halves, 8-byte stores)
      uint16_t* Mh = reinterpret_cast<uint16_t*>(Mout) + (size_t)b * Mb * Nb;
      auto hi = [](float x) { return __float_as_uint(x) >> 16; };
      if (m0 + DBM <= Mb && n0 + DBN <= Nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float v0 = bf(ofl[i][j][0]), v1 = bf(ofl[i][j][1]);
            const float v2 = bf(ofl[i][j][2]), v3 = bf(ofl[i][j][3]);
            if constexpr (OB)
              *reinterpret_cast<uint2*>(Mh + (size_t)(r_base + i * 16) * Nb + c_base + j * 16) =
                  make_uint2(hi(v0) | (hi(v1) << 16), hi(v2) | (hi(v3) << 16));
            else
              *reinterpret_cast<float4*>(Mo + (size_t)(r_base + i * 16) * Nb + c_base + j * 16) =
                  make_float4(v0, v1, v2, v3);
          }
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
              if (row < Mb && col < Nb) {
                if constexpr (OB) Mh[(size_t)row * Nb + col] = (uint16_t)hi(bf(ofl[i][j][v]));
                else Mo[(size_t)row * Nb + col] = bf(ofl[i][j][v]);
              }
            }
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) ofl[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
    } else if (vec_store && m0 + DBM <= Mb && n0 + DBN <= Nb) {
      float sT[4];
      float4 sS[4];
      if constexpr (SC) {
#pragma unroll
        for (int i = 0; i < 4; ++i) sT[i] = dT[(size_t)b * Mb + r_base + i * 16];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          sS[j] = *reinterpret_cast<const float4*>(dS + (size_t)b * Nb + c_base + j * 16);
      } else {
        const float t = dT[b], u = dS[b];
#pragma unroll
        for (int i = 0; i < 4; ++i) sT[i] = t;
#pragma unroll
        for (int j = 0; j < 4; ++j) sS[j] = make_float4(u, u, u, u);
      }
      // tiled layout (full tiles only): the 16-byte pieces of a tile in
      // the order (wave, i, j, row l16, column group q), so each store of a
      // wave is one contiguous kilobyte
      float* tbase = Mo + (size_t)tt * (DBM * DBN) + (size_t)wave * 4096 + (l16 * 4 + q) * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float* prow = Mo + (size_t)(r_base + i * 16) * Nb + c_base;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float4 o;
          o.x = (acc[i][j][0] * sT[i]) * sS[j].x;
          o.y = (acc[i][j][1] * sT[i]) * sS[j].y;
          o.z = (acc[i][j][2] * sT[i]) * sS[j].z;
          o.w = (acc[i][j][3] * sT[i]) * sS[j].w;
          // whole lines of products read once, by the reconstruction:
          // non-temporal
          if (tiled)
            __builtin_nontemporal_store((v4f){o.x, o.y, o.z, o.w},
                                        reinterpret_cast<v4f*>(tbase + (i * 4 + j) * 256));
          else
            *reinterpret_cast<float4*>(prow + j * 16) = o;
        }
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
            if (row < Mb && col < Nb) {
              const float sT = SC ? dT[(size_t)b * Mb + row] : dT[b];
              const float sS = SC ? dS[(size_t)b * Nb + col] : dS[b];
              Mo[(size_t)row * Nb + col] = (acc[i][j][v] * sT) * sS;
            }
          }
      }
      // a data-dependent number of stores: counted as none (a lower bound)
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};
    return counted;
  };

  // Sequence of (tile, K-step) pairs p_0, p_1, ...; p_s lives in LDS buffer
  // s mod 3.  Iteration s: read the high half of p_s while the matrix cores
  // work on its low half; wait until p_{s+1} has landed and every wave is done
  // reading p_s; start the loads of p_{s+3} into the buffer of p_s; read the
  // low half of p_{s+1} while the matrix cores work on the high half of p_s.
  auto advance = [&](int& tt, int& kk) {
    if (++kk == nk) {
      kk = 0;
      tt += tstep;
    }
  };
  int t1 = t, k1 = 0;  // p_{s+1}
  advance(t1, k1);
  int t2 = t1, k2 = k1;  // p_{s+2}
  advance(t2, k2);
  int t3 = t2, k3 = k2;  // p_{s+3}
  advance(t3, k3);
  int ct = t, ck = 0;  // p_s
  issue(ct, ck, 0);
  int after1 = 0;  // vector-memory operations issued after the group of p_{s+1}
  if (t1 < t_end) issue(t1, k1, 1);
  if (t2 < t_end) {
    issue(t2, k2, 2);
    after1 = DLOADS;
  }
  wait_vm(t1 < t_end ? after1 + DLOADS : 0);  // p_0 has landed
  FM_COMPILER_FENCE();
  __builtin_amdgcn_s_barrier();
  FM_COMPILER_FENCE();
  read_half(0, 0);
  int cb = 0;  // buffer of p_s
  while (true) {
    read_half(1, cb);
    if constexpr (SC == 2) read_scales(cb, ct, ck);
    compute_half(0);
    wait_vm(after1);                     // p_{s+1} has landed (this wave's share)
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of p_s are done
    FM_COMPILER_FENCE();
    __builtin_amdgcn_s_barrier();
    FM_COMPILER_FENCE();
    const int nb = cb == 2 ? 0 : cb + 1;
    int after2 = 0;  // operations issued after the group of p_{s+2}
    if (t3 < t_end) {
      issue(t3, k3, cb);
      after2 = DLOADS;
    }
    FM_COMPILER_FENCE();
    const bool more = t1 < t_end;
    if (more) read_half(0, nb);
    compute_half(1);
    if constexpr (SC == 2) rescale();
    if (ck == nk - 1) after2 += epilogue(ct);
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


// Wide persistent kernel (tensor or row/column scales, bf16 products, Mb a
// multiple of 512, Nb of 128, Kb of 64): workgroup tile 512 x 128, K step 64
// bytes, a ring of 4 LDS stages of 40 KB (512 + 128 rows of 64 bytes; all
// 160 KB of the CU's LDS) filled by direct global-to-LDS loads two to three
// K steps ahead, 8 waves, two per SIMD.  Each wave computes 128 rows x 64
// columns = 4 x 2 tiles of 32 x 32 (v_mfma_f32_32x32x16_bf16, 128
// accumulators), so a widened A fragment feeds 2 matrix instructions and a
// B fragment 4, and the two waves of a SIMD share its matrix unit: while one
// issues its loads, LDS reads or conversions (which stall a wave, and with
// one wave per SIMD the matrix unit with it), the other's matrix
// instructions run.  Waves w and w + 4 (one SIMD) take the same 128 A rows
// (w % 4) and the two 64-column halves of B.  Per stage a wave loads 4 x 16
// A rows and 16 B rows (5 of the 40 wave-loads).  The raw codes of a stage
// are read from LDS in two halves (the first 16 bytes of each lane's 32,
// sub-steps 0 and 1; then the second), each as soon as the previous stage's
// half is widened, so one stage of raw codes and two sub-steps of widened
// fragments are held.
//
// Within a K step, lane (r, h) = (lane % 32, lane / 32) of a 32-row fragment
// holds the 32 bytes [32h, 32h + 32) of row r; sub-step t (16 k values)
// takes bytes [8t, 8t + 8) of them, for both operands alike (the 64 k values
// of the step are summed in another order than in gemm_dma_kernel: the
// products are exact, the fp32 sums differ only by rounding).  Rows of 64
// bytes hold their 4 chunks XOR-swizzled by (row / 4) % 4: the 16 lanes
// served per LDS cycle of a 16-byte fragment read (16 consecutive rows, 4
// rows per 256-byte bank window) then hit 16 distinct 16-byte bank groups.
namespace wide {
constexpr int BM = 512, BN = 128, KS = 64;

// global_load_lds_dwordx4 with a scalar base and a 32-bit per-lane offset:
// lane L writes the 16 bytes it fetched at M0 + 16 L (M0 written by SALU
// then read by an LDS-DMA load needs one wait state).  Device scope (sc1):
// the codes are used once, from LDS, so the CU's vector L1 need not keep
// them (measured a few percent faster than the default scope)
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 sc1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_addr)
               : "memory", "m0");
}
}  // namespace wide

typedef float v16f __attribute__((ext_vector_type(16)));

namespace wide8 {
constexpr int BM = 512, BN = 128, KS = 64, NT = 512, NSTG = 4;
constexpr int ROWS = BM + BN;         // rows of KS bytes per stage
constexpr int STAGE = ROWS * KS;      // 40 KB
constexpr int LOADS = ROWS / 16 / 8;  // 1 KB wave-loads per wave per stage (5)
constexpr int STORES = 32;            // 16-byte stores per lane per tile

// the counts used: after a tile's stores, or not; anything less waits for
// everything (a count above the one needed waits for more than needed)
__device__ __forceinline__ void wait_vm(int n) {
  if (n >= LOADS + 2 + STORES) ring::wait_vm_n<LOADS + 2 + STORES>();
  else if (n >= LOADS + 2) ring::wait_vm_n<LOADS + 2>();
  else ring::wait_vm_n<0>();
}
}  // namespace wide8

template <int FMT, int SC>
__global__ __launch_bounds__(wide8::NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_wide8_kernel(const uint8_t* __restrict__ Tq, const uint8_t* __restrict__ Sq,
                       const float* __restrict__ dT, const float* __restrict__ dS,
                       float* __restrict__ Mout, int Mb, int Nb, int Kb, int tiles_m, int tiles_n,
                       int total, int tiled) {
  using namespace wide8;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[NSTG * STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 3, wn = wave >> 2;
  const int r32 = lane & 31, h = lane >> 5;
  const int tiles = tiles_m * tiles_n;
  const int nk = Kb / KS;

  // workgroups go round-robin over the 8 XCDs: give each XCD a contiguous
  // range of tiles (whole products), so a product's operand panels stay in
  // one L2: XCD x takes tiles [x per, (x + 1) per), per = ceil(total / 8)
  const int G = gridDim.x;
  const bool xcd_split = (G & 7) == 0;
  const int per = (total + 7) >> 3;
  const int t = xcd_split ? (blockIdx.x & 7) * per + (blockIdx.x >> 3) : blockIdx.x;
  const int tstep = xcd_split ? (G >> 3) : G;
  const int t_end = xcd_split ? min(total, ((blockIdx.x & 7) + 1) * per) : total;
  if (t >= t_end) return;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;

  // A wave-load fills 16 rows of 64 bytes: lane L writes row L / 4, slot L %
  // 4, and fetches the chunk (L % 4) ^ ((row / 4) % 4); rows start at
  // multiples of 16, so the chunk and the row's offset in the operand depend
  // on the lane alone (one 32-bit offset), and the row block's address is
  // uniform (a scalar base)
  const uint32_t dma_off =
      (uint32_t)(lane >> 2) * (uint32_t)Kb + (uint32_t)(((lane & 3) ^ ((lane >> 4) & 3)) << 4);
  const size_t kb16 = (size_t)16 * Kb;
  // this wave's first A row (64 wave) and B row (16 wave) of a tile's panels
  auto tile_base = [&](int tile, const uint8_t*& Ab, const uint8_t*& Bb) {
    const int b = tile / tiles, tt = tile - b * tiles;
    const int tmi = tt / tiles_n;
    Ab = Tq + ((size_t)b * Mb + (size_t)tmi * BM + (size_t)wave * 64) * Kb;
    Bb = Sq + ((size_t)b * Nb + (size_t)(tt - tmi * tiles_n) * BN + (size_t)wave * 16) * Kb;
  };
  // wave-load j of a stage: j < 4 A rows 64 wave + 16 j, j = 4 B rows 16 wave
  auto dma_one = [&](const uint8_t* Ab, const uint8_t* Bb, int kt, int buf, int j) {
    const uint32_t l0 = lds_base + (uint32_t)(buf * STAGE);
    if (j < 4)
      wide::dma16s(Ab + j * kb16 + kt * KS, dma_off, l0 + (uint32_t)((wave * 64 + 16 * j) * KS));
    else
      wide::dma16s(Bb + kt * KS, dma_off, l0 + (uint32_t)((BM + wave * 16) * KS));
  };
  auto issue = [&](const uint8_t* Ab, const uint8_t* Bb, int kt, int buf) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) dma_one(Ab, Bb, kt, buf, j);
  };

  // one stage's raw codes: A rows 128 wm + 32 i + r32, B rows 64 wn + 32 j +
  // r32, 32 bytes each (two 16-byte chunks: sub-steps 0-1 and 2-3)
  uint4 ra[4][2], rb[2][2];
  const uint32_t rd0 = (uint32_t)r32 * KS + (uint32_t)(((2 * h) ^ ((r32 >> 2) & 3)) << 4);
  const uint32_t rd1 = (uint32_t)r32 * KS + (uint32_t)(((2 * h + 1) ^ ((r32 >> 2) & 3)) << 4);
  auto read_half = [&](int buf, auto cc) {
    constexpr int c = decltype(cc)::value;
    const uint32_t rd = c ? rd1 : rd0;
    const uint8_t* sa = lds + buf * STAGE + wm * 128 * KS;
    const uint8_t* sb = lds + buf * STAGE + (BM + wn * 64) * KS;
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[i][c] = *reinterpret_cast<const uint4*>(sa + i * 32 * KS + rd);
#pragma unroll
    for (int j = 0; j < 2; ++j) rb[j][c] = *reinterpret_cast<const uint4*>(sb + j * 32 * KS + rd);
  };
  using C0 = std::integral_constant<int, 0>;
  using C1 = std::integral_constant<int, 1>;
  auto sel = [](const uint4 (&r)[2], int tsub, int d) -> int {
    const uint4& c = r[tsub >> 1];
    return (tsub & 1) ? (d ? (int)c.w : (int)c.z) : (d ? (int)c.y : (int)c.x);
  };
  v8bf wa[2][4], wb[2][2];  // widened fragments of two sub-steps
  auto widen_sub = [&](int tsub, int slot) {
#pragma unroll
    for (int i = 0; i < 4; ++i) wa[slot][i] = widen8<FMT>(sel(ra[i], tsub, 0), sel(ra[i], tsub, 1));
#pragma unroll
    for (int j = 0; j < 2; ++j) wb[slot][j] = widen8<FMT>(sel(rb[j], tsub, 0), sel(rb[j], tsub, 1));
  };
  auto pin = [&](int slot) {
#pragma unroll
    for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(wa[slot][i]));
#pragma unroll
    for (int j = 0; j < 2; ++j) asm volatile("" : "+v"(wb[slot][j]));
  };

  // acc[i][j]: the transposed 32 x 32 product, element v of lane (r32, h)
  // at row i*32 + r32, column j*32 + 8 (v / 4) + 4 h + v % 4 of the wave's
  // 128 x 64 block
  v16f acc[4][2];
  auto epilogue = [&](int tile) {
    const int b = tile / tiles, tt = tile - b * tiles;
    const int tmi = tt / tiles_n;
    const int m0 = tmi * BM, n0 = (tt - tmi * tiles_n) * BN;
    float* Mo = Mout + (size_t)b * Mb * Nb;
    const int r_base = m0 + wm * 128 + r32, c_base = n0 + wn * 64 + 4 * h;
    // tiled layout: pieces in the order (row block wm, i, column tile 2 wn +
    // j, column group g, lane), one contiguous kilobyte per wave store
    float* tbase = Mo + (size_t)tt * (BM * BN) + (size_t)wm * (128 * 128) + lane * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = r_base + i * 32;
      const float sT = SC == 1 ? dT[(size_t)b * Mb + row] : dT[b];
      float* prow = Mo + (size_t)row * Nb + c_base;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float4 sS;
          if constexpr (SC == 1) {
            sS = *reinterpret_cast<const float4*>(dS + (size_t)b * Nb + c_base + j * 32 + 8 * g);
          } else {
            const float u = dS[b];
            sS = make_float4(u, u, u, u);
          }
          v4f o;
          o[0] = (acc[i][j][4 * g + 0] * sT) * sS.x;
          o[1] = (acc[i][j][4 * g + 1] * sT) * sS.y;
          o[2] = (acc[i][j][4 * g + 2] * sT) * sS.z;
          o[3] = (acc[i][j][4 * g + 3] * sT) * sS.w;
          if (tiled)
            __builtin_nontemporal_store(
                o, reinterpret_cast<v4f*>(tbase + ((i * 4 + 2 * wn + j) * 4 + g) * 256));
          else
            *reinterpret_cast<v4f*>(prow + j * 32 + 8 * g) = o;
        }
      }
    }
  };

  // Iteration s over the (tile, K step) pairs p_s, in four phases of 8
  // matrix instructions (one sub-step each), with the 5 wave-loads of
  // p_{s+3} (into the buffer of p_{s-1}) after matrix instructions 1 and 5:
  //   A: sub-step 0 (slot 0), widening sub-step 1 into slot 1; 2 loads;
  //   wait until p_{s+1} has landed and every wave's reads of p_s are done;
  //   B: sub-step 1 (slot 1), widening sub-step 2 into slot 0, reading the
  //      first half of p_{s+1}; 1 load;
  //   C: sub-step 2 (slot 0), widening sub-step 3 into slot 1; 1 load;
  //   D: sub-step 3 (slot 1), reading the second half of p_{s+1}, widening
  //      its sub-step 0 into slot 0; 1 load.
  auto advance = [&](int& tt, int& kk) {
    if (++kk == nk) {
      kk = 0;
      tt += tstep;
    }
  };
  auto mma_dma = [&](int slot, const uint8_t* Ab, const uint8_t* Bb, int kt, int buf, auto j0c,
                     auto j1c) {
    constexpr int j0 = decltype(j0c)::value, j1 = decltype(j1c)::value;
    sfor<0, 8>([&](auto qc) {
      constexpr int q = decltype(qc)::value;
      acc[q >> 1][q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wb[slot][q & 1], wa[slot][q >> 1], acc[q >> 1][q & 1], 0, 0, 0);
      if constexpr (q % 4 == 1 && j0 + q / 4 < j1) dma_one(Ab, Bb, kt, buf, j0 + q / 4);
    });
  };
  // 8 matrix instructions, each followed by N vector-ALU and R LDS-read
  // instructions (R for the first 6 only)
  auto groups = [](auto nc, auto rc) {
    constexpr int N = decltype(nc)::value, R = decltype(rc)::value;
    sfor<0, 8>([&](auto qc) {
      constexpr int q = decltype(qc)::value;
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if constexpr (R > 0 && q < 6) __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, N, 0);
    });
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  using I5 = std::integral_constant<int, 5>;
  int t1 = t, k1 = 0;  // p_{s+1}
  advance(t1, k1);
  int t2 = t1, k2 = k1;  // p_{s+2}
  advance(t2, k2);
  int t3 = t2, k3 = k2;  // p_{s+3}
  advance(t3, k3);
  const uint8_t *A0, *B0;
  tile_base(t, A0, B0);
  issue(A0, B0, 0, 0);
  int after1 = 0;  // vector-memory operations issued after the group of p_{s+1}
  if (t1 < t_end) {
    if (t1 != t) tile_base(t1, A0, B0);
    issue(A0, B0, k1, 1);
  }
  if (t2 < t_end) {
    if (t2 != t1) tile_base(t2, A0, B0);
    issue(A0, B0, k2, 2);
    after1 += LOADS;
  }
  const uint8_t *A3 = A0, *B3 = B0;  // panels of the tile of p_{s+3}
  if (t3 < t_end && t3 != t2) tile_base(t3, A3, B3);
  wait_vm(t1 < t_end ? after1 + LOADS : 0);  // p_0 has landed
  FM_COMPILER_FENCE();
  __builtin_amdgcn_s_barrier();
  FM_COMPILER_FENCE();
  read_half(0, C0{});
  read_half(0, C1{});
  widen_sub(0, 0);
  int cb = 0;  // buffer of p_s
  bool more = true;
  for (int tile = t; more; tile += tstep) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
    for (int kk = 0; kk < nk; ++kk) {
      const int b3 = cb == 0 ? NSTG - 1 : cb - 1;  // buffer of p_{s+3} (that of p_{s-1})
      // A
      mma_dma(0, A3, B3, k3, b3, I0{}, I2{});
      widen_sub(1, 1);
      groups(std::integral_constant<int, 3>{}, I0{});
      pin(1);
      __builtin_amdgcn_sched_barrier(0);
      // p_{s+1} was issued before p_{s+2}'s 5 loads and 2 of p_{s+3}
      wait_vm(after1 + 2);
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of p_s are done
      FM_COMPILER_FENCE();
      __builtin_amdgcn_s_barrier();
      FM_COMPILER_FENCE();
      const int nb = cb == NSTG - 1 ? 0 : cb + 1;
      more = t1 < t_end;
      // B
      mma_dma(1, A3, B3, k3, b3, I2{}, I3{});
      widen_sub(2, 0);
      read_half(nb, C0{});
      groups(std::integral_constant<int, 3>{}, I1{});
      pin(0);
      __builtin_amdgcn_sched_barrier(0);
      // C
      mma_dma(0, A3, B3, k3, b3, I3{}, I4{});
      widen_sub(3, 1);
      groups(std::integral_constant<int, 3>{}, I0{});
      pin(1);
      __builtin_amdgcn_sched_barrier(0);
      // D
      mma_dma(1, A3, B3, k3, b3, I4{}, I5{});
      read_half(nb, C1{});
      widen_sub(0, 0);
      groups(std::integral_constant<int, 3>{}, I1{});
      pin(0);
      __builtin_amdgcn_sched_barrier(0);
      t1 = t2;
      k1 = k2;
      t2 = t3;
      k2 = k3;
      advance(t3, k3);
      if (k3 == 0 && t3 < t_end) tile_base(t3, A3, B3);
      after1 = LOADS;
      cb = nb;
    }
    epilogue(tile);
    after1 += STORES;
  }
  ring::wait_vm_n<0>();  // the loads past the last pair land before the workgroup ends
}

}  // namespace

namespace {
int g_block_product_arith = FM_ACC_BF16;

// The wide kernel is the default where it applies; FM_BLOCK_GEMM=dma in the
// environment selects gemm_dma_kernel instead (for comparisons).
bool wide_enabled() {
  static const bool on = [] {
    const char* e = std::getenv("FM_BLOCK_GEMM");
    return !(e && std::strcmp(e, "dma") == 0);
  }();
  return on;
}

bool use_wide(int Mb, int Nb, int Kb, int sc, bool out_bf16) {
  return wide_enabled() && g_block_product_arith == FM_ACC_BF16 && (sc == 0 || sc == 1) &&
         !out_bf16 && Mb % wide::BM == 0 && Nb % wide::BN == 0 && Kb % wide::KS == 0;
}
}  // namespace

int block_gemm_tile_rows(int Mb, int Nb, int Kb, int scale_mode, bool out_bf16) {
  const int sc = scale_mode == FM_SCALE_ROWCOL ? 1 : (scale_mode == FM_SCALE_GROUP ? 2 : 0);
  if (use_wide(Mb, Nb, Kb, sc, out_bf16)) return wide::BM;
  if (Kb % GK == 0) return DBM;
  return 0;
}

int set_block_product_arith(int a) {
  if (a != FM_ACC_BF16 && a != FM_ACC_FP8) return fail(FM_E_ARG, "unknown product arithmetic");
  g_block_product_arith = a;
  return FM_OK;
}

namespace {
template <int SC, bool OB = false>
int launch_block_gemm_sc(const uint8_t* Tq, const uint8_t* Sq, const float* dT, const float* dS,
                         float* Mout, int batch, int Mb, int Nb, int Kb, int fmt, hipStream_t st,
                         int tiled = 0) {
  const bool fp8acc = g_block_product_arith == FM_ACC_FP8;
  if (use_wide(Mb, Nb, Kb, SC, OB)) {
    if constexpr (SC == 0 || SC == 1) {
      // persistent: one 160 KB-LDS workgroup of 4 waves per CU
      const int tm = Mb / wide::BM, tn = Nb / wide::BN;
      const long long total = (long long)batch * tm * tn;
      if (total > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many GEMM tiles in one launch");
      const int T = (int)total;
      const int grid = (int)std::min<long long>(total, 256);
      if (tiled && SC != 0)
        return fail(FM_E_UNSUPPORTED, "the tiled product layout needs tensor scales");
      if (fmt == FM_E4M3)
        gemm_wide8_kernel<FM_E4M3, SC><<<grid, wide8::NT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
      else
        gemm_wide8_kernel<FM_E5M2, SC><<<grid, wide8::NT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
      return launched("gemm_wide8_kernel");
    }
  }
  if (Kb % GK == 0) {
    // pipelined persistent kernel: one 144 KB-LDS workgroup per CU
    const int tm = (Mb + DBM - 1) / DBM, tn = (Nb + DBN - 1) / DBN;
    const long long total = (long long)batch * tm * tn;
    if (total > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many GEMM tiles in one launch");
    const int T = (int)total;
    const int grid = (int)std::min<long long>(total, 256);
    if (tiled && (SC != 0 || Mb % DBM || Nb % DBN))
      return fail(FM_E_UNSUPPORTED, "the tiled product layout needs whole tiles and tensor scales");
    if (fmt == FM_E4M3) {
      if (fp8acc) gemm_dma_kernel<FM_E4M3, 1, SC, OB><<<grid, DNT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
      else gemm_dma_kernel<FM_E4M3, 0, SC, OB><<<grid, DNT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
    } else {
      if (fp8acc) gemm_dma_kernel<FM_E5M2, 1, SC, OB><<<grid, DNT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
      else gemm_dma_kernel<FM_E5M2, 0, SC, OB><<<grid, DNT, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T, tiled);
    }
    return launched("gemm_dma_kernel");
  }
  if (tiled) return fail(FM_E_UNSUPPORTED, "the tiled product layout needs inner blocks of 128");
  if constexpr (SC == 2) {
    return fail(FM_E_SHAPE, "group scales need inner blocks of a multiple of 128");
  } else {
  // inner length a multiple of 16 only: one 128 x 128 tile per workgroup
  const int tm = (Mb + GT - 1) / GT, tn = (Nb + GT - 1) / GT;
  const long long total = (long long)batch * tm * tn;
  if (total > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many GEMM tiles in one launch");
  const int T = (int)total;
  if (fmt == FM_E4M3) {
    if (fp8acc) gemm_tile_kernel<FM_E4M3, 1, SC><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
    else gemm_tile_kernel<FM_E4M3, 0, SC><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
  } else {
    if (fp8acc) gemm_tile_kernel<FM_E5M2, 1, SC><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
    else gemm_tile_kernel<FM_E5M2, 0, SC><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
  }
  return launched("gemm_tile_kernel");
  }
}
}  // namespace

int launch_block_gemm(const uint8_t* Tq, const uint8_t* Sq, const float* dT, const float* dS,
                      float* Mout, int batch, int Mb, int Nb, int Kb, int fmt, int scale_mode,
                      hipStream_t st, bool out_bf16, bool tiled) {
  if (tiled && scale_mode != FM_SCALE_TENSOR)
    return fail(FM_E_UNSUPPORTED, "the tiled product layout needs tensor scales");
  if (scale_mode == FM_SCALE_ROWCOL)
    return launch_block_gemm_sc<1>(Tq, Sq, dT, dS, Mout, batch, Mb, Nb, Kb, fmt, st);
  if (scale_mode == FM_SCALE_GROUP) {
    if (Kb % 128 || Nb % 128 || Mb % 4)
      return fail(FM_E_SHAPE, "group scales need Kb, Nb multiples of 128 and Mb of 4");
    if (out_bf16)
      return launch_block_gemm_sc<2, true>(Tq, Sq, dT, dS, Mout, batch, Mb, Nb, Kb, fmt, st);
    return launch_block_gemm_sc<2>(Tq, Sq, dT, dS, Mout, batch, Mb, Nb, Kb, fmt, st);
  }
  return launch_block_gemm_sc<0>(Tq, Sq, dT, dS, Mout, batch, Mb, Nb, Kb, fmt, st, tiled ? 1 : 0);
}

}  // namespace fm
