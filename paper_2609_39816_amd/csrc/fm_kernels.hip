// HIP kernels of libfm for CDNA4 (gfx950), wave64.
//
//  form_kernel      block sums of an operand for every product of a chunk of
//                   gauged schemes (eq. (1), Sec. 2.1), in two modes: per-
//                   tensor amax (atomic max on the uint bits of |x|), then
//                   FP8 codes of x * (FMAX / amax) (App. B.1 schedule).
//  gemm_fp8_kernel  batched block products M_r on FP8 operands with the
//                   gfx950 matrix cores (v_mfma_scale_f32_16x16x128_f8f6f4,
//                   unit scales), fp32 accumulation, scale epilogue.
//  recon_kernel     C_ij = sum_r w_{r,ij} M_r (eq. (1)) with the squared
//                   error against the float64 reference reduced on chip.
//  ref_f64_kernel   float64 reference product (App. F).
// plus small kernels: fill, transpose, scales, fixed-order reductions.
//
// Arithmetic contract (matched bit for bit by the CPU oracle for everything
// up to the FP8 codes and scales): fp32 fused multiply-adds in the order of
// the coefficient lists, accumulators from +0, correctly rounded fp32
// divisions for the scales, one fp32 multiply before FP8 rounding (nearest
// even).  Built with -ffp-contract=off and fp32 denormals kept.
#include <hip/hip_runtime.h>

#include "fm_device.h"


namespace fm {
namespace {
using namespace dev;

__global__ void fp8_encode_kernel(const float* x, uint8_t* out, size_t n, int fmt, int impl) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint32_t c;
  if (impl == 1)
    c = enc2<1>(x[i], 0.0f, fmt);
  else if (impl == 2)
    c = enc2<0>(x[i], 0.0f, fmt);
  else
    c = enc2d(x[i], 0.0f, fmt);
  out[i] = (uint8_t)(c & 0xffu);
}

// ------------------------------------------------------------------ fill
__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ------------------------------------------------------------- transpose
// Xt (cols x rows) = X^T through a padded 32 x 32 LDS tile.
__global__ __launch_bounds__(256) void transpose_kernel(const float* __restrict__ X,
                                                        float* __restrict__ Xt, int rows,
                                                        int cols) {
  __shared__ float tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int k = 0; k < 32; k += 8) {
    const int r = r0 + ty + k, c = c0 + tx;
    if (r < rows && c < cols) tile[ty + k][tx] = X[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int k = 0; k < 32; k += 8) {
    const int c = c0 + ty + k, r = r0 + tx;
    if (r < rows && c < cols) Xt[(size_t)c * rows + r] = tile[tx][ty + k];
  }
}

// --------------------------------------------------------------- scales
__global__ void scales_kernel(const uint32_t* amax, float* q, float* d, int n, float fmax,
                              uint32_t* flag) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t u = amax[i];
  if (u >= 0x7f800000u) {
    atomicOr(flag, 1u);
    q[i] = 1.0f;
    d[i] = 1.0f;
    return;
  }
  const float m = __uint_as_float(u);
  if (m == 0.0f) {
    q[i] = 1.0f;
    d[i] = 1.0f;
  } else {
    q[i] = __fdiv_rn(fmax, m);
    d[i] = __fdiv_rn(m, fmax);
  }
}

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
constexpr int GK = 128;  // K step in bytes

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

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

template <int FMT, int ACC>
__global__ __launch_bounds__(kThreads) void gemm_fp8_kernel(const uint8_t* __restrict__ Tq,
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

  const float sT = dT[b], sS = dS[b];
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
          float m = acc[i][j][v] * sT;
          m = m * sS;
          Mo[(size_t)row * Nb + col] = m;
        }
      }
    }
}

__global__ void reduce_rows_kernel(const double* partial, int nblk, int G, double* out) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  double s = 0.0;
  for (int b = 0; b < nblk; ++b) s = s + partial[(size_t)g * nblk + b];
  out[g] = s;
}

// ----------------------------------------------------- float64 reference
// 64 x 64 output tile per workgroup, 4 x 4 per thread, K step 16; operands
// staged in LDS as fp32 and widened to float64 (products of two fp32 values
// are exact in float64).
__global__ __launch_bounds__(kThreads) void ref_f64_kernel(const float* __restrict__ A,
                                                           const float* __restrict__ B,
                                                           double* __restrict__ C, int M, int N,
                                                           int K) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double c[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + kThreads * i;
      const int row = idx >> 4, kk = idx & 15;
      const int gr = m0 + row, gk = k0 + kk;
      As[kk][row] = (gr < M && gk < K) ? A[(size_t)gr * K + gk] : 0.0f;
      const int kb = idx >> 6, col = idx & 63;
      const int gkb = k0 + kb, gc = n0 + col;
      Bs[kb][col] = (gkb < K && gc < N) ? B[(size_t)gkb * N + gc] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      const float4 av = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
      const float4 bv = *reinterpret_cast<const float4*>(&Bs[kk][tx * 4]);
      const double a4[4] = {(double)av.x, (double)av.y, (double)av.z, (double)av.w};
      const double b4[4] = {(double)bv.x, (double)bv.y, (double)bv.z, (double)bv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) c[i][j] = __fma_rn(a4[i], b4[j], c[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col < N) C[(size_t)row * N + col] = c[i][j];
    }
  }
}

// --------------------------------------------------------- error stats
__global__ __launch_bounds__(kThreads) void error_stats_kernel(const float* __restrict__ C,
                                                               const double* __restrict__ Cref,
                                                               size_t n, double* partial) {
  __shared__ double r0[kThreads], r1[kThreads], r2[kThreads];
  double e = 0.0, rs = 0.0, mx = 0.0;
  for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (size_t)gridDim.x * kThreads) {
    const double ref = Cref[i];
    const double d = (C ? (double)C[i] : 0.0) - ref;
    e = __fma_rn(d, d, e);
    rs = __fma_rn(ref, ref, rs);
    mx = fmax(mx, fabs(d));
  }
  r0[threadIdx.x] = e;
  r1[threadIdx.x] = rs;
  r2[threadIdx.x] = mx;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      r0[threadIdx.x] = r0[threadIdx.x] + r0[threadIdx.x + s];
      r1[threadIdx.x] = r1[threadIdx.x] + r1[threadIdx.x + s];
      r2[threadIdx.x] = fmax(r2[threadIdx.x], r2[threadIdx.x + s]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    partial[3 * blockIdx.x] = r0[0];
    partial[3 * blockIdx.x + 1] = r1[0];
    partial[3 * blockIdx.x + 2] = r2[0];
  }
}

__global__ void error_finalize_kernel(const double* partial, int nblk, double* out3) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double e = 0.0, r = 0.0, m = 0.0;
  for (int b = 0; b < nblk; ++b) {
    e = e + partial[3 * b];
    r = r + partial[3 * b + 1];
    m = fmax(m, partial[3 * b + 2]);
  }
  out3[0] = e;
  out3[1] = r;
  out3[2] = m;
}


}  // namespace

int launch_fill_u32(uint32_t* p, size_t n, uint32_t value, hipStream_t st) {
  if (n == 0) return FM_OK;
  const int grid = (int)std::min<size_t>((n + kThreads - 1) / kThreads, 4096);
  fill_u32_kernel<<<grid, kThreads, 0, st>>>(p, n, value);
  return launched("fill_u32_kernel");
}

int launch_transpose(const float* X, float* Xt, int rows, int cols, hipStream_t st) {
  dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  transpose_kernel<<<grid, kThreads, 0, st>>>(X, Xt, rows, cols);
  return launched("transpose_kernel");
}

int launch_form(const FormArgs& a, int mode, int pattern, int side, hipStream_t st) {
  if (a.gr * a.gc > 64) return fail(FM_E_UNSUPPORTED, "block grid larger than 64 blocks per operand");
  int id = 0;
#define FM_FORM_CASE(P)                                        \
  if (pattern == id) {                                         \
    const int rc = form_family_##P(a, mode, side, st);         \
    if (rc != 1) return rc;                                    \
  }                                                            \
  ++id;
  FM_PATTERN_FAMILIES(FM_FORM_CASE)
#undef FM_FORM_CASE
  return launch_form_generic(a, mode, st);
}

int launch_scales(const uint32_t* amax, float* q, float* d, int n, int fmt, uint32_t* flag,
                  hipStream_t st) {
  const float fmax = fmt == FM_E4M3 ? 448.0f : 57344.0f;
  scales_kernel<<<(n + kThreads - 1) / kThreads, kThreads, 0, st>>>(amax, q, d, n, fmax, flag);
  return launched("scales_kernel");
}

namespace {
int g_block_product_arith = FM_ACC_BF16;
}

int set_block_product_arith(int a) {
  if (a != FM_ACC_BF16 && a != FM_ACC_FP8) return fail(FM_E_ARG, "unknown product arithmetic");
  g_block_product_arith = a;
  return FM_OK;
}

int launch_block_gemm(const uint8_t* Tq, const uint8_t* Sq, const float* dT, const float* dS,
                      float* Mout, int batch, int Mb, int Nb, int Kb, int fmt, hipStream_t st) {
  const int tm = (Mb + GT - 1) / GT, tn = (Nb + GT - 1) / GT;
  const long long total = (long long)batch * tm * tn;
  if (total > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many GEMM tiles in one launch");
  const int T = (int)total;
  const bool fp8acc = g_block_product_arith == FM_ACC_FP8;
  if (fmt == FM_E4M3) {
    if (fp8acc)
      gemm_fp8_kernel<FM_E4M3, 1><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
    else
      gemm_fp8_kernel<FM_E4M3, 0><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
  } else {
    if (fp8acc)
      gemm_fp8_kernel<FM_E5M2, 1><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
    else
      gemm_fp8_kernel<FM_E5M2, 0><<<T, kThreads, 0, st>>>(Tq, Sq, dT, dS, Mout, Mb, Nb, Kb, tm, tn, T);
  }
  return launched("gemm_fp8_kernel");
}

int recon_blocks(const ReconArgs& a) {
  // the same for every kernel choice: positions counted at width 4 when the
  // shape allows it, else 1
  const int vw = (a.Nb % 4 == 0 && a.N % 4 == 0) ? 4 : 1;
  const int P = a.Mb * (a.Nb / vw);
  const int nblk = (P + kThreads - 1) / kThreads;
  const int target = std::max(64, 4096 / std::max(1, a.G));
  return std::max(1, std::min(nblk, target));
}

int launch_recon(const ReconArgs& a, int pattern, hipStream_t st) {
  if (a.gm * a.gn > 64) return fail(FM_E_UNSUPPORTED, "output grid larger than 64 blocks");
  int id = 0;
#define FM_RECON_CASE(P)                          \
  if (pattern == id) {                            \
    const int rc = recon_family_##P(a, st);       \
    if (rc != 1) return rc;                       \
  }                                               \
  ++id;
  FM_PATTERN_FAMILIES(FM_RECON_CASE)
#undef FM_RECON_CASE
  return launch_recon_generic(a, st);
}

int launch_reduce_rows(const double* partial, int nblk, int G, double* out, hipStream_t st) {
  reduce_rows_kernel<<<(G + 63) / 64, 64, 0, st>>>(partial, nblk, G, out);
  return launched("reduce_rows_kernel");
}

int launch_reference_f64(const float* A, const float* B, double* C, int M, int N, int K,
                         hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  ref_f64_kernel<<<grid, kThreads, 0, st>>>(A, B, C, M, N, K);
  return launched("ref_f64_kernel");
}

int error_stats_blocks(size_t n) {
  return (int)std::max<size_t>(1, std::min<size_t>((n + kThreads - 1) / kThreads, 1024));
}

int launch_error_stats(const float* C, const double* Cref, size_t n, double* partial,
                       hipStream_t st) {
  error_stats_kernel<<<error_stats_blocks(n), kThreads, 0, st>>>(C, Cref, n, partial);
  return launched("error_stats_kernel");
}

int launch_error_finalize(const double* partial, int nblk, double* out3, hipStream_t st) {
  error_finalize_kernel<<<1, 64, 0, st>>>(partial, nblk, out3);
  return launched("error_finalize_kernel");
}

int launch_fp8_encode(const float* x, uint8_t* out, size_t n, int fmt, int impl, hipStream_t st) {
  if (n == 0) return FM_OK;
  fp8_encode_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, st>>>(x, out, n, fmt,
                                                                                   impl);
  return launched("fp8_encode_kernel");
}

}  // namespace fm
