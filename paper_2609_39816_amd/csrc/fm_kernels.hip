// HIP kernels of libfm for CDNA4 (gfx950), wave64.
//
//  form_kernel      block sums of an operand for every product of a chunk of
//                   gauged schemes (eq. (1), Sec. 2.1), in two modes: per-
//                   tensor amax (atomic max on the uint bits of |x|), then
//                   FP8 codes of x * (FMAX / amax) (App. B.1 schedule).
//  (block products: fm_gemm.hip)
//  recon_kernel     C_ij = sum_r w_{r,ij} M_r (eq. (1)) with the squared
//                   error against the float64 reference reduced on chip.
//  ref_f64_mfma_kernel  float64 reference product (App. F) on the float64
//                   matrix cores.
// plus small kernels: fill, transpose, scales, fixed-order reductions.
//
// Arithmetic contract (matched bit for bit by the CPU oracle for everything
// up to the FP8 codes and scales): fp32 fused multiply-adds in the order of
// the coefficient lists, accumulators from +0, correctly rounded fp32
// divisions for the scales, one fp32 multiply before FP8 rounding (nearest
// even).  Built with -ffp-contract=off and fp32 denormals kept.
#include <hip/hip_runtime.h>

#include "fm_device.h"
#include "fm_joint.h"


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

__global__ void bf16_round_kernel(const float* x, float* out, size_t n, int impl) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float v = x[i];
  if (impl == 2) {
    v = bf16_round_int(v);
  } else {
    float w = v;
    bf16_round_pair(v, w);
  }
  out[i] = v;
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

// ------------------------------------------------------------- repairs
// Outside power-of-two row scaling (the repair rules): one wave per row t of
// A computes the float64 sum of squares (lane l over the indices = l mod 64
// in ascending order, then the fixed butterfly), m2 = sum / K, the least k
// with 4^k >= m2 (at least -9; a non-finite row gets 0), writes
// As[t] = A[t] * 2^-k and up[t] = 2^k.
__global__ __launch_bounds__(kThreads) void row_repair_kernel(const float* __restrict__ A, int M,
                                                              int K, float* __restrict__ As,
                                                              float* __restrict__ up) {
  const int lane = threadIdx.x & 63;
  const long long t = (long long)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (t >= M) return;
  const float* x = A + (size_t)t * K;
  double s = 0.0;
  for (int i = lane; i < K; i += 64) s += (double)x[i] * (double)x[i];
  for (int off = 32; off > 0; off >>= 1) s = s + __shfl_xor(s, off, 64);
  const double m2 = s / (double)K;
  int k;
  if (!isfinite(m2)) {
    k = 0;
  } else if (m2 == 0.0) {
    k = -9;
  } else {
    int e;
    const double fr = frexp(m2, &e);
    const int c = fr == 0.5 ? e - 1 : e;
    k = c >= 0 ? (c + 1) / 2 : -((-c) / 2);
    k = k < -9 ? -9 : k;
  }
  const float down = ldexpf(1.0f, -k);
  float* y = As + (size_t)t * K;
  for (int i = lane; i < K; i += 64) y[i] = x[i] * down;
  if (lane == 0) up[t] = ldexpf(1.0f, k);
}

// Joint rounding of B's bf16 block sums (the repair rules), one thread per
// position (z, k) of the block sums (B^T orientation) of gauge g: every
// product's block sum there (the formation's fmaf order, then bf16), the
// two codes bracketing s q, the start at the value-nearer one, then sweeps
// over r with the fp32 decisions of the definition; writes all R codes.  A
// workgroup (one wave) covers 64 consecutive k of one row z, inside one
// 128 x 128 block.  LDS: the gauge's H, the block's scales q and d per
// product, and per thread (column `lane` of R x 64 arrays) its block sums,
// errors, H e and the candidate codes.
__global__ __launch_bounds__(kJointLanes) void joint_round_kernel(FormArgs a,
                                                                  const float* __restrict__ qS,
                                                                  const float* __restrict__ dS,
                                                                  JointH hg, int max_sweeps) {
  extern __shared__ float sm[];
  const int R = a.R;
  const int lane = threadIdx.x;
  const int g = blockIdx.y;
  const int32_t* hpg = hg.hp + (size_t)g * (R + 1);
  const int nnz = hpg[R];
  float* hv = sm;                                              // nnz
  float* qs = hv + R * R;                                      // R
  float* dsc = qs + R;                                         // R
  float* hd = dsc + R;                                         // R: the diagonal
  float* ev = hd + R;                                          // R x 64
  float* gv = ev + R * kJointLanes;                            // R x 64
  uint32_t* pk = reinterpret_cast<uint32_t*>(gv + R * kJointLanes);  // R x 64
  int32_t* hp = reinterpret_cast<int32_t*>(pk + R * kJointLanes);    // R + 1
  uint16_t* hc = reinterpret_cast<uint16_t*>(hp + R + 1);            // nnz
  const int nkg = a.bc / kGroup, nzb = a.br / kGroup;
  const int per_row = a.bc / kJointLanes;
  const int z = blockIdx.x / per_row, k = (blockIdx.x - z * per_row) * kJointLanes + lane;
  const int kg = k / kGroup, zb = z / kGroup;
  for (int i = lane; i < nnz; i += kJointLanes) {
    hv[i] = hg.hv[(size_t)g * R * R + i];
    hc[i] = hg.hc[(size_t)g * R * R + i];
  }
  for (int i = lane; i <= R; i += kJointLanes) hp[i] = hpg[i];
  for (int r = lane; r < R; r += kJointLanes) {
    const size_t o = ((size_t)((size_t)g * a.R + r) * nkg + kg) * nzb + zb;
    qs[r] = qS[o];
    dsc[r] = dS[o];
  }
  __syncthreads();
  for (int r = lane; r < R; r += kJointLanes) {
    float h = 0.0f;
    for (int i = hp[r]; i < hp[r + 1]; ++i)
      if (hc[i] == r) h = hv[i];
    hd[r] = h;
  }
  __syncthreads();
  const auto off = ro(a.off);
  // pk: bits 0-7 the nearest code, 8-15 its neighbour (bit 16: none),
  // bit 17: the neighbour is the current choice
  for (int r = 0; r < R; ++r) {
    const int e0 = off[(size_t)g * (a.R + 1) + r], e1 = off[(size_t)g * (a.R + 1) + r + 1];
    float acc = 0.0f;
    for (int i = e0; i < e1; ++i) {
      const float c = ro(a.coef)[i];
      const int b = ro(a.idx)[i];
      const int p = b / a.gc, qb = b - (b / a.gc) * a.gc;
      acc = __builtin_fmaf(c, a.X[(size_t)(p * a.br + z) * a.cols + (size_t)qb * a.bc + k], acc);
    }
    const float s = bf16_rne(acc);
    const float y = s * qs[r];
    const uint32_t c0 = enc2d(y, 0.0f, a.fmt) & 0xffu;
    const float v0 = fp8_value(c0, a.fmt);
    uint32_t c1 = 0x100u;
    if (v0 != y) c1 = fp8_neighbour(c0, fabsf(y) > fabsf(v0), a.fmt);
    float er = v0 * dsc[r] - s;
    uint32_t word = c0 | (c1 << 8);
    if (c1 != 0x100u) {
      const float ea = fp8_value(c1, a.fmt) * dsc[r] - s;
      if (fabsf(ea) < fabsf(er)) {
        er = ea;
        word |= 1u << 17;
      }
    }
    ev[r * kJointLanes + lane] = er;
    pk[r * kJointLanes + lane] = word;
  }
  for (int r = 0; r < R; ++r) {
    float acc = 0.0f;
    for (int i = hp[r]; i < hp[r + 1]; ++i)
      acc = __builtin_fmaf(hv[i], ev[hc[i] * kJointLanes + lane], acc);
    gv[r * kJointLanes + lane] = acc;
  }
  for (int sw = 0; sw < max_sweeps; ++sw) {
    bool changed = false;
    for (int r = 0; r < R; ++r) {
      const uint32_t word = pk[r * kJointLanes + lane];
      bool flip = false;
      float delta = 0.0f;
      if (!(word & (1u << 16))) {
        const bool on_alt = (word >> 17) & 1u;
        const uint32_t ccur = on_alt ? (word >> 8) & 0xffu : word & 0xffu;
        const uint32_t calt = on_alt ? word & 0xffu : (word >> 8) & 0xffu;
        const float vcur = fp8_value(ccur, a.fmt) * dsc[r];
        const float valt = fp8_value(calt, a.fmt) * dsc[r];
        delta = valt - vcur;
        const float two = 2.0f * delta;
        const float lin = two * gv[r * kJointLanes + lane];
        const float sq = delta * delta;
        const float quad = sq * hd[r];
        const float change = lin + quad;
        flip = change < 0.0f;
      }
      if (flip) {
        pk[r * kJointLanes + lane] = word ^ (1u << 17);
        for (int i = hp[r]; i < hp[r + 1]; ++i) {
          const int t = hc[i];
          gv[t * kJointLanes + lane] = __builtin_fmaf(hv[i], delta, gv[t * kJointLanes + lane]);
        }
        changed = true;
      }
    }
    if (!__builtin_amdgcn_ballot_w64(changed)) break;
  }
  for (int r = 0; r < R; ++r) {
    const uint32_t word = pk[r * kJointLanes + lane];
    const uint32_t c = ((word >> 17) & 1u) ? (word >> 8) & 0xffu : word & 0xffu;
    a.codes[((size_t)((size_t)g * a.R + r) * a.br + z) * a.bc + k] = (uint8_t)c;
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

// One wave per row: lane l sums entries l, l+64, ... in order, then a fixed
// butterfly over the lanes; the result does not depend on scheduling.
__device__ __forceinline__ double wave_sum_f64(double s) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s = s + __shfl_xor(s, off, 64);
  return s;
}

__global__ __launch_bounds__(64) void reduce_rows_kernel(const double* partial, int nblk, int G,
                                                          double* out) {
  const int g = blockIdx.x, lane = threadIdx.x;
  if (g >= G) return;
  double s = 0.0;
  for (int b = lane; b < nblk; b += 64) s = s + partial[(size_t)g * nblk + b];
  s = wave_sum_f64(s);
  if (lane == 0) out[g] = s;
}

// ----------------------------------------------------- float64 reference
// On the float64 matrix cores: 128 x 128 output tile per workgroup of 8
// waves (64 x 32 each: 4 x 2 blocks of v_mfma_f64_16x16x4_f64; two waves
// per SIMD hide each other's LDS reads and conversions), K step 64;
// operands staged in LDS as fp32 (67 KB) and widened to float64 when read
// (products of two fp32 values are exact in float64; the sums are float64,
// in ascending K steps of 4 for every output, whatever the tiling).
// Lane l of a 16 x 16 x 4 step holds A[l % 16][l / 16] and B[l / 16][l % 16];
// its four results v = 0..3 are rows l / 16 + 4 v, column l % 16 of the block
// (checked on the device with small integer operands).
typedef double v4d __attribute__((ext_vector_type(4)));
constexpr int kRefThreads = 512;
__global__ __launch_bounds__(kRefThreads) void ref_f64_mfma_kernel(const float* __restrict__ A,
                                                                   const float* __restrict__ B,
                                                                   double* __restrict__ C, int M,
                                                                   int N, int K) {
  constexpr int KS = 64;  // K step
  constexpr int NL = 128 * KS / kRefThreads;  // loads per thread and operand (16)
  __shared__ float As[128][KS + 1];
  __shared__ float Bs[KS][128 + 4];
  const int m0 = blockIdx.y * 128, n0 = blockIdx.x * 128;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;  // 64-row half, 32-column quarter
  const int l16 = lane & 15, lq = lane >> 4;
  v4d acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (v4d){0.0, 0.0, 0.0, 0.0};
  // the next step's operands are loaded into registers while this step's
  // products run
  float ra[NL], rb[NL];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int idx = tid + kRefThreads * i;  // 0 .. 8191
      const int r = idx >> 6, kk = idx & 63;
      const int gr = m0 + r, gk = k0 + kk;
      ra[i] = (gr < M && gk < K) ? A[(size_t)gr * K + gk] : 0.0f;
      const int kb = idx >> 7, c = idx & 127;
      const int gkb = k0 + kb, gc = n0 + c;
      rb[i] = (gkb < K && gc < N) ? B[(size_t)gkb * N + gc] : 0.0f;
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int idx = tid + kRefThreads * i;
      As[idx >> 6][idx & 63] = ra[i];
      Bs[idx >> 7][idx & 127] = rb[i];
    }
  };
  load(0);
  for (int k0 = 0; k0 < K; k0 += KS) {
    store();
    __syncthreads();
    if (k0 + KS < K) load(k0 + KS);
#pragma unroll
    for (int kk = 0; kk < KS; kk += 4) {
      double a[4], b[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = (double)As[wm * 64 + i * 16 + l16][kk + lq];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = (double)Bs[kk + lq][wn * 32 + j * 16 + l16];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + wm * 64 + i * 16 + lq + 4 * v;
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 32 + j * 16 + l16;
        if (col < N) C[(size_t)row * N + col] = acc[i][j][v];
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

__global__ __launch_bounds__(64) void error_finalize_kernel(const double* partial, int nblk,
                                                             double* out3) {
  if (blockIdx.x != 0) return;
  const int lane = threadIdx.x;
  double e = 0.0, r = 0.0, m = 0.0;
  for (int b = lane; b < nblk; b += 64) {
    e = e + partial[3 * b];
    r = r + partial[3 * b + 1];
    m = fmax(m, partial[3 * b + 2]);
  }
  e = wave_sum_f64(e);
  r = wave_sum_f64(r);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
  if (lane == 0) {
    out3[0] = e;
    out3[1] = r;
    out3[2] = m;
  }
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

int launch_form_merged(const FormArgs& aq, const FormArgs& am, int pattern, int side,
                       hipStream_t st) {
  int id = 0;
#define FM_MERGED_CASE(P)                                            \
  if (pattern == id) return form_merged_family_##P(aq, am, side, st); \
  ++id;
  FM_PATTERN_FAMILIES(FM_MERGED_CASE)
#undef FM_MERGED_CASE
  return 1;
}

int launch_scales(const uint32_t* amax, float* q, float* d, int n, int fmt, uint32_t* flag,
                  hipStream_t st) {
  const float fmax = fmt == FM_E4M3 ? 448.0f : 57344.0f;
  scales_kernel<<<(n + kThreads - 1) / kThreads, kThreads, 0, st>>>(amax, q, d, n, fmax, flag);
  return launched("scales_kernel");
}

int recon_blocks(const ReconArgs& a) {
  // one position group per thread (the static kernels assume it); positions
  // counted at the width both kernel kinds use: 4 for grids of at most 16
  // blocks when the shape allows it, else 1
  const int vw = recon_width(a);
  const long long P = (long long)a.Mb * (a.Nb / vw);
  return (int)std::max<long long>(1, (P + kThreads - 1) / kThreads);
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
  if (a.tiled) return fail(FM_E_UNSUPPORTED, "tiled products need a family kernel");
  return launch_recon_generic(a, st);
}

int launch_reduce_rows(const double* partial, int nblk, int G, double* out, hipStream_t st) {
  if (G <= 0) return FM_OK;
  reduce_rows_kernel<<<G, 64, 0, st>>>(partial, nblk, G, out);
  return launched("reduce_rows_kernel");
}

int launch_reference_f64(const float* A, const float* B, double* C, int M, int N, int K,
                         hipStream_t st) {
  dim3 grid((N + 127) / 128, (M + 127) / 128);
  ref_f64_mfma_kernel<<<grid, kRefThreads, 0, st>>>(A, B, C, M, N, K);
  return launched("ref_f64_mfma_kernel");
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

int launch_bf16_round(const float* x, float* out, size_t n, int impl, hipStream_t st) {
  if (n == 0) return FM_OK;
  bf16_round_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, st>>>(x, out, n, impl);
  return launched("bf16_round_kernel");
}

int launch_row_repair(const float* A, int M, int K, float* As, float* up, hipStream_t st) {
  const long long blocks = ((long long)M + kThreads / 64 - 1) / (kThreads / 64);
  if (M < 1 || K < 1 || blocks > 0x7fffffffLL) return fail(FM_E_SHAPE, "row repair shape");
  row_repair_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(A, M, K, As, up);
  return launched("row_repair_kernel");
}

int launch_joint_round(const FormArgs& a, const float* qS, const float* dS, const float* hv,
                       const uint16_t* hc, const int32_t* hp, int pattern, hipStream_t st) {
  if (a.bc % kGroup || a.br % kGroup) return fail(FM_E_SHAPE, "joint rounding needs 128 x 128 blocks");
  int id = 0;
#define FM_JOINT_CASE(P)                                            \
  if (pattern == id) {                                              \
    const int rc = joint_family_##P(a, qS, dS, hv, hc, hp, st);     \
    if (rc != 1) return rc;                                         \
  }                                                                 \
  ++id;
  FM_PATTERN_FAMILIES(FM_JOINT_CASE)
#undef FM_JOINT_CASE
  if (a.R > kJointMaxR)
    return fail(FM_E_UNSUPPORTED, "joint rounding is built for at most 64 products");
  if (a.G > 65535) return fail(FM_E_SHAPE, "too many gauges");
  const long long blocks = (long long)a.br * (a.bc / kJointLanes);
  if (blocks > 0x7fffffffLL) return fail(FM_E_SHAPE, "too many positions");
  // H values (room for R x R), q, d, diagonal, three R x 64 lane arrays,
  // row pointers, then the columns (R x R halves)
  const size_t shm = ((size_t)a.R * a.R + 3 * a.R + 3 * (size_t)a.R * kJointLanes + a.R + 1) * 4 +
                     (size_t)a.R * a.R * 2;
  if (int rc = hip_check(hipFuncSetAttribute(reinterpret_cast<const void*>(&joint_round_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm),
                         "hipFuncSetAttribute"))
    return rc;
  joint_round_kernel<<<dim3((unsigned)blocks, a.G), kJointLanes, shm, st>>>(
      a, qS, dS, JointH{hv, hc, hp}, kRepairSweeps);
  return launched("joint_round_kernel");
}

}  // namespace fm
