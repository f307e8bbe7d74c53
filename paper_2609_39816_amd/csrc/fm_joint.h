// Device side of the joint rounding of B's block sums (the repair rules of
// the group schedule): helpers shared with the generic kernel, the kernel
// specialized per scheme family (state in registers, H at compile-time
// offsets) and its launcher.  Included by fm_kernels.hip (generic kernel)
// and by each family's translation unit (fm_fam_*.hip).
#pragma once

#include "fm_device.h"

namespace fm {
namespace dev {

// ------------------------------------------------------------- repairs
inline constexpr int kGroup = 128;         // edge of the group schedule's scale groups
inline constexpr int kRepairSweeps = 12;   // the repair rules' bound on the sweeps
inline constexpr int kJointLanes = 64;
inline constexpr int kJointMaxR = 64;

__device__ __forceinline__ float bf16_rne(float x) {
  // nearest bf16, ties to even (finite inputs; non-finite values are flagged)
  const uint32_t u = __float_as_uint(x);
  return __uint_as_float((u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u);
}

__device__ __forceinline__ float fp8_value(uint32_t code, int fmt) {
  return fmt == FM_E4M3 ? __builtin_amdgcn_cvt_f32_fp8((int)code, 0)
                        : __builtin_amdgcn_cvt_f32_bf8((int)code, 0);
}

__device__ __forceinline__ uint32_t fp8_neighbour(uint32_t c, bool up, int fmt) {
  // one step larger (up) or smaller in magnitude; 0x100 when there is none
  const uint32_t mag = c & 0x7fu, sign = c & 0x80u;
  const uint32_t maxmag = fmt == FM_E4M3 ? 0x7eu : 0x7bu;
  if (up) return mag >= maxmag ? 0x100u : (sign | (mag + 1u));
  return mag == 0u ? 0x100u : (sign | (mag - 1u));
}

// H of a gauge in compressed rows over its support, the pairs of products
// that share a block of A and a block of C (symmetric, so a row is also a
// column): hv values and hc columns of row r at [hp[r], hp[r + 1]),
// ascending columns.  Outside the support H is an exact zero and is
// skipped; an entry inside it may still be zero and adds an exact zero to a
// fused multiply-add; either way every sum equals the dense one (up to the
// sign of a zero sum, which no decision can see).
struct JointH {
  const float* hv;       // G x R*R (per gauge, the first hp[R] used)
  const uint16_t* hc;    // G x R*R
  const int32_t* hp;     // G x (R + 1)
};

// Position of H_rr within row r of a family's H pattern.
template <class HP>
constexpr int joint_diag(int r) {
  for (int e = HP::rowptr[r]; e < HP::rowptr[r + 1]; ++e)
    if (HP::idx[e] == r) return e;
  return -1;
}

// Joint rounding specialized for one family F: the block sums follow F::B's
// compile-time lists and H's support is F::H (pairs of products that share
// a block of A and a block of C; the host uploads every gauge's H in
// compressed rows over exactly its support, and dispatches here only when
// that support is F::H).  The arithmetic is the generic kernel's, operation
// for operation: the same fmaf chains for the block sums and for H e, the
// same start, the same fp32 decision terms, the same updates.  What changes
// is where the state lives: a lane owns one position and keeps per product
// (H e)_r (each error is folded in as soon as it is known; H is symmetric,
// so column r is row r) and the signed step delta to the other bracketing
// value (0 when there is none, which can never pass the decision; a flip
// negates it exactly) in registers, with one flip-parity bit per product;
// its start codes and their XOR with the other bracketing codes wait in LDS
// until the end.  H's compressed rows sit in LDS as uploaded and are read at
// compile-time offsets (wave-uniform, broadcast).  A wave covers 64
// consecutive k of one row z, inside one 128 x 128 block, so its scales are
// wave-uniform scalar loads.
template <class F, int FMT>
__global__ __launch_bounds__(kThreads, 4) void joint_static_kernel(FormArgs a,
                                                                const float* __restrict__ qS,
                                                                const float* __restrict__ dS,
                                                                JointH hg) {
  using B = typename F::B;
  using HP = typename F::H;
  constexpr int R = HP::R;
  constexpr int NW = (R + 1) / 2;
  __shared__ float hs[HP::NNZ];
  // per thread, two products per word: the start code in bits 0-7 (16-23)
  // and its XOR with the other bracketing code in bits 8-15 (24-31);
  // [word][thread], so every access is one conflict-free row
  __shared__ uint32_t cpair[NW][kThreads];
  const int g = blockIdx.y;
  for (int i = threadIdx.x; i < HP::NNZ; i += kThreads) hs[i] = hg.hv[(size_t)g * R * R + i];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int per_row = a.bc / kJointLanes;
  const int wi = (int)blockIdx.x * (kThreads / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wi >= a.br * per_row) return;
  const int z = wi / per_row;
  const int k0 = (wi - z * per_row) * kJointLanes, k = k0 + lane;
  const int nkg = a.bc / kGroup, nzb = a.br / kGroup;
  const size_t sbase = ((size_t)g * R * nkg + k0 / kGroup) * nzb + z / kGroup;
  const size_t sstride = (size_t)nkg * nzb;
  const auto coef = ro(a.coef) + ro(a.off)[(size_t)g * (R + 1)];

  float xv[B::NB];
#pragma unroll
  for (int b = 0; b < B::NB; ++b) {
    const int bi = b / a.gc, bj = b - (b / a.gc) * a.gc;
    xv[b] = a.X[(size_t)(bi * a.br + z) * a.cols + (size_t)bj * a.bc + k];
  }
  float gv[R], dl[R];
  uint32_t flipped[2] = {0u, 0u};  // bit r: product r is on its other code
  uint32_t pair = 0u;
#pragma unroll
  for (int r = 0; r < R; ++r) gv[r] = 0.0f;
  sfor<0, R>([&](auto rc) {
    constexpr int r = decltype(rc)::value;
    float acc = 0.0f;
    asm volatile("" : "+v"(acc));  // product r starts after product r - 1
    sfor<B::rowptr[r], B::rowptr[r + 1]>([&](auto ec) {
      constexpr int e = decltype(ec)::value;
      acc = __builtin_fmaf(coef[e], xv[B::idx[e]], acc);
    });
    const float s = bf16_rne(acc);
    const float q = ro(qS)[sbase + r * sstride], d = ro(dS)[sbase + r * sstride];
    const float y = s * q;
    const uint32_t c0 = enc2d(y, 0.0f, FMT) & 0xffu;
    const float v0 = fp8_value(c0, FMT);
    // the bracketing neighbour (fp8_neighbour's rule) and the value-nearer
    // start, as selects: the start stays one straight block of code, so
    // nothing of it is sunk towards the sweeps with its operands held live
    const uint32_t mag = c0 & 0x7fu, sgn = c0 & 0x80u;
    const bool up = fabsf(y) > fabsf(v0);
    const bool has = v0 != y && (up ? mag < (FMT == FM_E4M3 ? 0x7eu : 0x7bu) : mag != 0u);
    const uint32_t c1 = has ? (sgn | (up ? mag + 1u : mag - 1u)) : c0;
    const float v0d = v0 * d, v1d = fp8_value(c1, FMT) * d;
    const float e0 = v0d - s, e1 = v1d - s;
    const bool take1 = has && fabsf(e1) < fabsf(e0);
    const float er = take1 ? e1 : e0;
    const uint32_t cur = take1 ? c1 : c0, alt = take1 ? c0 : c1;
    dl[r] = has ? (take1 ? v0d - v1d : v1d - v0d) : 0.0f;
    pair |= (cur | ((cur ^ alt) << 8)) << (16 * (r & 1));
    if constexpr ((r & 1) || r == R - 1) {
      cpair[r / 2][threadIdx.x] = pair;
      pair = 0u;
    }
    // H e as the errors arrive: every (H e)_t gets its terms in ascending
    // product order from +0, the order of the row sums themselves.  The
    // offset depends on the error, so column r of H is read only now (not
    // all of H up front, into registers)
    int ho = 0;
    asm volatile("" : "+v"(ho) : "v"(er));
    constexpr int h0 = HP::rowptr[r], ne = HP::rowptr[r + 1] - h0;
    float hcol[ne];
    sfor<0, ne>([&](auto ec) {
      constexpr int e = decltype(ec)::value;
      hcol[e] = hs[ho + h0 + e];  // H_tr = H_rt
    });
    sfor<0, ne>([&](auto ec) {
      constexpr int e = decltype(ec)::value, t = HP::idx[h0 + e];
      gv[t] = __builtin_fmaf(hcol[e], er, gv[t]);
      asm volatile("" : "+v"(gv[t]));  // formed here, not sunk to its use
    });
  });
  // (a compile-time bound: the first sweep always runs, so nothing of the
  // start is sunk into a conditional block)
  for (int sw = 0; sw < kRepairSweeps; ++sw) {
    bool changed = false;
    // H stays in LDS: an offset opaque to the compiler keeps its reads
    // inside the loop instead of hoisting all of H into registers
    int ho = 0;
    asm volatile("" : "+v"(ho));
    sfor<0, R>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      const float delta = dl[r];
      const float two = 2.0f * delta;
      const float lin = two * gv[r];
      const float sq = delta * delta;
      constexpr int dg = joint_diag<HP>(r);
      static_assert(dg >= 0, "H's support holds its diagonal");
      const float quad = sq * hs[ho + dg];
      // fl(lin + quad) < 0 exactly when lin < -quad (a nonzero sum of two
      // floats never rounds to zero)
      if (lin < -quad) {
        sfor<HP::rowptr[r], HP::rowptr[r + 1]>([&](auto ec) {
          constexpr int e = decltype(ec)::value, t = HP::idx[e];
          gv[t] = __builtin_fmaf(hs[ho + e], delta, gv[t]);
        });
        dl[r] = -delta;
        flipped[r / 32] ^= 1u << (r % 32);
        changed = true;
      }
    });
    if (!__builtin_amdgcn_ballot_w64(changed)) break;
  }
  // the gauge's R code tensors through one buffer descriptor: product
  // offset scalar, position offset per lane (the launcher checks that the
  // R tensors fit 31-bit offsets)
  const uint32_t plane = (uint32_t)a.br * (uint32_t)a.bc;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      a.codes + (size_t)g * R * plane, (short)0, (int)(R * plane), 0x00020000);
  const uint32_t voff = (uint32_t)z * (uint32_t)a.bc + (uint32_t)k;
  sfor<0, NW>([&](auto wc) {
    constexpr int w = decltype(wc)::value;
    const uint32_t wd = cpair[w][threadIdx.x];
    sfor<2 * w, (2 * w + 2 < R ? 2 * w + 2 : R)>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      const uint32_t h = wd >> (16 * (r & 1));
      const uint32_t c = (h ^ (((flipped[r / 32] >> (r % 32)) & 1u) ? h >> 8 : 0u)) & 0xffu;
      __builtin_amdgcn_raw_buffer_store_b8((uint8_t)c, rsrc, (int)voff, (int)(r * plane), 0);
    });
  });
}

// Launches the family's joint rounding; 1 when the arguments do not fit it
// (more than 64 products, another structure or shape).
template <class F>
int launch_joint_static(const FormArgs& a, const float* qS, const float* dS, const JointH& h,
                        hipStream_t st) {
  if constexpr (F::H::JOINT) {
    if (a.R != F::H::R || a.gr * a.gc != F::B::NB || a.bc % kGroup || a.br % kGroup) return 1;
    if (a.G > 65535) return fail(FM_E_SHAPE, "too many gauges");
    const long long waves = (long long)a.br * (a.bc / kJointLanes);
    const long long blocks = (waves + kThreads / 64 - 1) / (kThreads / 64);
    if (blocks > 0x7fffffffLL || (size_t)a.R * a.br * a.bc >= ((size_t)1 << 31)) return 1;
    if (a.fmt == FM_E4M3)
      joint_static_kernel<F, FM_E4M3><<<dim3((unsigned)blocks, a.G), kThreads, 0, st>>>(
          a, qS, dS, h);
    else
      joint_static_kernel<F, FM_E5M2><<<dim3((unsigned)blocks, a.G), kThreads, 0, st>>>(
          a, qS, dS, h);
    return launched("joint_static_kernel");
  } else {
    return 1;
  }
}

}  // namespace dev

// Joint rounding of one specialized family (defined in fm_fam_<P>.hip);
// 1 when the arguments do not fit the family's kernel (the caller then uses
// the generic kernel), else FM_OK or an error code.
#define FM_DECLARE_JOINT(P)                                                  \
  int joint_family_##P(const FormArgs& a, const float* qS, const float* dS,   \
                       const float* hv, const uint16_t* hc, const int32_t* hp, \
                       hipStream_t st);
FM_PATTERN_FAMILIES(FM_DECLARE_JOINT)
#undef FM_DECLARE_JOINT

#define FM_DEFINE_JOINT(P)                                                           \
  int joint_family_##P(const FormArgs& a, const float* qS, const float* dS,          \
                       const float* hv, const uint16_t* hc, const int32_t* hp,        \
                       hipStream_t st) {                                             \
    return dev::launch_joint_static<pat::P>(a, qS, dS, dev::JointH{hv, hc, hp}, st); \
  }

}  // namespace fm
