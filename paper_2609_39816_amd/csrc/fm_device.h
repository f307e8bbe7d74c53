// Device-side building blocks of libfm shared by the kernel translation
// units: wave reductions, FP8 encoders, compile-time loops, and the
// operand-formation and reconstruction kernels (specialized for a nonzero
// structure, or generic) with their launch helpers.  Each specialized
// family is instantiated in its own translation unit (fm_fam_*.hip) so the
// large unrolled kernels compile in parallel.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <utility>

#include "fm_internal.h"
#include "fm_patterns.inc"

#ifndef FM_FP8_HW
#define FM_FP8_HW 1  // 1: v_cvt_pk_{fp8,bf8}_f32 for FP8 rounding; 0: integer encoder
#endif

namespace fm {
namespace dev {

inline constexpr int kThreads = 256;

// Read-only tables (coefficient lists, per-product scales) are read through
// the constant address space: the kernels never write them, and this lets
// wave-uniform reads go through the scalar cache into SGPRs even in kernels
// that store to other global memory.
template <class T>
__device__ __forceinline__ const __attribute__((address_space(4))) T* ro(const T* p) {
  return (const __attribute__((address_space(4))) T*)p;
}

// ------------------------------------------------------------ wave helpers
// Maximum over the 64 lanes of a wave of non-negative values; every lane
// returns the result.  DPP row shifts build each row's maximum in its lane
// 15, two row broadcasts carry it to lane 63.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// ------------------------------------------------------------ FP8 encoding
// Integer encoders (round to nearest even, saturating to the largest finite
// value).  Normal range: round the fp32 significand at the FP8 mantissa
// width with the usual add-bias-and-truncate; the exponent follows through
// any carry.  Below the smallest normal the FP8 values are multiples of the
// subnormal quantum, so scaling by its inverse (a power of two, exact) and
// rounding to the nearest integer (ties to even) gives the code directly.
__device__ __forceinline__ uint32_t enc_e4m3_sw(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t s = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7fffffffu;
  uint32_t code;
  if (a >= 0x3C800000u) {  // |x| >= 2^-6
    const uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
    code = min((r >> 20) - (120u << 3), 0x7Eu);
  } else {
    code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
  }
  return s | code;
}

__device__ __forceinline__ uint32_t enc_e5m2_sw(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t s = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7fffffffu;
  uint32_t code;
  if (a >= 0x38800000u) {  // |x| >= 2^-14
    const uint32_t r = a + 0xFFFFFu + ((a >> 21) & 1u);
    code = min((r >> 21) - (112u << 2), 0x7Bu);
  } else {
    code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 65536.0f);
  }
  return s | code;
}

// Two values -> two code bytes (low half of the result).
template <int IMPL>
__device__ __forceinline__ uint32_t enc2(float x0, float x1, int fmt) {
  if (IMPL == 1) {
    if (fmt == FM_E4M3) return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false) & 0xffffu;
    return (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(x0, x1, 0, false) & 0xffffu;
  }
  if (fmt == FM_E4M3) return enc_e4m3_sw(x0) | (enc_e4m3_sw(x1) << 8);
  return enc_e5m2_sw(x0) | (enc_e5m2_sw(x1) << 8);
}

__device__ __forceinline__ uint32_t enc2d(float x0, float x1, int fmt) {
  return enc2<FM_FP8_HW>(x0, x1, fmt);
}

// ----------------------------------------------------- compile-time loops
// sfor<B, E>(f) calls f(std::integral_constant<int, i>) for i in [B, E), so
// the body sees i as a constant expression.
template <int B, class F, int... I>
__device__ __forceinline__ void sfor_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, B + I>{}), ...);
}
template <int B, int E, class F>
__device__ __forceinline__ void sfor(F&& f) {
  if constexpr (E > B) sfor_impl<B>(f, std::make_integer_sequence<int, E - B>{});
}

// Cache policy of the streams written or read once per launch (the FP8
// codes, the block products on their way to the reconstruction): the
// non-temporal bit of the buffer instructions' cache-policy operand.
constexpr int kStreamOut = 2;
constexpr int kStreamIn = 2;

// ------------------------------------------------------- operand formation
// A thread owns VW consecutive positions (x, y0..y0+VW-1) of the block-sum
// tensors and reads the matching entries of every grid block once per
// position group; for each gauge of its slice and each product r it forms
// the block sum as a chain of fmaf over the product's list (ascending grid
// order) from +0, then either folds |T| into the per-tensor maximum
// (MODE 0) or writes the FP8 codes of T * (FMAX / amax) (MODE 1).

template <int NB, int VW>
__device__ __forceinline__ void form_load(const FormArgs& a, float (&xv)[NB][VW], bool active,
                                          int x, int y0) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (active) {
      const int bi = b / a.gc, bj = b - (b / a.gc) * a.gc;
      const float* src = a.X + (size_t)(bi * a.br + x) * a.cols + (size_t)bj * a.bc + y0;
      if constexpr (VW % 4 == 0) {
#pragma unroll
        for (int v = 0; v < VW; v += 4) {
          const float4 t = *reinterpret_cast<const float4*>(src + v);
          xv[b][v] = t.x;
          xv[b][v + 1] = t.y;
          xv[b][v + 2] = t.z;
          xv[b][v + 3] = t.w;
        }
      } else {
#pragma unroll
        for (int v = 0; v < VW; ++v) xv[b][v] = src[v];
      }
    } else {
#pragma unroll
      for (int v = 0; v < VW; ++v) xv[b][v] = 0.0f;
    }
  }
}

// Index of the maximum / scale that covers entries (x, y0..) of product r
// of gauge g, for the finer granularities (a.per_row set).
// The index splits into a part shared by a product's whole tensor,
// (g R + r) group_span, and a part of the position alone, group_local:
// the static kernels form the local part once per position group, so the
// per-product address is one scalar product plus that offset.
__device__ __forceinline__ uint32_t group_span(const FormArgs& a) {
  if (a.gran == 1) return (uint32_t)a.br;
  return (uint32_t)(a.bc / 128) * (uint32_t)(a.gran == 2 ? a.br : a.br / 128);
}

__device__ __forceinline__ uint32_t group_local(const FormArgs& a, int x, int y0) {
  if (a.gran == 1) return (uint32_t)x;
  if (a.gran == 2) return (uint32_t)(y0 >> 7) * (uint32_t)a.br + (uint32_t)x;
  return (uint32_t)(y0 >> 7) * (uint32_t)(a.br / 128) + (uint32_t)(x >> 7);
}

__device__ __forceinline__ size_t group_index(const FormArgs& a, int g, int r, int x, int y0) {
  return ((size_t)g * a.R + r) * group_span(a) + group_local(a, x, y0);
}

// The B side of the group schedule rounds block sums to bf16 (nearest even)
// before their maxima and codes: two at a time with the gfx950 conversion
// (v_cvt_pk_bf16_f32, checked against the integer rounding on every fp32
// high half with low halves around each tie), back to fp32 exactly.
__device__ __forceinline__ float bf16_round_int(float x) {
  const uint32_t u = __float_as_uint(x);
  return __uint_as_float((u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u);
}

__device__ __forceinline__ void bf16_round_pair(float& x0, float& x1) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  typedef float f2 __attribute__((ext_vector_type(2)));
  const bf2 b = __builtin_convertvector((f2){x0, x1}, bf2);
  x0 = (float)b[0];
  x1 = (float)b[1];
}

template <int VW>
__device__ __forceinline__ void round_bf16(float (&acc)[VW]) {
#pragma unroll
  for (int v = 0; v + 1 < VW; v += 2) bf16_round_pair(acc[v], acc[v + 1]);
  if constexpr (VW % 2) acc[VW - 1] = bf16_round_int(acc[VW - 1]);
}

template <int VW, int MODE>
__device__ __forceinline__ void form_finish(const FormArgs& a, const float (&acc0)[VW], int g,
                                            int g0, int r, bool active, int x, int y0,
                                            uint32_t* smax, int lane) {
  float acc[VW];
#pragma unroll
  for (int v = 0; v < VW; ++v) acc[v] = acc0[v];
  if (a.per_row && a.gran == 3) round_bf16<VW>(acc);
  if constexpr (MODE == 0) {
    uint32_t mx = 0u;
#pragma unroll
    for (int v = 0; v < VW; ++v) mx = max(mx, __float_as_uint(acc[v]) & 0x7fffffffu);
    if (!active) mx = 0u;
    if (a.per_row) {  // one maximum per group: straight to global memory
      if (mx) atomicMax(&a.amax[group_index(a, g, r, x, y0)], mx);
      return;
    }
    mx = wave_max_u32(mx);
    if (lane == 0 && mx) atomicMax(&smax[(g - g0) * a.R + r], mx);
  } else {
    if (!active) return;
    const float q = a.per_row ? a.q[group_index(a, g, r, x, y0)] : a.q[(size_t)g * a.R + r];
    uint8_t* dst =
        a.codes + ((size_t)g * a.R + r) * ((size_t)a.br * a.bc) + (size_t)x * a.bc + y0;
    if constexpr (VW >= 4) {
      uint32_t w[VW / 4];
#pragma unroll
      for (int t = 0; t < VW / 4; ++t)
        w[t] = enc2d(acc[4 * t] * q, acc[4 * t + 1] * q, a.fmt) |
               (enc2d(acc[4 * t + 2] * q, acc[4 * t + 3] * q, a.fmt) << 16);
      if constexpr (VW == 4) {
        *reinterpret_cast<uint32_t*>(dst) = w[0];
      } else if constexpr (VW == 8) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
      } else {
#pragma unroll
        for (int t = 0; t < VW / 4; t += 4)
          *reinterpret_cast<uint4*>(dst + 4 * t) = make_uint4(w[t], w[t + 1], w[t + 2], w[t + 3]);
      }
    } else {
#pragma unroll
      for (int v = 0; v < VW; ++v) dst[v] = (uint8_t)(enc2d(acc[v] * q, 0.0f, a.fmt) & 0xffu);
    }
  }
}

template <int MODE>
__device__ __forceinline__ void form_flush(const FormArgs& a, const uint32_t* smax, int g0,
                                           int g1) {
  if constexpr (MODE == 0) {
    if (a.per_row) return;
    __syncthreads();
    const int n = (g1 - g0) * a.R;
    for (int i = threadIdx.x; i < n; i += kThreads)
      if (smax[i]) atomicMax(&a.amax[(size_t)g0 * a.R + i], smax[i]);
  }
}

// Specialized for one nonzero structure P (fm_patterns.inc): block indices
// are compile-time constants, so the operand blocks stay in registers.
// Products are handled in groups of 8.  Mode 0 folds each product's values
// into a per-lane maximum, reduces the group's 8 maxima within 16-lane rows
// with interleaved DPP steps (no hazard stalls between dependent steps), and
// the last lane of each row keeps the result in its own LDS slot (plain
// stores, no atomics); the workgroup combines the 16 slots of each product
// once at the end.  Mode 1
// writes the codes through a buffer descriptor over the gauge's R tensors
// (product offset in the scalar offset, position in the vector offset); an
// inactive lane gets an offset past the end, so its store is dropped by the
// range check instead of branched around.  The launcher checks that the R
// tensors of one gauge fit the 31-bit offsets.
template <int FMT, int VW>
__device__ __forceinline__ void form_encode_store(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                                  uint32_t soff, const float (&acc)[VW], float q) {
  static_assert(VW == 2 || VW % 4 == 0, "code store width");
  uint32_t w[(VW + 3) / 4];
#pragma unroll
  for (int t = 0; t < (VW + 3) / 4; ++t) {
    const float x0 = acc[4 * t] * q, x1 = acc[4 * t + 1] * q;
    // the conversion keeps the other half of its destination; that half is
    // written next (VW >= 4) or never stored (VW == 2), so the first
    // conversion is issued as a plain definition of the register (the
    // intrinsic would have the compiler clear the register first)
    if constexpr (FMT == FM_E4M3) asm("v_cvt_pk_fp8_f32 %0, %1, %2" : "=v"(w[t]) : "v"(x0), "v"(x1));
    else asm("v_cvt_pk_bf8_f32 %0, %1, %2" : "=v"(w[t]) : "v"(x0), "v"(x1));
    if constexpr (VW >= 4) {
      const float x2 = acc[4 * t + 2] * q, x3 = acc[4 * t + 3] * q;
      if constexpr (FMT == FM_E4M3) w[t] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x2, x3, (int)w[t], true);
      else w[t] = (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(x2, x3, (int)w[t], true);
    }
  }
  if constexpr (VW == 2) {
    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)(w[0] & 0xffffu), rsrc, (int)voff, (int)soff, kStreamOut);
  } else if constexpr (VW == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(w[0], rsrc, (int)voff, (int)soff, kStreamOut);
  } else if constexpr (VW == 8) {
    __builtin_amdgcn_raw_buffer_store_b64((__attribute__((ext_vector_type(2))) unsigned){w[0], w[1]},
                                          rsrc, (int)voff, (int)soff, kStreamOut);
  } else {
#pragma unroll
    for (int t = 0; t < VW / 4; t += 4)
      __builtin_amdgcn_raw_buffer_store_b128(
          (__attribute__((ext_vector_type(4))) unsigned){w[t], w[t + 1], w[t + 2], w[t + 3]}, rsrc,
          (int)(voff + 4 * t), (int)soff, kStreamOut);
  }
}

// Gauges g0 <= g < g1 of a at one position group (operand values xv); mode
// 0 keeps its maxima in the LDS slots of gauge g - g0.
template <class P, int VW, int MODE, int FMT, bool ROWS>
__device__ __forceinline__ void form_static_gauges(const FormArgs& a, int g0, int g1,
                                                   const float (&xv)[P::NB][VW], bool active,
                                                   int x, int y0, uint32_t voff, uint32_t* smax) {
  constexpr int GR = 8, NG = (P::R + GR - 1) / GR;
  const int lane = threadIdx.x & 63;
  const uint32_t bsz = (uint32_t)a.br * (uint32_t)a.bc;
  [[maybe_unused]] const int bcv = a.bc / VW;
  {
    // finer granularities: the position's offset among a product's groups
    [[maybe_unused]] const uint32_t gspan = ROWS ? group_span(a) : 0u;
    [[maybe_unused]] const uint32_t gloc = ROWS ? group_local(a, x, y0) : 0u;
    auto gidx = [&](int gg, int rr) { return ((size_t)gg * P::R + rr) * gspan + gloc; };
    for (int g = g0; g < g1; ++g) {
      const auto coef = ro(a.coef) + ro(a.off)[(size_t)g * (P::R + 1)];
      __amdgpu_buffer_rsrc_t rsrc;
      if constexpr (MODE == 1)
        rsrc = __builtin_amdgcn_make_buffer_rsrc(a.codes + (size_t)g * P::R * bsz, (short)0,
                                                 (int)(P::R * bsz), 0x00020000);
      sfor<0, NG>([&](auto gc) {
        constexpr int gi = decltype(gc)::value;
        uint32_t lm[GR];
        // the group's coefficients and per-tensor scales are read through
        // an offset the compiler cannot see through, so their scalar loads
        // stay with the group instead of all going out at the top of the
        // gauge (which needs more scalar registers than there are)
        int so = 0;
        asm volatile("" : "+s"(so));
        // finer scales: the group's scale loads go out before its block
        // sums, so their latency hides under the fused multiply-adds
        [[maybe_unused]] float qv[GR];
        if constexpr (MODE == 1 && ROWS)
          sfor<0, GR>([&](auto jc) {
            constexpr int j = decltype(jc)::value, r = gi * GR + j;
            if constexpr (r < P::R) qv[j] = ro(a.q)[gidx(g, r)];
          });
        sfor<0, GR>([&](auto jc) {
          constexpr int j = decltype(jc)::value, r = gi * GR + j;
          if constexpr (r < P::R) {
            float acc[VW];
#pragma unroll
            for (int v = 0; v < VW; ++v) acc[v] = 0.0f;
            sfor<P::rowptr[r], P::rowptr[r + 1]>([&](auto ec) {
              constexpr int e = decltype(ec)::value;
              constexpr int b = P::idx[e];
              const float c = coef[e + so];
#pragma unroll
              for (int v = 0; v < VW; ++v) acc[v] = __builtin_fmaf(c, xv[b][v], acc[v]);
            });
            if (ROWS && a.gran == 3) round_bf16<VW>(acc);
            if constexpr (MODE == 0) {
              // largest magnitude, NaN-propagating (v_maximum3_f32 on
              // absolute values: half an instruction per value); as bits it
              // orders like the magnitudes, and a NaN or infinity stays at
              // or above the bits of infinity, as the scales check expects
              float mf = 0.0f;
#pragma unroll
              for (int v = 0; v < VW; ++v) mf = __builtin_elementwise_maximum(mf, __builtin_fabsf(acc[v]));
              // inactive lanes hold zero operands: their sums and maxima are +0
              lm[j] = __float_as_uint(mf);
            } else {
              const float q = ROWS ? qv[j] : ro(a.q)[(size_t)g * P::R + r + so];
              form_encode_store<FMT, VW>(rsrc, voff, (uint32_t)r * bsz, acc, q);
            }
          }
        });
        if constexpr (MODE == 0 && ROWS) {
          // one maximum per group, folded into global memory: when a group
          // spans whole 16-lane DPP rows (bcv a multiple of 16, and 16 VW
          // entries within one group of 128 for the finer granularities)
          // they are reduced first and their last lane folds the result;
          // the same with 8-lane halves of a row when 8 VW = 128 (the
          // shifts by 1, 2, 4 leave lanes 7 and 15 with their half's
          // maximum); otherwise every lane folds its own
          constexpr int NJ = (gi * GR + GR <= P::R) ? GR : P::R - gi * GR;
          if (VW == 16 && a.gran != 1 && bcv % 8 == 0) {
            sfor<0, 3>([&](auto sc) {
              constexpr int ctl = 0x111 + (1 << decltype(sc)::value) - 1;  // row_shr:1,2,4
              uint32_t sh[NJ];
#pragma unroll
              for (int j = 0; j < NJ; ++j)
                sh[j] = (uint32_t)__builtin_amdgcn_mov_dpp((int)lm[j], ctl, 0xf, 0xf, true);
#pragma unroll
              for (int j = 0; j < NJ; ++j) lm[j] = max(lm[j], sh[j]);
            });
            if ((lane & 7) == 7 && active) {
#pragma unroll
              for (int j = 0; j < NJ; ++j)
                if (lm[j]) atomicMax(&a.amax[gidx(g, gi * GR + j)], lm[j]);
            }
          } else if (bcv % 16 == 0 && (a.gran == 1 || 16 * VW <= 128)) {
            sfor<0, 4>([&](auto sc) {
              constexpr int ctl = 0x111 + (1 << decltype(sc)::value) - 1;  // row_shr:1,2,4,8
              uint32_t sh[NJ];
#pragma unroll
              for (int j = 0; j < NJ; ++j)
                sh[j] = (uint32_t)__builtin_amdgcn_mov_dpp((int)lm[j], ctl, 0xf, 0xf, true);
#pragma unroll
              for (int j = 0; j < NJ; ++j) lm[j] = max(lm[j], sh[j]);
            });
            if ((lane & 15) == 15 && active) {
#pragma unroll
              for (int j = 0; j < NJ; ++j)
                if (lm[j]) atomicMax(&a.amax[gidx(g, gi * GR + j)], lm[j]);
            }
          } else if (active) {
#pragma unroll
            for (int j = 0; j < NJ; ++j)
              if (lm[j]) atomicMax(&a.amax[gidx(g, gi * GR + j)], lm[j]);
          }
        }
        if constexpr (MODE == 0 && !ROWS) {
          constexpr int NJ = (gi * GR + GR <= P::R) ? GR : P::R - gi * GR;
          // row maxima: after shifts 1, 2, 4, 8 lane 15 of each row holds
          // the maximum of its row (lanes shifted in from outside the row
          // read 0, the bound-control value)
          sfor<0, 4>([&](auto sc) {
            constexpr int ctl = 0x111 + (1 << decltype(sc)::value) - 1;  // row_shr:1,2,4,8
            uint32_t sh[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j)
              sh[j] = (uint32_t)__builtin_amdgcn_mov_dpp((int)lm[j], ctl, 0xf, 0xf, true);
#pragma unroll
            for (int j = 0; j < NJ; ++j) lm[j] = max(lm[j], sh[j]);
          });
          // the last lane of each row keeps its row's maximum in the
          // (wave, row) slot of the product; slots are combined per workgroup
          if ((lane & 15) == 15) {
            uint32_t* slot = smax + ((g - g0) * P::R + gi * GR) * 16 + (threadIdx.x >> 4);
#pragma unroll
            for (int j = 0; j < NJ; ++j) slot[j * 16] = max(slot[j * 16], lm[j]);
          }
        }
      });
    }
  }
}


// Gauges g0 <= g < g1 through the family's prefix-shared chains (P::TRIE,
// one scale per tensor), for sign variants of the family's base scheme: a
// coefficient is the base value of its list entry with the sign of its
// block, from the gauge's 64-bit block-sign mask (bit b set: block b
// negated).  fmaf(s c, x, acc) = fmaf(c, s x, acc) exactly for s = +-1, so
// the operand values of a negated block are negated in place (xv holds them
// under the signs in `applied`; a gauge flips the blocks whose sign changes)
// and the chains take the base values as compile-time constants: no
// coefficient is read or built per term.  Chains that begin with the same
// (block, base coefficient) entries share their partial sums, so the block
// sums are the nodes of a trie walked depth first: node t = fmaf(c_t,
// x[tblk[t]], value of the latest node one level up, or +0 at the root).  The value of the node where a product's chain ends is that
// product's block sum, with the fused multiply-adds of its chain in its
// order: the bits of the plain chain.  Mode 0 folds each lane's maximum
// into the product's slot lane % 16 (of the 16 per product that the
// kernels combine at the end) with an LDS atomic maximum; mode 1 encodes
// and stores each product's codes as it completes.
template <class P, int VW, int MODE, int FMT>
__device__ __forceinline__ void form_trie_gauges(const FormArgs& a, int g0, int g1,
                                                 float (&xv)[P::NB][VW], uint64_t& applied,
                                                 [[maybe_unused]] bool active, uint32_t voff,
                                                 uint32_t* smax) {
  const int lane = threadIdx.x & 63;
  const uint32_t bsz = (uint32_t)a.br * (uint32_t)a.bc;
  for (int g = g0; g < g1; ++g) {
    const uint64_t neg = ro(a.sgn)[g];
    const uint64_t flip = neg ^ applied;
    applied = neg;
    sfor<0, P::NB>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      // the sign bit of block b's change, on the scalar unit
      const uint32_t m = (uint32_t)((flip >> b) & 1u) << 31;
#pragma unroll
      for (int v = 0; v < VW; ++v) xv[b][v] = __uint_as_float(__float_as_uint(xv[b][v]) ^ m);
    });
    __amdgpu_buffer_rsrc_t rsrc;
    if constexpr (MODE == 1)
      rsrc = __builtin_amdgcn_make_buffer_rsrc(a.codes + (size_t)g * P::R * bsz, (short)0,
                                               (int)(P::R * bsz), 0x00020000);
    float nv[P::MAXD][VW];
    // Mode 1 scales, one group of 16 nodes ahead: the scales of the
    // products that complete in group G + 1 are loaded at the start of group
    // G (through an offset the compiler cannot see through, renewed every
    // group, so the loads neither move to the top of the gauge, which needs
    // more scalar registers than there are, nor down to their use)
    constexpr int QG = 16, NGR = (P::NN + QG - 1) / QG;
    [[maybe_unused]] float qb[2][QG];
    int so = 0;
    auto load_scales = [&](auto gc) {
      constexpr int G = decltype(gc)::value;
      if constexpr (MODE == 1 && G < NGR) {
        constexpr int k0 = P::tendptr[QG * G];
        constexpr int k1 = P::tendptr[QG * (G + 1) < P::NN ? QG * (G + 1) : P::NN];
        static_assert(k1 - k0 <= QG, "products completing in one group of nodes");
        sfor<k0, k1>([&](auto kc) {
          constexpr int kk = decltype(kc)::value;
          qb[G & 1][kk - k0] = ro(a.q)[(size_t)g * P::R + P::tendprod[kk] + so];
        });
      }
    };
    load_scales(std::integral_constant<int, 0>{});
    sfor<0, P::NN>([&](auto tc) {
      constexpr int t = decltype(tc)::value;
      if constexpr (t % QG == 0) {
        so = 0;
        asm volatile("" : "+s"(so));
        load_scales(std::integral_constant<int, t / QG + 1>{});
      }
      constexpr int d = P::tdepth[t], b = P::tblk[t];
      constexpr float c = __builtin_bit_cast(float, P::tval[t]);
#pragma unroll
      for (int v = 0; v < VW; ++v) {
        if constexpr (d == 0) nv[0][v] = __builtin_fmaf(c, xv[b][v], 0.0f);
        else nv[d][v] = __builtin_fmaf(c, xv[b][v], nv[d - 1][v]);
      }
      sfor<P::tendptr[t], P::tendptr[t + 1]>([&](auto kc) {
        constexpr int kk = decltype(kc)::value, r = P::tendprod[kk];
        if constexpr (MODE == 0) {
          // the lane's maximum folded into the product's 16 LDS slots (slot
          // = lane % 16) by an LDS atomic maximum: no cross-lane steps on
          // the vector unit; +0 on inactive lanes (zero operands)
          float mf = 0.0f;
#pragma unroll
          for (int v = 0; v < VW; ++v) mf = __builtin_elementwise_maximum(mf, __builtin_fabsf(nv[d][v]));
          atomicMax(smax + ((size_t)(g - g0) * P::R + r) * 16 + (lane & 15), __float_as_uint(mf));
        } else {
          constexpr int G = t / QG, k0 = P::tendptr[QG * G];
          form_encode_store<FMT, VW>(rsrc, voff, (uint32_t)r * bsz, nv[d], qb[G & 1][kk - k0]);
        }
      });
    });
  }
}

template <class P, int VW, int MODE, int FMT, bool ROWS>
__device__ __forceinline__ void form_static_body(const FormArgs& a, int gpb, uint32_t* smax) {
  const int bcv = a.bc / VW;
  const int Ptot = a.br * bcv;
  const int g0 = blockIdx.y * gpb;
  const int g1 = min(a.G, g0 + gpb);
  for (int base = blockIdx.x * kThreads; base < Ptot; base += gridDim.x * kThreads) {
    const int p = base + threadIdx.x;
    const bool active = p < Ptot;
    const int x = active ? p / bcv : 0;
    const int y0 = active ? (p - x * bcv) * VW : 0;
    const uint32_t voff = active ? (uint32_t)(x * a.bc + y0) : 0x80000000u;
    float xv[P::NB][VW];
    form_load<P::NB, VW>(a, xv, active, x, y0);
    [[maybe_unused]] uint64_t applied = 0;
    if constexpr (P::TRIE && !ROWS)
      form_trie_gauges<P, VW, MODE, FMT>(a, g0, g1, xv, applied, active, voff, smax);
    else
      form_static_gauges<P, VW, MODE, FMT, ROWS>(a, g0, g1, xv, active, x, y0, voff, smax);
  }
}

template <class P, int VW, int MODE, bool ROWS>
__global__ __launch_bounds__(kThreads) void form_static_kernel(FormArgs a, int gpb) {
  extern __shared__ uint32_t smax[];  // mode 0: [gauge][product][wave * 4 + row]
  const int g0 = blockIdx.y * gpb;
  const int g1 = min(a.G, g0 + gpb);
  if constexpr (MODE == 0 && ROWS) {
    form_static_body<P, VW, 0, FM_E4M3, true>(a, gpb, smax);
  } else if constexpr (MODE == 0) {
    for (int i = threadIdx.x; i < gpb * P::R * 16; i += kThreads) smax[i] = 0u;
    __syncthreads();
    form_static_body<P, VW, 0, FM_E4M3, false>(a, gpb, smax);
    __syncthreads();
    const int n = (g1 - g0) * P::R;
    for (int k = threadIdx.x; k < n; k += kThreads) {
      uint32_t m = 0u;
#pragma unroll
      for (int t = 0; t < 16; ++t) m = max(m, smax[k * 16 + t]);
      if (m) atomicMax(&a.amax[(size_t)g0 * P::R + k], m);
    }
  } else {
    if (a.fmt == FM_E4M3) form_static_body<P, VW, 1, FM_E4M3, ROWS>(a, gpb, smax);
    else form_static_body<P, VW, 1, FM_E5M2, ROWS>(a, gpb, smax);
  }
}

// One operand side of two consecutive chunks of an orbit in one pass: the
// FP8 codes of chunk c (aq, mode 1, scales known) and the per-tensor maxima
// of chunk c + 1 (am, mode 0), from one load of the operand blocks per
// position group.  The encoding is bound by its code stores and the maxima
// by vector arithmetic, so each fills the other's idle time.  Gauges split
// over grid.y as in the separate kernels: slice y encodes gauges
// [y gpbq, (y + 1) gpbq) of aq and folds the maxima of [y gpbm, ..) of am.
//
// The grid is one-dimensional over gx position blocks x gy slices.  With gx
// a multiple of 8, workgroup w takes position block 8 ((w / 8) / gy) + w % 8
// and slice (w / 8) % gy: the gy slices of a position block run on one XCD
// (workgroups go round-robin over the 8 XCDs) within a few dispatch rounds,
// so the block's operand values are read from memory once and from that
// XCD's L2 by the other slices.
template <class P, int VW, int FMT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 8))) void form_merged_kernel(FormArgs aq, FormArgs am, int gpbq,
                                                               int gpbm, int gx, int gy) {
  extern __shared__ uint32_t smax[];  // am's [gauge][product][wave * 4 + row]
  const int w = blockIdx.x;
  int bx, by;
  if ((gx & 7) == 0) {
    by = (w >> 3) % gy;
    bx = ((w >> 3) / gy) * 8 + (w & 7);
  } else {
    by = w / gx;
    bx = w - by * gx;
  }
  const int g0q = by * gpbq, g1q = min(aq.G, g0q + gpbq);
  const int g0m = by * gpbm, g1m = min(am.G, g0m + gpbm);
  for (int i = threadIdx.x; i < gpbm * P::R * 16; i += kThreads) smax[i] = 0u;
  __syncthreads();
  const int bcv = aq.bc / VW;
  const int Ptot = aq.br * bcv;
  for (int base = bx * kThreads; base < Ptot; base += gx * kThreads) {
    const int p = base + threadIdx.x;
    const bool active = p < Ptot;
    const int x = active ? p / bcv : 0;
    const int y0 = active ? (p - x * bcv) * VW : 0;
    const uint32_t voff = active ? (uint32_t)(x * aq.bc + y0) : 0x80000000u;
    float xv[P::NB][VW];
    form_load<P::NB, VW>(aq, xv, active, x, y0);
    if constexpr (P::TRIE) {
      uint64_t applied = 0;
      form_trie_gauges<P, VW, 1, FMT>(aq, g0q, g1q, xv, applied, active, voff, smax);
      form_trie_gauges<P, VW, 0, FM_E4M3>(am, g0m, g1m, xv, applied, active, voff, smax);
    } else {
      form_static_gauges<P, VW, 1, FMT, false>(aq, g0q, g1q, xv, active, x, y0, voff, smax);
      form_static_gauges<P, VW, 0, FM_E4M3, false>(am, g0m, g1m, xv, active, x, y0, voff, smax);
    }
  }
  __syncthreads();
  const int n = max(0, g1m - g0m) * P::R;
  for (int k = threadIdx.x; k < n; k += kThreads) {
    uint32_t m = 0u;
#pragma unroll
    for (int t = 0; t < 16; ++t) m = max(m, smax[k * 16 + t]);
    if (m) atomicMax(&am.amax[(size_t)g0m * P::R + k], m);
  }
}

// Any nonzero structure: each thread parks its operand values in its own
// slots of LDS ([block][thread][VW]) and gathers them by the run-time block
// index of each list entry.
template <int VW, int MODE>
__global__ __launch_bounds__(kThreads) void form_generic_kernel(FormArgs a, int gpb) {
  extern __shared__ float dyn[];
  const int nb = a.gr * a.gc;
  float* lx = dyn;
  uint32_t* smax = reinterpret_cast<uint32_t*>(dyn + (size_t)nb * kThreads * VW);
  const int R = a.R;
  const int bcv = a.bc / VW;
  const int Ptot = a.br * bcv;
  const int g0 = blockIdx.y * gpb;
  const int g1 = min(a.G, g0 + gpb);
  const int lane = threadIdx.x & 63;
  if constexpr (MODE == 0) {
    for (int i = threadIdx.x; i < gpb * R; i += kThreads) smax[i] = 0u;
    __syncthreads();
  }
  for (int base = blockIdx.x * kThreads; base < Ptot; base += gridDim.x * kThreads) {
    const int p = base + threadIdx.x;
    const bool active = p < Ptot;
    const int x = active ? p / bcv : 0;
    const int y0 = active ? (p - x * bcv) * VW : 0;
    for (int b = 0; b < nb; ++b) {
      float* slot = lx + ((size_t)b * kThreads + threadIdx.x) * VW;
      const int bi = b / a.gc, bj = b - (b / a.gc) * a.gc;
      const float* src = a.X + (size_t)(bi * a.br + x) * a.cols + (size_t)bj * a.bc + y0;
#pragma unroll
      for (int v = 0; v < VW; ++v) slot[v] = active ? src[v] : 0.0f;
    }
    for (int g = g0; g < g1; ++g) {
      const int32_t* off = a.off + (size_t)g * (R + 1);
      for (int r = 0; r < R; ++r) {
        const int e0 = off[r], e1 = off[r + 1];
        float acc[VW];
#pragma unroll
        for (int v = 0; v < VW; ++v) acc[v] = 0.0f;
        for (int e = e0; e < e1; ++e) {
          const float c = a.coef[e];
          const float* slot = lx + ((size_t)a.idx[e] * kThreads + threadIdx.x) * VW;
#pragma unroll
          for (int v = 0; v < VW; ++v) acc[v] = __builtin_fmaf(c, slot[v], acc[v]);
        }
        form_finish<VW, MODE>(a, acc, g, g0, r, active, x, y0, smax, lane);
      }
    }
  }
  form_flush<MODE>(a, smax, g0, g1);
}
// ------------------------------------------------- reconstruction + error
// A thread owns VW consecutive positions (x, z0..) of every output block;
// it reads each product's values there once, adds w * M_r into the output
// blocks the product feeds (ascending r for every block, fmaf from +0), and
// then writes C and/or accumulates (C - Cref)^2 in float64.
template <int VW>
__device__ __forceinline__ void recon_load_bf16(const uint16_t* src, float (&m)[VW]) {
  // bf16 products: each value is its fp32 high half
  if constexpr (VW % 4 == 0) {
#pragma unroll
    for (int v = 0; v < VW; v += 4) {
      const uint2 t = *reinterpret_cast<const uint2*>(src + v);
      m[v] = __uint_as_float(t.x << 16);
      m[v + 1] = __uint_as_float(t.x & 0xffff0000u);
      m[v + 2] = __uint_as_float(t.y << 16);
      m[v + 3] = __uint_as_float(t.y & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int v = 0; v < VW; ++v) m[v] = __uint_as_float((uint32_t)src[v] << 16);
  }
}

template <int VW>
__device__ __forceinline__ void recon_load(const float* src, float (&m)[VW]) {
  if constexpr (VW % 4 == 0) {
#pragma unroll
    for (int v = 0; v < VW; v += 4) {
      const float4 t = *reinterpret_cast<const float4*>(src + v);
      m[v] = t.x;
      m[v + 1] = t.y;
      m[v + 2] = t.z;
      m[v + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int v = 0; v < VW; ++v) m[v] = src[v];
  }
}

template <int VW>
__device__ __forceinline__ void recon_emit(const ReconArgs& a, int c, int x, int z0,
                                           const float (&acc)[VW], double& esq) {
  const int i = c / a.gn, j = c - (c / a.gn) * a.gn;
  const size_t o = (size_t)(i * a.Mb + x) * a.N + (size_t)j * a.Nb + z0;
  float out[VW];
  const float f = a.rowscale ? a.rowscale[i * a.Mb + x] : 1.0f;
#pragma unroll
  for (int v = 0; v < VW; ++v) out[v] = a.rowscale ? acc[v] * f : acc[v];
  if (a.C) {
#pragma unroll
    for (int v = 0; v < VW; ++v) a.C[o + v] = out[v];
  }
  if (a.Cref) {
#pragma unroll
    for (int v = 0; v < VW; ++v) {
      const double dlt = (double)out[v] - a.Cref[o + v];
      esq = __fma_rn(dlt, dlt, esq);
    }
  }
}

__device__ __forceinline__ void recon_reduce(const ReconArgs& a, double esq, double* red, int g,
                                             int nblk, int blk) {
  if (!a.Cref) return;
  red[threadIdx.x] = esq;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) a.partial[(size_t)g * nblk + blk] = red[0];
}

// Workgroup -> (gauge, position block).  The grid is 1-D over nblk * G
// workgroups; dispatch goes round-robin over the 8 XCDs, so remap to give
// each XCD a contiguous range of (position block major, gauge minor): the G
// gauges of a position block then share that XCD's L2 and the reference
// tile is fetched from memory about once per chunk instead of once per gauge.
__device__ __forceinline__ void recon_slot(int G, int nblk, int& g, int& blk) {
  const int total = G * nblk;
  int w = blockIdx.x;
  if ((total & 7) == 0) w = (w & 7) * (total >> 3) + (w >> 3);
  blk = w / G;
  g = w - blk * G;
}

// Products are read through a buffer resource over the gauge's slab of R
// products (base in the descriptor, r * block bytes as the scalar offset, the
// position as the vector offset), which keeps the 64-bit address arithmetic
// of the R product streams off the registers; the launcher checks that the
// slab fits the 32-bit offsets.  The gauge's coefficients are staged in LDS.
// Product loads go in groups of 8, double-buffered: the loads of group k+1
// are in flight while group k is accumulated (scheduling barriers keep the
// compiler from hoisting further).  The error epilogue goes 4 blocks at a
// time.  The grid gives every thread one position group (no loop), so no
// loop-invariant value is held across positions.
// Keeps the compiler from moving memory operations (or merging loads) across
// a group boundary, at the IR and the machine level; emits no instruction.
__device__ __forceinline__ void group_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Makes the accumulators appear read and written here, so every
// accumulation issued before this point in source order is done before it.
template <int NB, int VW>
__device__ __forceinline__ void pin_acc(float (&acc)[NB][VW]) {
#pragma unroll
  for (int c = 0; c < NB; ++c)
#pragma unroll
    for (int v = 0; v < VW; ++v) asm volatile("" : "+v"(acc[c][v]));
}

template <int VW, bool BF>
__device__ __forceinline__ void recon_load_buf(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                               uint32_t soff, float (&m)[VW]) {
  if constexpr (BF && VW == 4) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b64(rsrc, (int)voff, (int)soff, kStreamIn);
    m[0] = __uint_as_float(t[0] << 16);
    m[1] = __uint_as_float(t[0] & 0xffff0000u);
    m[2] = __uint_as_float(t[1] << 16);
    m[3] = __uint_as_float(t[1] & 0xffff0000u);
  } else if constexpr (BF) {
#pragma unroll
    for (int v = 0; v < VW; ++v)
      m[v] = __uint_as_float(
          (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rsrc, (int)(voff + 2 * v), (int)soff, kStreamIn) << 16);
  } else if constexpr (VW == 4) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)voff, (int)soff, kStreamIn);
#pragma unroll
    for (int v = 0; v < 4; ++v) m[v] = __uint_as_float(t[v]);
  } else {
#pragma unroll
    for (int v = 0; v < VW; ++v)
      m[v] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)(voff + 4 * v), (int)soff, kStreamIn));
  }
}

template <class P, int VW, bool BF>
__global__ __launch_bounds__(kThreads) void recon_static_kernel(ReconArgs a, int nblk) {
  constexpr int NNZ = P::rowptr[P::R];
  constexpr int GR = 8, NG = (P::R + GR - 1) / GR;
  __shared__ double red[kThreads];
  __shared__ float cl[NNZ];
  int g, blk;
  recon_slot(a.G, nblk, g, blk);
  const auto coef = ro(a.coef) + ro(a.off)[(size_t)g * (P::R + 1)];
  for (int e = threadIdx.x; e < NNZ; e += kThreads) cl[e] = coef[e];
  __syncthreads();
  const int bcv = a.Nb / VW;
  const int Ptot = a.Mb * bcv;
  const size_t bsz = (size_t)a.Mb * a.Nb;
  constexpr uint32_t esz = BF ? 2u : 4u;  // bytes per product value
  const uint32_t bbytes = (uint32_t)(bsz * esz);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(reinterpret_cast<const char*>(a.Mprod) + (size_t)g * P::R * bbytes),
      (short)0, (int)(P::R * bbytes), 0x00020000);
  double esq = 0.0;
  const int p = blk * kThreads + threadIdx.x;
  if (p < Ptot) {
    // products in the tiled layout: thread p takes the p-th 16-byte piece
    // (4 positions per thread) or the p-th value (one position: value p % 4
    // of piece p / 4), so a wave reads contiguous bytes either way
    const bool tl = (VW == 4 || VW == 1) && !BF && a.tiled;
    int x, z0;
    if (tl && VW == 4) {
      tile_layout_position(p, a.Nb, a.tiled, x, z0);
    } else if (tl) {
      tile_layout_position(p >> 2, a.Nb, a.tiled, x, z0);
      z0 += p & 3;
    } else {
      x = p / bcv;
      z0 = (p - x * bcv) * VW;
    }
    const uint32_t voff = tl ? (uint32_t)p * (uint32_t)(VW * 4) : (uint32_t)(x * a.Nb + z0) * esz;
    float acc[P::NB][VW];
#pragma unroll
    for (int c = 0; c < P::NB; ++c)
#pragma unroll
      for (int v = 0; v < VW; ++v) acc[c][v] = 0.0f;
    float mb[2][GR][VW];
    auto load_group = [&](auto gc) {
      constexpr int gi = decltype(gc)::value;
      sfor<0, GR>([&](auto jc) {
        constexpr int j = decltype(jc)::value, r = gi * GR + j;
        if constexpr (r < P::R) {
          if constexpr (P::rowptr[r + 1] > P::rowptr[r])
            recon_load_buf<VW, BF>(rsrc, voff, (uint32_t)r * bbytes, mb[gi & 1][j]);
        }
      });
    };
    load_group(std::integral_constant<int, 0>{});
    sfor<0, NG>([&](auto gc) {
      constexpr int gi = decltype(gc)::value;
      if constexpr (gi + 1 < NG) load_group(std::integral_constant<int, gi + 1>{});
      group_fence();
      sfor<0, GR>([&](auto jc) {
        constexpr int j = decltype(jc)::value, r = gi * GR + j;
        if constexpr (r < P::R) {
          sfor<P::rowptr[r], P::rowptr[r + 1]>([&](auto ec) {
            constexpr int e = decltype(ec)::value;
            constexpr int c = P::idx[e];
            const float w = cl[e];
#pragma unroll
            for (int v = 0; v < VW; ++v) acc[c][v] = __builtin_fmaf(w, mb[gi & 1][j][v], acc[c][v]);
          });
        }
      });
      pin_acc(acc);
      group_fence();
    });
    sfor<0, P::NB>([&](auto cc) {
      constexpr int c = decltype(cc)::value;
      if constexpr (c % 4 == 0) group_fence();
      recon_emit<VW>(a, c, x, z0, acc[c], esq);
    });
  }
  recon_reduce(a, esq, red, g, nblk, blk);
}

template <int VW, bool BF>
__global__ __launch_bounds__(kThreads) void recon_generic_kernel(ReconArgs a, int nblk) {
  __shared__ double red[kThreads];
  extern __shared__ float lacc[];  // [NC][thread][VW]
  int g, blk;
  recon_slot(a.G, nblk, g, blk);
  const int R = a.R, NC = a.gm * a.gn;
  const int bcv = a.Nb / VW;
  const int Ptot = a.Mb * bcv;
  const size_t bsz = (size_t)a.Mb * a.Nb;
  const int32_t* off = a.off + (size_t)g * (R + 1);
  double esq = 0.0;
  for (int base = blk * kThreads; base < Ptot; base += nblk * kThreads) {
    const int p = base + threadIdx.x;
    if (p >= Ptot) break;
    const int x = p / bcv, z0 = (p - x * bcv) * VW;
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int v = 0; v < VW; ++v) lacc[((size_t)c * kThreads + threadIdx.x) * VW + v] = 0.0f;
    const size_t o = (size_t)g * R * bsz + (size_t)x * a.Nb + z0;
    for (int r = 0; r < R; ++r) {
      const int e0 = off[r], e1 = off[r + 1];
      if (e0 == e1) continue;
      float m[VW];
      if constexpr (BF)
        recon_load_bf16<VW>(reinterpret_cast<const uint16_t*>(a.Mprod) + o + (size_t)r * bsz, m);
      else
        recon_load<VW>(a.Mprod + o + (size_t)r * bsz, m);
      for (int e = e0; e < e1; ++e) {
        const float w = a.coef[e];
        float* s = lacc + ((size_t)a.idx[e] * kThreads + threadIdx.x) * VW;
#pragma unroll
        for (int v = 0; v < VW; ++v) s[v] = __builtin_fmaf(w, m[v], s[v]);
      }
    }
    for (int c = 0; c < NC; ++c) {
      float acc[VW];
#pragma unroll
      for (int v = 0; v < VW; ++v) acc[v] = lacc[((size_t)c * kThreads + threadIdx.x) * VW + v];
      recon_emit<VW>(a, c, x, z0, acc, esq);
    }
  }
  recon_reduce(a, esq, red, g, nblk, blk);
}

inline int launched(const char* what) { return hip_check(hipGetLastError(), what); }

// Workgroups for operand formation: enough to cover the GPU several times,
// each looping over position groups; gauges split over grid.y.
inline dim3 form_grid(const FormArgs& a, int vw, int max_gpb, int& gpb) {
  const int P = a.br * (a.bc / vw);
  const int gx_full = (P + kThreads - 1) / kThreads;
  // Split the gauges over grid.y so that the launch has at least ~2048
  // workgroups (8 per CU), keeping at most 16 KB of amax slots in LDS.
  const int target = 2048;
  const int slices = std::max(1, std::min(a.G, (target + gx_full - 1) / gx_full));
  gpb = (a.G + slices - 1) / slices;
  gpb = std::max(1, std::min(gpb, max_gpb));
  const int gy = (a.G + gpb - 1) / gpb;
  int gx = gx_full;
  if ((long long)gx * gy > 4 * target) gx = std::max(1, 4 * target / gy);
  return dim3(gx, gy);
}

template <class P>
constexpr int static_vw() {
  return P::NB <= 4 ? 16 : (P::NB <= 16 ? 8 : 2);
}

template <class P, int MODE>
int launch_form_static(const FormArgs& a, hipStream_t st) {
  constexpr int VW = static_vw<P>();
  int gpb;
  if (a.per_row) {  // maxima go straight to global memory: no LDS table
    const dim3 grid = form_grid(a, VW, a.G, gpb);
    form_static_kernel<P, VW, MODE, true><<<grid, kThreads, 0, st>>>(a, gpb);
    return launched("form_static_kernel");
  }
  // mode 0 LDS: 16 row slots per (gauge, product), at most 48 KB
  const int max_gpb = MODE == 0 ? std::max(1, 12288 / (P::R * 16)) : a.G;
  const dim3 grid = form_grid(a, VW, max_gpb, gpb);
  const size_t shm = (MODE == 0) ? (size_t)gpb * P::R * 16 * 4 : 0;
  form_static_kernel<P, VW, MODE, false><<<grid, kThreads, shm, st>>>(a, gpb);
  return launched("form_static_kernel");
}

// The merged pass (form_merged_kernel): the encoding's grid, the maxima's
// gauges spread over the same slices, with more slices when a slice's
// maxima would not fit their LDS slots (at most 48 KB, as the separate
// maxima pass).
template <class P>
int launch_form_merged(const FormArgs& aq, const FormArgs& am, hipStream_t st) {
  constexpr int VW = static_vw<P>();
  constexpr int max_gpbm = 12288 / (P::R * 16);
  if (max_gpbm < 1) return 1;
  int gpbq;
  dim3 grid = form_grid(aq, VW, aq.G, gpbq);
  if ((am.G + (int)grid.y - 1) / (int)grid.y > max_gpbm) {
    const int gy = (am.G + max_gpbm - 1) / max_gpbm;
    gpbq = (aq.G + gy - 1) / gy;
    grid.y = (unsigned)std::max(gy, (aq.G + gpbq - 1) / gpbq);
    if ((long long)grid.x * grid.y > 4 * 2048) grid.x = (unsigned)std::max(1, 4 * 2048 / (int)grid.y);
  }
  const int gpbm = (am.G + (int)grid.y - 1) / (int)grid.y;
  if (gpbm > max_gpbm || (long long)gpbq * grid.y < aq.G) return 1;
  const size_t shm = (size_t)gpbm * P::R * 16 * 4;
  const int gx = (int)grid.x, gy = (int)grid.y;
  if (aq.fmt == FM_E4M3)
    form_merged_kernel<P, VW, FM_E4M3><<<gx * gy, kThreads, shm, st>>>(aq, am, gpbq, gpbm, gx, gy);
  else
    form_merged_kernel<P, VW, FM_E5M2><<<gx * gy, kThreads, shm, st>>>(aq, am, gpbq, gpbm, gx, gy);
  return launched("form_merged_kernel");
}

template <class P>
bool static_ok(const FormArgs& a) {
  constexpr int VW = static_vw<P>();
  // prefix-shared families: tensor scales only for sign variants of the
  // base scheme (a.trie, with their block signs in a.sgn); others go generic
  if (P::TRIE && !a.per_row && (!a.trie || !a.sgn)) return false;
  return a.gr * a.gc == P::NB && a.R == P::R && a.bc % VW == 0 && (VW < 4 || a.cols % 4 == 0) &&
         (size_t)P::R * a.br * a.bc < ((size_t)1 << 31);
}

template <int VW>
int launch_form_generic_t(const FormArgs& a, int mode, hipStream_t st) {
  int gpb;
  const dim3 grid = form_grid(a, VW, mode == 0 ? std::max(1, 4096 / std::max(1, a.R)) : a.G, gpb);
  const size_t shm = (size_t)a.gr * a.gc * kThreads * VW * 4 + (mode == 0 ? (size_t)gpb * a.R * 4 : 0);
  if (shm > 160 * 1024) return fail(FM_E_UNSUPPORTED, "formation needs too much LDS");
  const void* fn = mode == 0 ? reinterpret_cast<const void*>(&form_generic_kernel<VW, 0>)
                             : reinterpret_cast<const void*>(&form_generic_kernel<VW, 1>);
  if (int rc = hip_check(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)shm),
                         "hipFuncSetAttribute"))
    return rc;
  if (mode == 0)
    form_generic_kernel<VW, 0><<<grid, kThreads, shm, st>>>(a, gpb);
  else
    form_generic_kernel<VW, 1><<<grid, kThreads, shm, st>>>(a, gpb);
  return launched("form_generic_kernel");
}

inline int launch_form_generic(const FormArgs& a, int mode, hipStream_t st) {
  const int nb = a.gr * a.gc;
  if (nb <= 16 && a.bc % 4 == 0) return launch_form_generic_t<4>(a, mode, st);
  return launch_form_generic_t<1>(a, mode, st);
}

template <class P>
constexpr int recon_vw() {
  return P::NB <= 16 ? 4 : 1;
}

template <class P>
int launch_recon_static(const ReconArgs& a, hipStream_t st) {
  constexpr int VW = recon_vw<P>();
  const int nblk = recon_blocks(a);
  // the kernel gives each thread exactly one position group
  if (recon_width(a) != VW || (long long)nblk * kThreads < (long long)a.Mb * (a.Nb / VW))
    return fail(FM_E_UNSUPPORTED, "reconstruction grid does not cover the block");
  if (a.tiled && a.prod_bf16) return fail(FM_E_UNSUPPORTED, "tiled products need fp32 values");
  if (a.prod_bf16)
    recon_static_kernel<P, VW, true><<<nblk * a.G, kThreads, 0, st>>>(a, nblk);
  else
    recon_static_kernel<P, VW, false><<<nblk * a.G, kThreads, 0, st>>>(a, nblk);
  return launched("recon_static_kernel");
}

inline int launch_recon_generic(const ReconArgs& a, hipStream_t st) {
  const int nc = a.gm * a.gn;
  const int nblk = recon_blocks(a);
  const int grid = nblk * a.G;
  const bool wide = recon_width(a) == 4;
  const size_t shm = (size_t)nc * kThreads * 4 * (wide ? 4 : 1);
  const bool bf = a.prod_bf16 != 0;
  const void* fn = wide ? (bf ? reinterpret_cast<const void*>(&recon_generic_kernel<4, true>)
                              : reinterpret_cast<const void*>(&recon_generic_kernel<4, false>))
                        : (bf ? reinterpret_cast<const void*>(&recon_generic_kernel<1, true>)
                              : reinterpret_cast<const void*>(&recon_generic_kernel<1, false>));
  if (int rc = hip_check(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)shm),
                         "hipFuncSetAttribute"))
    return rc;
  if (wide && bf)
    recon_generic_kernel<4, true><<<grid, kThreads, shm, st>>>(a, nblk);
  else if (wide)
    recon_generic_kernel<4, false><<<grid, kThreads, shm, st>>>(a, nblk);
  else if (bf)
    recon_generic_kernel<1, true><<<grid, kThreads, shm, st>>>(a, nblk);
  else
    recon_generic_kernel<1, false><<<grid, kThreads, shm, st>>>(a, nblk);
  return launched("recon_generic_kernel");
}


}  // namespace dev

// Entry points of one specialized family (defined in fm_fam_<P>.hip).
// Return 1 when the arguments do not fit the family's kernels (the caller
// then uses the generic kernels), else FM_OK or an error code.
#define FM_DECLARE_FAMILY(P)                                                  \
  int form_family_##P(const FormArgs& a, int mode, int side, hipStream_t st); \
  int form_merged_family_##P(const FormArgs& aq, const FormArgs& am, int side,  \
                             hipStream_t st);                                  \
  int recon_family_##P(const ReconArgs& a, hipStream_t st);
FM_PATTERN_FAMILIES(FM_DECLARE_FAMILY)
#undef FM_DECLARE_FAMILY

#define FM_DEFINE_FAMILY(P)                                                          \
  int form_family_##P(const FormArgs& a, int mode, int side, hipStream_t st) {       \
    using namespace dev;                                                             \
    if (side == 0) {                                                                 \
      if (!static_ok<pat::P::A>(a)) return 1;                                        \
      return mode ? launch_form_static<pat::P::A, 1>(a, st)                          \
                  : launch_form_static<pat::P::A, 0>(a, st);                         \
    }                                                                                \
    if (!static_ok<pat::P::B>(a)) return 1;                                          \
    return mode ? launch_form_static<pat::P::B, 1>(a, st)                            \
                : launch_form_static<pat::P::B, 0>(a, st);                           \
  }                                                                                  \
  int form_merged_family_##P(const FormArgs& aq, const FormArgs& am, int side,       \
                             hipStream_t st) {                                       \
    using namespace dev;                                                             \
    if (aq.per_row || am.per_row) return 1;                                          \
    if (side == 0) {                                                                 \
      if (!static_ok<pat::P::A>(aq) || !static_ok<pat::P::A>(am)) return 1;          \
      return launch_form_merged<pat::P::A>(aq, am, st);                              \
    }                                                                                \
    if (!static_ok<pat::P::B>(aq) || !static_ok<pat::P::B>(am)) return 1;            \
    return launch_form_merged<pat::P::B>(aq, am, st);                                \
  }                                                                                  \
  int recon_family_##P(const ReconArgs& a, hipStream_t st) {                         \
    using namespace dev;                                                             \
    using W = pat::P::W;                                                             \
    if (a.gm * a.gn != W::NB || a.R != W::R || a.Nb % recon_vw<W>() != 0 || a.N % 4 || \
        (size_t)a.R * a.Mb * a.Nb * 4 >= ((size_t)1 << 32))                          \
      return a.tiled ? fail(FM_E_UNSUPPORTED, "tiled products need the family kernel") : 1; \
    return launch_recon_static<W>(a, st);                                            \
  }

}  // namespace fm
