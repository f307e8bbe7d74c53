// The LDS ring shared by the pipelined matrix kernels (block products and
// the integer operators): a persistent workgroup of 8 waves computes 256 x
// 128 output tiles, K step 128 bytes, through a ring of 3 LDS stages of 48 KB
// (256 + 128 rows of 128 bytes) filled by direct global-to-LDS loads.
//
// global_load_lds_dwordx4: lane L of a wave writes the 16 bytes it fetched at
// M0 + 16 L, so one wave-load fills 8 rows of 128 bytes; the XOR swizzle of
// the 16-byte chunks within a row (chunk ^ swz(row), so that fragment reads
// of 16 rows x one chunk hit distinct banks) is applied by choosing each
// lane's source chunk.  The loads are issued from inline assembly and
// awaited with explicit vmcnt counts: the compiler's own tracking of LDS DMA
// cannot tell the ring stages apart and would drain every load in flight
// before each LDS read.  Vector memory operations complete in issue order
// on this architecture, so "the group for stage s is complete" is "at most n
// operations outstanding", n = the number issued after that group (the next
// group's loads and any epilogue stores); a lower bound on n is always safe.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fm {
namespace ring {

constexpr int GK = 128;  // K step in bytes
constexpr int DBM = 256, DBN = 128, DROWS = DBM + DBN, DSTAGE = DROWS * GK, DNS = 3;
constexpr int DNT = 512;                       // 8 waves
constexpr int DLOADS = DROWS * GK / 1024 / 8;  // 1 KB wave-loads per wave per stage (= 6)
constexpr int DSTORES = 16;                    // 16-byte stores per lane, interior tile

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

__device__ __forceinline__ void dma16(const void* src, uint32_t lds_addr) {
  // M0 written by SALU then read by an LDS-DMA load needs one wait state
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds_addr)
               : "memory", "m0");
}

// s_waitcnt constraining only the vector-memory counter (gfx9 encoding:
// vmcnt low bits [3:0], expcnt [6:4], lgkmcnt [11:8], vmcnt high bits [15:14])
template <int N>
__device__ __forceinline__ void wait_vm_n() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_vm(int n) {
  // n is uniform and one of few values; anything else waits for everything
  if (n >= DLOADS + DSTORES) wait_vm_n<DLOADS + DSTORES>();
  else if (n >= DSTORES) wait_vm_n<DSTORES>();
  else if (n >= DLOADS) wait_vm_n<DLOADS>();
  else wait_vm_n<0>();
}

}  // namespace ring
}  // namespace fm

#define FM_COMPILER_FENCE() asm volatile("" ::: "memory")
