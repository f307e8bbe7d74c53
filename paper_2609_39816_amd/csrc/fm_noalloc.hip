// fm_error_stats_noalloc (include/fm.h): the relative Frobenius error of
// fm_error_stats (App. B.1, against a float64 reference as in App. F) for
// callers that cannot allocate device memory.  The reduction's partial sums
// live in a file-scope device array of the library (one copy per device,
// held until the process ends) instead of a caller's workspace; the kernels
// are the ones fm_error_stats launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>

#include "fm_internal.h"

namespace {
// Layout: the per-workgroup partial sums (at most 1024 workgroups x 3
// doubles = 24 KB), then the 3 totals at the next 256-byte boundary.
constexpr size_t kScratchBytes = 32768;
constexpr size_t kMaxDevices = 64;
}  // namespace

static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

namespace fm {
namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current) by hipGetSymbolAddress.  In host
// code the array's own name is a host-side stand-in, never a device address.
int scratch_address(void** out) {
  int dev = -1;
  if (int rc = hip_check(hipGetDevice(&dev), "hipGetDevice")) return rc;
  if (dev < 0 || (size_t)dev >= kMaxDevices) return fail(FM_E_UNSUPPORTED, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (int rc = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress"))
      return rc;
    if (!p) return fail(FM_E_HIP, "hipGetSymbolAddress returned no address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FM_OK;
}

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }
}  // namespace
}  // namespace fm

extern "C" int fm_error_stats_noalloc(const float* C, const double* C_ref, int M, int N,
                                      fm_stats* out, void* hip_stream) try {
  using namespace fm;
  clear_error();
  if (!C || !C_ref || !out) return fail(FM_E_ARG, "null pointer");
  if (M < 1 || N < 1) return fail(FM_E_ARG, "sizes must be positive");
  const size_t n = (size_t)M * N;
  const int nblk = error_stats_blocks(n);
  const size_t tot_off = round256((size_t)nblk * 3 * sizeof(double));
  if (tot_off + 3 * sizeof(double) > kScratchBytes)
    return fail(FM_E_WORKSPACE, "the reduction needs more than the 32768-byte static scratch");
  void* base = nullptr;
  if (int rc = scratch_address(&base)) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  double* partial = (double*)base;
  double* tot = (double*)((char*)base + tot_off);
  // every partial and total is written before it is read: nothing to clear
  if (int rc = launch_error_stats(C, C_ref, n, partial, st)) return rc;
  if (int rc = launch_error_finalize(partial, nblk, tot, st)) return rc;
  double h[3];
  if (int rc = hip_check(hipMemcpyAsync(h, tot, sizeof(h), hipMemcpyDeviceToHost, st),
                         "hipMemcpyAsync(D2H)"))
    return rc;
  if (int rc = hip_check(hipStreamSynchronize(st), "hipStreamSynchronize")) return rc;
  out->err_sq = h[0];
  out->ref_sq = h[1];
  out->max_abs = h[2];
  out->rel_fro = h[1] > 0 ? std::sqrt(h[0]) / std::sqrt(h[1]) : 0.0;
  if (!std::isfinite(h[0])) return fail(FM_E_NONFINITE, "non-finite error sum");
  return FM_OK;
} catch (...) {
  return fm::host_failure();
}
