// CPU stand-in for what the library's host code needs from the HIP runtime and from its own
// kernel files, so that the host code (frame construction, plan building, argument checks,
// plan groups) can be built with AddressSanitizer and UndefinedBehaviorSanitizer and run on a
// machine without a GPU.  Test infrastructure only: nothing here is linked into libframeft.so.
//
// "Device" memory is host memory from malloc, so a device allocation that the library fails to
// free is reported by LeakSanitizer like any other leak.  hipMalloc fails on the call whose
// ordinal (1-based, counted from the last stub_fail_malloc_at) was requested.  Kernel launchers
// and configuration calls succeed and do nothing: the host code's checks run, no kernel does.
#include <cstdlib>
#include <cstring>

#include "ff_internal.h"

namespace {
long g_calls = 0;
long g_fail_at = 0;
}  // namespace

extern "C" void stub_fail_malloc_at(long n) {
  g_calls = 0;
  g_fail_at = n;
}
extern "C" long stub_malloc_calls() { return g_calls; }

extern "C" {
hipError_t hipMalloc(void** ptr, size_t size) {
  ++g_calls;
  if (!ptr) return hipErrorInvalidValue;
  *ptr = nullptr;
  if (g_fail_at && g_calls == g_fail_at) return hipErrorOutOfMemory;
  *ptr = std::malloc(size ? size : 1);
  return *ptr ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void* ptr) {
  std::free(ptr);
  return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  if (n) std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipMemset(void* dst, int v, size_t n) {
  if (n) std::memset(dst, v, n);
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipGetDeviceCount(int* n) {
  *n = 1;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t attr, int) {
  *v = attr == hipDeviceAttributeMultiprocessorCount ? 256 : 0;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stub"; }
hipError_t hipGetSymbolAddress(void** ptr, const void* symbol) {
  *ptr = const_cast<void*>(symbol);
  return hipSuccess;
}
}  // extern "C"

namespace ff {

hipError_t configure_kernels() { return hipSuccess; }
hipError_t configure_fast128() { return hipSuccess; }

// LDS and workspace sizes of the 128-wide kernels (their formulas in kernels_w128.hip: 8-token
// tiles of 128-wide blocks, four 4 KB wave tiles; the 16-token backward's 32-byte rows and
// eight wave tiles; at least the 16 KB of staged synthesis fragments), so that plans take the
// same paths as on the GPU.
size_t fast128_lds_bytes(int nblk) {
  const size_t b = (size_t)nblk * 128 * 8 * 2 + (size_t)4 * 2 * 128 * 8 * 2;
  return b < 16384 ? 16384 : b;
}
size_t fast128_partial_floats(size_t bwd_slots) { return bwd_slots + 256; }
size_t fast16_lds_bytes(int nblk_out) {
  const size_t b = (size_t)nblk_out * 128 * 16 * 2 + (size_t)8 * 2 * 128 * 8 * 2;
  return b < 16384 ? 16384 : b;
}

size_t bwd_scratch_floats(const ff_plan*, int, int T) { return T > 0 ? 4096 + (size_t)T : 0; }

hipError_t launch_fwd(const ff_plan*, int, int, int, ActPtrs, int64_t, const float*, const float* const*, float, float,
                      ActPtrs, int64_t, float*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_bwd(const ff_plan*, int, int, int, ActPtrs, int64_t, ActPtrs, int64_t, const float*,
                      const float* const*, float, float, ActPtrs, int64_t, bool, int, float*, float* const*, bool,
                      const float*, hipStream_t, const BwdScratch*) {
  return hipSuccess;
}
hipError_t launch_merge(const ff_plan*, const float*, float, int, float, void*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_fwd_lifted(const ff_plan*, int, int, const void*, int64_t, const float*, float, float, void*, int64_t,
                             hipStream_t) {
  return hipSuccess;
}
hipError_t launch_bwd_lifted(const ff_plan*, int, int, const void*, int64_t, const void*, int64_t, const float*, float,
                             float, void*, int64_t, bool, int, float*, bool, hipStream_t, const BwdScratch*) {
  return hipSuccess;
}
hipError_t launch_merge_lifted(const ff_plan*, const float*, float, int, float, void*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_fwd_group(const ff_plan_group*, int, int, const int*, const void* const*, int64_t,
                            const float* const*, float, float, void* const*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_bwd_group(const ff_plan_group*, int, int, const int*, const void* const*, int64_t,
                            const void* const*, int64_t, const float* const*, float, float, void* const*, int64_t,
                            bool, int, float* const*, bool, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_coef_to_plan(const ff_plan*, const float*, float*, hipStream_t) { return hipSuccess; }
hipError_t launch_coef_to_user(const ff_plan*, const float*, float*, int, hipStream_t) { return hipSuccess; }

}  // namespace ff
