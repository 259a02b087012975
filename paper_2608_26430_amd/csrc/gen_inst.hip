// Instantiation of one generic kernel (fwd_kernel or bwd_kernel, GEN_BWD) for one activation type
// (GEN_BF16), and for frames applied in several radix-4 stages or the others (GEN_MS): the build
// compiles this file eight times with those macros set, in parallel.
#include "gen_kernels.h"

#if !defined(GEN_BWD) || !defined(GEN_BF16) || !defined(GEN_MS)
#error "compile with -DGEN_BWD=0|1 -DGEN_BF16=0|1 -DGEN_MS=0|1"
#endif

namespace ff {
namespace gen {

#if GEN_BWD
#define GEN_KERNEL bwd_kernel
#define GEN_ARGS BwdArgs
#if GEN_BF16
#define GEN_LAUNCH launch_bwd_bf16
#define GEN_CONFIGURE configure_bwd_bf16
#else
#define GEN_LAUNCH launch_bwd_f32
#define GEN_CONFIGURE configure_bwd_f32
#endif
#else
#define GEN_KERNEL fwd_kernel
#define GEN_ARGS FwdArgs
#if GEN_BF16
#define GEN_LAUNCH launch_fwd_bf16
#define GEN_CONFIGURE configure_fwd_bf16
#else
#define GEN_LAUNCH launch_fwd_f32
#define GEN_CONFIGURE configure_fwd_f32
#endif
#endif
#define GEN_CAT2(a, b) a##b
#define GEN_CAT(a, b) GEN_CAT2(a, b)
#define GEN_LAUNCH_MS GEN_CAT(GEN_LAUNCH, _ms)
#define GEN_CONFIGURE_MS GEN_CAT(GEN_CONFIGURE, _ms)

// The instantiation for frames applied in several radix-4 stages (GEN_MS=1, its own compile unit:
// one block per frame side there, so never input-side chunks), and the other two (GEN_MS=0).
hipError_t GEN_LAUNCH_MS(const GEN_ARGS& a, dim3 grid, size_t lds, hipStream_t s);
hipError_t GEN_CONFIGURE_MS();

#if GEN_MS
hipError_t GEN_LAUNCH_MS(const GEN_ARGS& a, dim3 grid, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL((GEN_KERNEL<GEN_BF16 != 0, false, true>), grid, dim3(kFusedThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t GEN_CONFIGURE_MS() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&GEN_KERNEL<GEN_BF16 != 0, false, true>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
}
#else
hipError_t GEN_LAUNCH(const GEN_ARGS& a, dim3 grid, size_t lds, hipStream_t s) {
  if (a.fin.nst >= 2 || a.fout.nst >= 2) return GEN_LAUNCH_MS(a, grid, lds, s);
#if GEN_BF16
  if (a.g4) {   // token-grouped tiles (the plan sets g4 only for frames in at most one radix-4 stage)
    if (a.nch > 1)
      hipLaunchKernelGGL((GEN_KERNEL<true, true, false, true>), grid, dim3(kFusedThreads), lds, s, a);
    else
      hipLaunchKernelGGL((GEN_KERNEL<true, false, false, true>), grid, dim3(kFusedThreads), lds, s, a);
    return hipGetLastError();
  }
#endif
  if (a.nch > 1)
    hipLaunchKernelGGL((GEN_KERNEL<GEN_BF16 != 0, true>), grid, dim3(kFusedThreads), lds, s, a);
  else
    hipLaunchKernelGGL((GEN_KERNEL<GEN_BF16 != 0, false>), grid, dim3(kFusedThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t GEN_CONFIGURE() {
  hipError_t e = GEN_CONFIGURE_MS();
  for (const void* fn : {reinterpret_cast<const void*>(&GEN_KERNEL<GEN_BF16 != 0, true>),
                         reinterpret_cast<const void*>(&GEN_KERNEL<GEN_BF16 != 0, false>),
#if GEN_BF16
                         reinterpret_cast<const void*>(&GEN_KERNEL<true, false, false, true>),
                         reinterpret_cast<const void*>(&GEN_KERNEL<true, true, false, true>)
#else
                         reinterpret_cast<const void*>(&GEN_KERNEL<false, false>)
#endif
       }) {
    const hipError_t r = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (r != hipSuccess) e = r;
  }
  return e;
}
#endif

}  // namespace gen
}  // namespace ff
