// Instantiation of one generic kernel (fwd_kernel or bwd_kernel, GEN_BWD) for one activation type
// (GEN_BF16): the build compiles this file four times with those macros set, in parallel.
#include "gen_kernels.h"

#if !defined(GEN_BWD) || !defined(GEN_BF16)
#error "compile with -DGEN_BWD=0|1 -DGEN_BF16=0|1"
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

hipError_t GEN_LAUNCH(const GEN_ARGS& a, dim3 grid, size_t lds, hipStream_t s) {
  if (a.nch > 1)
    hipLaunchKernelGGL((GEN_KERNEL<GEN_BF16 != 0, true>), grid, dim3(kFusedThreads), lds, s, a);
  else
    hipLaunchKernelGGL((GEN_KERNEL<GEN_BF16 != 0, false>), grid, dim3(kFusedThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t GEN_CONFIGURE() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&GEN_KERNEL<GEN_BF16 != 0, true>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
  const hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(&GEN_KERNEL<GEN_BF16 != 0, false>),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
  return e != hipSuccess ? e : e2;
}

}  // namespace gen
}  // namespace ff
