// AdamW step on the coefficient values of C (the optimizer of Appendix G), for one adapter or a
// stack of adapters in one launch.  The arrays are elementwise, so any layout works (the plan
// layout included: padding slots hold c = g = m = v = 0 and stay 0).
//
// Per element, with the bias corrections bc1 = 1 - beta1^t, bc2 = 1 - beta2^t from the host:
//   c <- c (1 - lr wd);  m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2
//   c <- c - lr (m / bc1) / (sqrt(v / bc2) + eps)
// Each thread handles four consecutive elements with 16-byte accesses where the arrays allow.
#include <cmath>

#include "ff_internal.h"

namespace ff {
namespace {

struct AdamArgs {
  float* c;
  const float* g;
  float* m;
  float* v;
  float* const* cs;
  const float* const* gs;
  float* const* ms;
  float* const* vs;
  long n;
  float lr, beta1, beta2, eps, decay, inv_bc1, inv_bc2;
};

__device__ __forceinline__ void adam_elem(float& c, float g, float& m, float& v, const AdamArgs& a) {
  c *= a.decay;
  m = fmaf(a.beta1, m, (1.f - a.beta1) * g);
  v = fmaf(a.beta2, v, (1.f - a.beta2) * (g * g));
  const float den = sqrtf(v * a.inv_bc2) + a.eps;
  c -= a.lr * ((m * a.inv_bc1) / den);
}

__global__ void __launch_bounds__(256) adamw_kernel(AdamArgs a, int vec) {
  const int bi = blockIdx.y;
  float* c = a.cs ? a.cs[bi] : a.c;
  const float* g = a.gs ? a.gs[bi] : a.g;
  float* m = a.ms ? a.ms[bi] : a.m;
  float* v = a.vs ? a.vs[bi] : a.v;
  const long i0 = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i0 >= a.n) return;
  if (vec && i0 + 4 <= a.n) {
    float4 cc = *reinterpret_cast<const float4*>(c + i0);
    const float4 gg = *reinterpret_cast<const float4*>(g + i0);
    float4 mm = *reinterpret_cast<const float4*>(m + i0);
    float4 vv = *reinterpret_cast<const float4*>(v + i0);
    adam_elem(cc.x, gg.x, mm.x, vv.x, a);
    adam_elem(cc.y, gg.y, mm.y, vv.y, a);
    adam_elem(cc.z, gg.z, mm.z, vv.z, a);
    adam_elem(cc.w, gg.w, mm.w, vv.w, a);
    *reinterpret_cast<float4*>(c + i0) = cc;
    *reinterpret_cast<float4*>(m + i0) = mm;
    *reinterpret_cast<float4*>(v + i0) = vv;
    return;
  }
  for (long i = i0; i < a.n && i < i0 + 4; ++i) {
    float cc = c[i], mm = m[i], vv = v[i];
    adam_elem(cc, g[i], mm, vv, a);
    c[i] = cc;
    m[i] = mm;
    v[i] = vv;
  }
}

}  // namespace

hipError_t launch_adamw(int count, long n, float* c, const float* g, float* m, float* v, float* const* cs,
                        const float* const* gs, float* const* ms, float* const* vs, float lr, float beta1,
                        float beta2, float eps, float weight_decay, long step, int aligned16, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  AdamArgs a{c, g, m, v, cs, gs, ms, vs, n, lr, beta1, beta2, eps, 0.f, 0.f, 0.f};
  a.decay = (float)(1.0 - (double)lr * (double)weight_decay);
  a.inv_bc1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)step)));
  a.inv_bc2 = (float)(1.0 / (1.0 - std::pow((double)beta2, (double)step)));
  const dim3 grid((unsigned)((n + 1023) / 1024), (unsigned)count);
  hipLaunchKernelGGL(adamw_kernel, grid, dim3(256), 0, s, a, aligned16);
  return hipGetLastError();
}

namespace {

ff_status check_hparams(int64_t n, int64_t count, float lr, float beta1, float beta2, float eps, float wd,
                        int64_t step) {
  if (n < 0 || n > ((int64_t)1 << 40) || count < 1 || count > 65535)
    return fail(FF_EINVAL, "n=%lld or count=%lld out of range", (long long)n, (long long)count);
  if (step < 1) return fail(FF_EINVAL, "step numbers start at 1 (got %lld)", (long long)step);
  if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f))
    return fail(FF_EINVAL, "betas must lie in [0, 1)");
  if (!(eps > 0.f) || !std::isfinite(lr) || !std::isfinite(wd) || !(lr >= 0.f) || !(wd >= 0.f))
    return fail(FF_EINVAL, "need eps > 0 and finite lr, weight_decay >= 0");
  return FF_OK;
}

ff_status launched(hipError_t e) {
  return e == hipSuccess ? FF_OK : fail(FF_EDEVICE, "AdamW launch: %s", hipGetErrorString(e));
}

}  // namespace

}  // namespace ff

extern "C" {

ff_status ff_adamw_step(int64_t n, float* c, const float* g, float* m, float* v, float lr, float beta1, float beta2,
                        float eps, float weight_decay, int64_t step, void* stream) {
  ff::clear_error();
  ff_status st = ff::check_hparams(n, 1, lr, beta1, beta2, eps, weight_decay, step);
  if (st != FF_OK || n == 0) return st;
  if (!c || !g || !m || !v) return ff::fail(FF_EINVAL, "NULL array");
  for (const void* p : {(const void*)c, (const void*)g, (const void*)m, (const void*)v})
    if ((uintptr_t)p % 4) return ff::fail(FF_EINVAL, "arrays must be 4-byte aligned");
  const int aligned16 = ((uintptr_t)c | (uintptr_t)g | (uintptr_t)m | (uintptr_t)v) % 16 == 0;
  return ff::launched(ff::launch_adamw(1, (long)n, c, g, m, v, nullptr, nullptr, nullptr, nullptr, lr, beta1, beta2,
                                      eps, weight_decay, (long)step, aligned16, (hipStream_t)stream));
}

ff_status ff_adamw_step_batched(int64_t count, int64_t n, float* const* c, const float* const* g, float* const* m,
                                float* const* v, float lr, float beta1, float beta2, float eps, float weight_decay,
                                int64_t step, void* stream) {
  ff::clear_error();
  ff_status st = ff::check_hparams(n, count, lr, beta1, beta2, eps, weight_decay, step);
  if (st != FF_OK || n == 0) return st;
  if (!c || !g || !m || !v) return ff::fail(FF_EINVAL, "NULL pointer array");
  return ff::launched(ff::launch_adamw((int)count, (long)n, nullptr, nullptr, nullptr, nullptr, c, g, m, v, lr, beta1,
                                      beta2, eps, weight_decay, (long)step, 1, (hipStream_t)stream));
}

double ff_lr_linear_warmup(int64_t step, int64_t warmup, int64_t total, double base_lr) {
  if (step < warmup) return base_lr * (double)step / (double)(warmup > 1 ? warmup : 1);
  const double left = (double)(total - step) / (double)(total - warmup > 1 ? total - warmup : 1);
  return base_lr * (left > 0.0 ? left : 0.0);
}

}  // extern "C"
