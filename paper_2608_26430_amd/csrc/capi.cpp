// C entry points of the hot path: argument checks, then one stream-ordered
// launch sequence.  Nothing here allocates or synchronises.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "ff_internal.h"

namespace ff {

namespace {
thread_local char g_msg[512] = "";
thread_local hipEvent_t g_ev_start = nullptr;
thread_local hipEvent_t g_ev_stop = nullptr;
}  // namespace

ff_status fail(ff_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() { g_msg[0] = '\0'; }

void take_timing_events(hipEvent_t* start, hipEvent_t* stop) {
  *start = g_ev_start;
  *stop = g_ev_stop;
  g_ev_start = g_ev_stop = nullptr;
}

}  // namespace ff

namespace {

bool aligned(const void* ptr, int act) {
  return ((uintptr_t)ptr % 16) == 0;
}

// Activation arrays.  Plans with a lift read and write the caller's rows one element at a time
// (lift.hip), so they need only element alignment; the other kernels use 16-byte accesses.
ff_status check_act(const char* name, const void* ptr, int64_t ld, int64_t width, int act, bool lifted = false) {
  if (!ptr) return ff::fail(FF_EINVAL, "%s is NULL", name);
  if (ld < width) return ff::fail(FF_EINVAL, "leading dimension of %s (%lld) < %lld", name, (long long)ld,
                                  (long long)width);
  if (lifted) {
    if ((uintptr_t)ptr % (act == FF_BF16 ? 2 : 4)) return ff::fail(FF_EINVAL, "%s is misaligned", name);
    return FF_OK;
  }
  const int64_t mult = act == FF_BF16 ? 8 : 4;
  if (ld % mult) return ff::fail(FF_EINVAL, "leading dimension of %s must be a multiple of %lld", name,
                                 (long long)mult);
  if (!aligned(ptr, act)) return ff::fail(FF_EINVAL, "%s is not 16-byte aligned", name);
  return FF_OK;
}

ff_status check_common(const ff_plan* p, int64_t T, int act, int64_t count) {
  if (!p) return ff::fail(FF_EINVAL, "plan is NULL");
  if (act != FF_F32 && act != FF_BF16) return ff::fail(FF_EINVAL, "unknown activation dtype %d", act);
  if (T < 0 || T > p->max_tokens)
    return ff::fail(FF_EINVAL, "T=%lld outside [0, max_tokens=%lld]", (long long)T, (long long)p->max_tokens);
  if (count < 1 || count > p->max_batch)
    return ff::fail(FF_EINVAL, "count=%lld outside [1, max_batch=%lld]", (long long)count,
                    (long long)p->max_batch);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != p->device)
    return ff::fail(FF_EINVAL, "current device %d is not the plan's device %d", dev, p->device);
  return FF_OK;
}

ff_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return ff::fail(FF_EDEVICE, "%s: %s", what, hipGetErrorString(e));
  return FF_OK;
}

// Argument checks of a single-adapter backward.  Sets *done when the call has nothing to launch.
ff_status check_bwd(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx, const void* G, int64_t ldg,
                    const float* c_vals, void* dX, int64_t lddx, int accumulate_dc, float* dC, bool* want_dx,
                    bool* want_dc, bool* done) {
  ff_status st = check_common(p, T, act, 1);
  if (st != FF_OK) return st;
  *want_dx = dX != nullptr;
  *want_dc = dC != nullptr && p->coef_slots > 0;
  *done = false;
  if (dC && ((uintptr_t)dC % 4)) return ff::fail(FF_EINVAL, "dC is not 4-byte aligned");
  if (T == 0) {
    *done = !*want_dc || accumulate_dc;               // empty sum: dC = 0 unless accumulating
    return FF_OK;
  }
  if (!*want_dx && !*want_dc) {
    *done = true;
    return FF_OK;
  }
  if ((st = check_act("G", G, ldg, p->fout->d, act, p->lifted)) != FF_OK) return st;
  if (*want_dc && (st = check_act("X", X, ldx, p->fin->d, act, p->lifted)) != FF_OK) return st;
  if (*want_dx && (st = check_act("dX", dX, lddx, p->fin->d, act, p->lifted)) != FF_OK) return st;
  if (*want_dx && p->coef_slots > 0 && !c_vals) return ff::fail(FF_EINVAL, "c_vals is NULL");
  if ((uintptr_t)c_vals % 16) return ff::fail(FF_EINVAL, "c_vals is not 16-byte aligned");
  return FF_OK;
}

// Scratch of ff_adapter_bwd_noalloc: the backward's dC partial sums and reordered coefficients,
// in device memory that the code object itself holds (no allocation at run time).  Each device
// has its own copy of the array at its own address, taken once per device with
// hipGetSymbolAddress; host code uses that address only, never the array's name.  Calls on one
// device share the array, so overlapping calls on one device race.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

ff_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return ff::fail(FF_EDEVICE, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return ff::fail(FF_EDEVICE, "address of the static scratch on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return FF_OK;
}

}  // namespace

extern "C" {

const char* ff_status_string(int status) {
  switch (status) {
    case FF_OK: return "FF_OK";
    case FF_EINVAL: return "FF_EINVAL";
    case FF_ENOTFF: return "FF_ENOTFF";
    case FF_EUNSUPPORTED: return "FF_EUNSUPPORTED";
    case FF_ENOMEM: return "FF_ENOMEM";
    case FF_EDEVICE: return "FF_EDEVICE";
    default: return "FF_UNKNOWN";
  }
}

const char* ff_last_error(void) { return ff::g_msg; }

int ff_abi_version(void) { return 1; }

ff_status ff_time_next_kernel(void* ev_start, void* ev_stop) {
  ff::clear_error();
  if ((ev_start == nullptr) != (ev_stop == nullptr))
    return ff::fail(FF_EINVAL, "pass both events or neither");
  ff::g_ev_start = (hipEvent_t)ev_start;
  ff::g_ev_stop = (hipEvent_t)ev_stop;
  return FF_OK;
}

ff_status ff_adapter_fwd(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx,
                         const float* c_vals, float scale, float beta, void* Y, int64_t ldy,
                         void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, T, act, 1);
  if (st != FF_OK) return st;
  if (T == 0) return FF_OK;
  if ((st = check_act("X", X, ldx, p->fin->d, act, p->lifted)) != FF_OK) return st;
  if ((st = check_act("Y", Y, ldy, p->fout->d, act, p->lifted)) != FF_OK) return st;
  if (p->coef_slots > 0 && !c_vals) return ff::fail(FF_EINVAL, "c_vals is NULL");
  if ((uintptr_t)c_vals % 16) return ff::fail(FF_EINVAL, "c_vals is not 16-byte aligned");
  if (p->lifted)
    return launched(ff::launch_fwd_lifted(p, act == FF_BF16, (int)T, X, ldx, c_vals, scale, beta, Y, ldy,
                                          (hipStream_t)stream),
                    "forward launch");
  return launched(ff::launch_fwd(p, act == FF_BF16, 1, (int)T, {X, nullptr}, ldx, c_vals, nullptr, scale,
                                 beta, {Y, nullptr}, ldy, nullptr, (hipStream_t)stream),
                  "forward launch");
}

ff_status ff_adapter_fwd_save(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx,
                              const float* c_vals, float scale, float beta, void* Y, int64_t ldy,
                              float* c_saved, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, T, act, 1);
  if (st != FF_OK) return st;
  const bool saves = act == FF_BF16 && p->fast.enabled;
  if (!saves) return ff_adapter_fwd(p, T, act, X, ldx, c_vals, scale, beta, Y, ldy, stream);
  if (!c_saved || (uintptr_t)c_saved % 16) return ff::fail(FF_EINVAL, "c_saved is NULL or not 16-byte aligned");
  if (!c_vals || (uintptr_t)c_vals % 16) return ff::fail(FF_EINVAL, "c_vals is NULL or not 16-byte aligned");
  if (T > 0) {
    if ((st = check_act("X", X, ldx, p->fin->d, act)) != FF_OK) return st;
    if ((st = check_act("Y", Y, ldy, p->fout->d, act)) != FF_OK) return st;
  }
  return launched(ff::launch_fwd(p, 1, 1, (int)T, {X, nullptr}, ldx, c_vals, nullptr, scale, beta, {Y, nullptr},
                                 ldy, c_saved, (hipStream_t)stream),
                  "forward launch");
}

ff_status ff_adapter_bwd(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx,
                         const void* G, int64_t ldg, const float* c_vals, float scale,
                         float beta_dx, void* dX, int64_t lddx, int accumulate_dc, float* dC,
                         void* stream) {
  ff::clear_error();
  bool want_dx, want_dc, done;
  const ff_status st = check_bwd(p, T, act, X, ldx, G, ldg, c_vals, dX, lddx, accumulate_dc, dC, &want_dx, &want_dc,
                                 &done);
  if (st != FF_OK || done) return st;
  if (p->lifted)
    return launched(ff::launch_bwd_lifted(p, act == FF_BF16, (int)T, X, ldx, G, ldg, c_vals, scale, beta_dx, dX, lddx,
                                          want_dx, accumulate_dc, dC, want_dc, (hipStream_t)stream),
                    "backward launch");
  return launched(ff::launch_bwd(p, act == FF_BF16, 1, (int)T, {X, nullptr}, ldx, {G, nullptr}, ldg, c_vals,
                                 nullptr, scale, beta_dx, {dX, nullptr}, lddx, want_dx, accumulate_dc, dC,
                                 nullptr, want_dc, nullptr, (hipStream_t)stream),
                  "backward launch");
}

ff_status ff_adapter_bwd_noalloc(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx,
                                 const void* G, int64_t ldg, const float* c_vals, float scale,
                                 float beta_dx, void* dX, int64_t lddx, int accumulate_dc, float* dC,
                                 void* stream) {
  ff::clear_error();
  bool want_dx, want_dc, done;
  ff_status st = check_bwd(p, T, act, X, ldx, G, ldg, c_vals, dX, lddx, accumulate_dc, dC, &want_dx, &want_dc,
                           &done);
  if (st != FF_OK || done) return st;
  // plans with a lift run the kernels in fp32 whatever the activation type
  const int kbf16 = act == FF_BF16 && !p->lifted;
  const size_t need = ff::bwd_scratch_floats(p, kbf16, (int)T) * sizeof(float);
  if (need > kScratchBytes)
    return ff::fail(FF_EINVAL, "this backward needs %zu bytes of scratch, more than the %zu bytes of the static "
                    "scratch (use fewer tokens per call)", need, kScratchBytes);
  void* base = nullptr;
  if ((st = scratch_address(p->device, &base)) != FF_OK) return st;
  const ff::BwdScratch ws{static_cast<float*>(base), kScratchBytes / sizeof(float)};
  if (p->lifted)
    return launched(ff::launch_bwd_lifted(p, act == FF_BF16, (int)T, X, ldx, G, ldg, c_vals, scale, beta_dx, dX, lddx,
                                          want_dx, accumulate_dc, dC, want_dc, (hipStream_t)stream, &ws),
                    "backward launch");
  return launched(ff::launch_bwd(p, act == FF_BF16, 1, (int)T, {X, nullptr}, ldx, {G, nullptr}, ldg, c_vals,
                                 nullptr, scale, beta_dx, {dX, nullptr}, lddx, want_dx, accumulate_dc, dC,
                                 nullptr, want_dc, nullptr, (hipStream_t)stream, &ws),
                  "backward launch");
}

ff_status ff_adapter_bwd_saved(const ff_plan* p, int64_t T, int act, const void* X, int64_t ldx,
                               const void* G, int64_t ldg, const float* c_vals, const float* c_saved,
                               float scale, float beta_dx, void* dX, int64_t lddx, int accumulate_dc,
                               float* dC, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, T, act, 1);
  if (st != FF_OK) return st;
  if (!(act == FF_BF16 && p->fast.enabled) || T == 0 || !dX)
    return ff_adapter_bwd(p, T, act, X, ldx, G, ldg, c_vals, scale, beta_dx, dX, lddx, accumulate_dc, dC, stream);
  if (!c_saved || (uintptr_t)c_saved % 16) return ff::fail(FF_EINVAL, "c_saved is NULL or not 16-byte aligned");
  const bool want_dc = dC != nullptr;
  if (dC && ((uintptr_t)dC % 4)) return ff::fail(FF_EINVAL, "dC is not 4-byte aligned");
  if ((st = check_act("G", G, ldg, p->fout->d, act)) != FF_OK) return st;
  if (want_dc && (st = check_act("X", X, ldx, p->fin->d, act)) != FF_OK) return st;
  if ((st = check_act("dX", dX, lddx, p->fin->d, act)) != FF_OK) return st;
  return launched(ff::launch_bwd(p, 1, 1, (int)T, {X, nullptr}, ldx, {G, nullptr}, ldg, c_vals, nullptr, scale,
                                 beta_dx, {dX, nullptr}, lddx, true, accumulate_dc, dC, nullptr, want_dc, c_saved,
                                 (hipStream_t)stream),
                  "backward launch");
}

ff_status ff_merge_delta(const ff_plan* p, const float* c_vals, float scale, int w_dtype, float beta,
                         void* W, int64_t ldw, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, 0, FF_F32, 1);
  if (st != FF_OK) return st;
  if (w_dtype != FF_F32 && w_dtype != FF_BF16) return ff::fail(FF_EINVAL, "unknown weight dtype %d", w_dtype);
  if (!W) return ff::fail(FF_EINVAL, "W is NULL");
  if (ldw < p->fin->d) return ff::fail(FF_EINVAL, "ldw < n");
  if ((uintptr_t)W % (w_dtype == FF_BF16 ? 2 : 4)) return ff::fail(FF_EINVAL, "W is misaligned");
  if (p->coef_slots > 0 && !c_vals) return ff::fail(FF_EINVAL, "c_vals is NULL");
  if ((uintptr_t)c_vals % 16) return ff::fail(FF_EINVAL, "c_vals is not 16-byte aligned");
  if (p->lifted)
    return launched(ff::launch_merge_lifted(p, c_vals, scale, w_dtype == FF_BF16, beta, W, ldw, (hipStream_t)stream),
                    "merge launch");
  return launched(ff::launch_merge(p, c_vals, scale, w_dtype == FF_BF16, beta, W, ldw, (hipStream_t)stream),
                  "merge launch");
}

ff_status ff_coef_to_plan(const ff_plan* p, const float* c_user, float* c_plan, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, 0, FF_F32, 1);
  if (st != FF_OK) return st;
  if (p->coef_slots == 0) return FF_OK;
  if (!c_plan || (uintptr_t)c_plan % 16) return ff::fail(FF_EINVAL, "c_plan is NULL or not 16-byte aligned");
  if (p->nnz > 0 && (!c_user || (uintptr_t)c_user % 4)) return ff::fail(FF_EINVAL, "c_user is NULL or misaligned");
  if (p->nnz > 0 && (const void*)c_user < (const void*)(c_plan + p->coef_slots) &&
      (const void*)c_plan < (const void*)(c_user + p->nnz))
    return ff::fail(FF_EINVAL, "c_user and c_plan overlap");
  return launched(ff::launch_coef_to_plan(p, c_user, c_plan, (hipStream_t)stream), "coefficient layout launch");
}

ff_status ff_coef_to_user(const ff_plan* p, const float* c_plan, float* c_user, int accumulate, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, 0, FF_F32, 1);
  if (st != FF_OK) return st;
  if (p->nnz == 0) return FF_OK;
  if (!c_plan || (uintptr_t)c_plan % 16) return ff::fail(FF_EINVAL, "c_plan is NULL or not 16-byte aligned");
  if (!c_user || (uintptr_t)c_user % 4) return ff::fail(FF_EINVAL, "c_user is NULL or misaligned");
  if ((const void*)c_user < (const void*)(c_plan + p->coef_slots) && (const void*)c_plan < (const void*)(c_user + p->nnz))
    return ff::fail(FF_EINVAL, "c_user and c_plan overlap");
  return launched(ff::launch_coef_to_user(p, c_plan, c_user, accumulate, (hipStream_t)stream),
                  "coefficient layout launch");
}

ff_status ff_adapter_fwd_batched(const ff_plan* p, int64_t count, int64_t T, int act,
                                 const void* const* X, int64_t ldx, const float* const* c_vals,
                                 float scale, float beta, void* const* Y, int64_t ldy, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, T, act, count);
  if (st != FF_OK) return st;
  if (p->lifted) return ff::fail(FF_EUNSUPPORTED, "batched calls need frames with k rho == d");
  if (T == 0) return FF_OK;
  if (!X || !Y || !c_vals) return ff::fail(FF_EINVAL, "pointer array is NULL");
  if (ldx < p->fin->d || ldy < p->fout->d) return ff::fail(FF_EINVAL, "leading dimension too small");
  const int64_t mult = act == FF_BF16 ? 8 : 4;
  if (ldx % mult || ldy % mult) return ff::fail(FF_EINVAL, "leading dimension not a multiple of %lld",
                                                (long long)mult);
  return launched(ff::launch_fwd(p, act == FF_BF16, (int)count, (int)T, {nullptr, X}, ldx, nullptr, c_vals,
                                 scale, beta, {nullptr, (const void* const*)Y}, ldy, nullptr, (hipStream_t)stream),
                  "batched forward launch");
}

ff_status ff_adapter_bwd_batched(const ff_plan* p, int64_t count, int64_t T, int act,
                                 const void* const* X, int64_t ldx, const void* const* G,
                                 int64_t ldg, const float* const* c_vals, float scale,
                                 float beta_dx, void* const* dX, int64_t lddx, int accumulate_dc,
                                 float* const* dC, void* stream) {
  ff::clear_error();
  ff_status st = check_common(p, T, act, count);
  if (st != FF_OK) return st;
  if (p->lifted) return ff::fail(FF_EUNSUPPORTED, "batched calls need frames with k rho == d");
  const bool want_dx = dX != nullptr, want_dc = dC != nullptr && p->coef_slots > 0;
  if (T == 0 && (!want_dc || accumulate_dc)) return FF_OK;
  if (T > 0) {
    if (!want_dx && !want_dc) return FF_OK;
    if (!G) return ff::fail(FF_EINVAL, "G pointer array is NULL");
    if (want_dc && !X) return ff::fail(FF_EINVAL, "X pointer array is NULL");
    if (want_dx && !c_vals && p->coef_slots > 0) return ff::fail(FF_EINVAL, "c_vals pointer array is NULL");
    const int64_t mult = act == FF_BF16 ? 8 : 4;
    if (ldg < p->fout->d || ldg % mult) return ff::fail(FF_EINVAL, "bad ldg");
    if (want_dc && (ldx < p->fin->d || ldx % mult)) return ff::fail(FF_EINVAL, "bad ldx");
    if (want_dx && (lddx < p->fin->d || lddx % mult)) return ff::fail(FF_EINVAL, "bad lddx");
  }
  return launched(ff::launch_bwd(p, act == FF_BF16, (int)count, (int)T, {nullptr, X}, ldx, {nullptr, G}, ldg,
                                 nullptr, c_vals, scale, beta_dx, {nullptr, (const void* const*)dX}, lddx,
                                 want_dx, accumulate_dc, nullptr, dC, want_dc, nullptr, (hipStream_t)stream),
                  "batched backward launch");
}

}  // extern "C"
