// Plan groups: adapters that share a frame pair but each have their own support of C (per-layer
// random masks, Sec. 4.6; tenants with different adapters over one backbone, Sec. 3.4 "Storage
// efficiency"), run in one launch per kernel.  The group holds, per adapter, a device descriptor
// of its plan's tables and workspace; the plans keep their own allocations.
#include <algorithm>
#include <cstring>
#include <memory>
#include <set>
#include <vector>

#include "ff_internal.h"

namespace {

ff_status check_group_call(const ff_plan_group* g, int64_t T, int act) {
  if (!g) return ff::fail(FF_EINVAL, "group is NULL");
  if (act != FF_F32 && act != FF_BF16) return ff::fail(FF_EINVAL, "unknown activation dtype %d", act);
  if (T < 0 || T > g->max_tokens)
    return ff::fail(FF_EINVAL, "T=%lld outside [0, %lld] (the plans' smallest max_tokens)", (long long)T,
                    (long long)g->max_tokens);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != g->ref->device)
    return ff::fail(FF_EINVAL, "current device %d is not the group's device %d", dev, g->ref->device);
  return FF_OK;
}

ff_status check_ld(const char* name, int64_t ld, int64_t width, int act) {
  const int64_t mult = act == FF_BF16 ? 8 : 4;
  if (ld < width || ld % mult)
    return ff::fail(FF_EINVAL, "leading dimension of %s (%lld) must be >= %lld and a multiple of %lld", name,
                    (long long)ld, (long long)width, (long long)mult);
  return FF_OK;
}

ff_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return ff::fail(FF_EDEVICE, "%s: %s", what, hipGetErrorString(e));
  return FF_OK;
}

}  // namespace

extern "C" {

ff_status ff_plan_group_create(int64_t count, const ff_plan* const* plans, ff_plan_group** out) {
  ff::clear_error();
  if (!out) return ff::fail(FF_EINVAL, "out is NULL");
  *out = nullptr;
  if (count < 1 || count > 65535 || !plans) return ff::fail(FF_EINVAL, "need 1 <= count <= 65535 plans");
  const ff_plan* ref = plans[0];
  if (!ref) return ff::fail(FF_EINVAL, "plan 0 is NULL");
  if (ref->lifted) return ff::fail(FF_EUNSUPPORTED, "plan groups need frames with k rho == d");
  std::set<const ff_plan*> seen;
  for (int64_t i = 0; i < count; ++i) {
    const ff_plan* p = plans[i];
    if (!p) return ff::fail(FF_EINVAL, "plan %lld is NULL", (long long)i);
    if (!seen.insert(p).second)
      return ff::fail(FF_EINVAL, "plan %lld appears twice (adapters that share a support use the batched calls)",
                      (long long)i);
    if (p->fin != ref->fin || p->fout != ref->fout)
      return ff::fail(FF_EINVAL, "plan %lld uses other frames than plan 0", (long long)i);
    if (p->device != ref->device) return ff::fail(FF_EINVAL, "plan %lld is on another device", (long long)i);
    if (p->fast.enabled != ref->fast.enabled)
      return ff::fail(FF_EUNSUPPORTED, "plan %lld takes another kernel path than plan 0", (long long)i);
    bool same = p->gen_nch == ref->gen_nch && p->gen_g4 == ref->gen_g4 && p->dev.fwd_by_pos == ref->dev.fwd_by_pos;
    for (int k = 0; k < 2; ++k)
      same = same && p->gen_tile_tokens[k] == ref->gen_tile_tokens[k] && p->gen_ldt_in[k] == ref->gen_ldt_in[k] &&
             p->ldt_out[k] == ref->ldt_out[k] && p->gen_lds_bytes[k] == ref->gen_lds_bytes[k];
    for (int k = 0; same && k <= ref->gen_nch; ++k) same = p->gen_chunk_blk[k] == ref->gen_chunk_blk[k];
    if (!same)
      return ff::fail(FF_EUNSUPPORTED, "plan %lld splits the input side differently from plan 0 (supports of "
                      "very different density)", (long long)i);
  }
  auto g = std::make_unique<ff_plan_group>();
  g->count = count;
  g->plans.assign(plans, plans + count);
  g->ref = ref;
  g->max_tokens = ref->max_tokens;
  g->min_gen_rows = ref->gen_rows;
  std::vector<ff::FastDesc> fast((size_t)count);
  std::vector<ff::GenDesc> gen((size_t)count);
  for (int64_t i = 0; i < count; ++i) {
    const ff_plan* p = plans[i];
    g->max_tokens = std::min(g->max_tokens, p->max_tokens);
    g->min_gen_rows = std::min(g->min_gen_rows, p->gen_rows);
    const ff::FastPlanDev& f = p->fast;
    fast[i] = ff::FastDesc{f.fwd_pl, f.fwd_st, f.fwd_em, f.bwd_pl, f.bwd_st, f.bwd_em, f.bwd_dst, f.pad, f.bwd_pad,
                           f.bwd_pos, f.coef_bwd, p->partial, f.npad, f.nbpad, f.bwd_slots, f.coef_slots,
                           f.bwd16};
    g->fast16 |= f.bwd16 ? 1 : 0;
    g->fast8 |= f.bwd16 ? 0 : 1;
    const ff::PlanDev& d = p->dev;
    gen[i] = ff::GenDesc{d.fwd, d.bwd, d.coef_pad, d.c_fwd, d.c_bwd, p->partial, d.fwd_by_pos, d.ncoef_pad};
    g->max_fast_items = std::max(g->max_fast_items, f.coef_slots + f.nbpad);
    g->max_fast_slots = std::max(g->max_fast_slots, f.bwd_slots);
    g->max_fast_npad = std::max(g->max_fast_npad, f.npad);
    g->max_gen_fwd = std::max(g->max_gen_fwd, 64 * d.fwd.rows);
    g->max_gen_bwd = std::max(g->max_gen_bwd, 64 * d.bwd.rows);
    g->max_gen_npad = std::max(g->max_gen_npad, d.ncoef_pad);
    g->any_fwd_gather |= d.fwd_by_pos ? 0 : 1;
  }
  const size_t fb = fast.size() * sizeof(ff::FastDesc), gb = gen.size() * sizeof(ff::GenDesc);
  const size_t goff = (fb + 255) & ~(size_t)255;
  void* mem = nullptr;
  if (hipMalloc(&mem, goff + gb) != hipSuccess) {
    (void)hipGetLastError();
    return ff::fail(FF_ENOMEM, "hipMalloc of the group's descriptors failed");
  }
  if (hipMemcpy(mem, fast.data(), fb, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy((char*)mem + goff, gen.data(), gb, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(mem);
    return ff::fail(FF_EDEVICE, "copying the group's descriptors failed");
  }
  g->dev_mem = mem;
  g->fast = static_cast<const ff::FastDesc*>(mem);
  g->gen = reinterpret_cast<const ff::GenDesc*>((char*)mem + goff);
  *out = g.release();
  return FF_OK;
}

void ff_plan_group_destroy(ff_plan_group* g) {
  if (!g) return;
  if (g->dev_mem) (void)hipFree(g->dev_mem);
  delete g;
}

ff_status ff_adapter_fwd_group(const ff_plan_group* g, int64_t T, const int32_t* tokens, int act,
                               const void* const* X, int64_t ldx, const float* const* c_vals, float scale, float beta,
                               void* const* Y, int64_t ldy, void* stream) {
  ff::clear_error();
  ff_status st = check_group_call(g, T, act);
  if (st != FF_OK || T == 0) return st;
  if (!X || !Y || !c_vals) return ff::fail(FF_EINVAL, "pointer array is NULL");
  if ((st = check_ld("X", ldx, g->ref->fin->d, act)) != FF_OK) return st;
  if ((st = check_ld("Y", ldy, g->ref->fout->d, act)) != FF_OK) return st;
  return launched(ff::launch_fwd_group(g, act == FF_BF16, (int)T, tokens, X, ldx, c_vals, scale, beta, Y, ldy,
                                       (hipStream_t)stream),
                  "group forward launch");
}

ff_status ff_adapter_bwd_group(const ff_plan_group* g, int64_t T, const int32_t* tokens, int act,
                               const void* const* X, int64_t ldx, const void* const* G, int64_t ldg,
                               const float* const* c_vals, float scale, float beta_dx, void* const* dX, int64_t lddx,
                               int accumulate_dc, float* const* dC, void* stream) {
  ff::clear_error();
  ff_status st = check_group_call(g, T, act);
  if (st != FF_OK) return st;
  const bool want_dx = dX != nullptr, want_dc = dC != nullptr;
  if (!want_dx && !want_dc) return FF_OK;
  if (T == 0 && (!want_dc || accumulate_dc)) return FF_OK;   // empty sums: only an overwritten dC changes
  if (T == 0) {   // dC = 0 for every adapter
    return launched(ff::launch_bwd_group(g, act == FF_BF16, 0, tokens, X, ldx, G, ldg, c_vals, scale, beta_dx,
                                         nullptr, lddx, false, 0, dC, true, (hipStream_t)stream),
                    "group backward launch");
  }
  if (!G) return ff::fail(FF_EINVAL, "G pointer array is NULL");
  if (want_dc && !X) return ff::fail(FF_EINVAL, "X pointer array is NULL");
  if (want_dx && !c_vals) return ff::fail(FF_EINVAL, "c_vals pointer array is NULL");
  if ((st = check_ld("G", ldg, g->ref->fout->d, act)) != FF_OK) return st;
  if (want_dc && (st = check_ld("X", ldx, g->ref->fin->d, act)) != FF_OK) return st;
  if (want_dx && (st = check_ld("dX", lddx, g->ref->fin->d, act)) != FF_OK) return st;
  return launched(ff::launch_bwd_group(g, act == FF_BF16, (int)T, tokens, X, ldx, G, ldg, c_vals, scale, beta_dx, dX,
                                       lddx, want_dx, accumulate_dc, dC, want_dc, (hipStream_t)stream),
                  "group backward launch");
}

}  // extern "C"
