// Frames with k rho != d (Sec. 3.2 construction, appendix "Fusion Frames Construction: an
// example", whose (6, 3, 11) frame is redundant and whose rows end in the T(x) blocks): P = L^T Pv,
// Pv the block frame of the coefficient-space dimension k rho and L the sparse lift of the
// Spectral Tetris rows (LiftDev).  A call lifts its inputs into fp32 rows of width k rho (each
// output element is one product F[r][j] x_j, rounded once), runs the block-frame kernels on them
// in fp32 and lifts the results back (each user coordinate sums at most two weighted virtual
// values, then beta times the old value, then one rounding to the caller's type).
#include <algorithm>

#include "ff_internal.h"

namespace ff {
namespace {

using u16 = unsigned short;

__device__ __forceinline__ float bf16_to_f(u16 h) { return __uint_as_float((unsigned)h << 16); }
__device__ __forceinline__ u16 f_to_bf16(float f) {   // round to nearest even; NaN stays NaN
  const unsigned u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u16)((u >> 16) | 0x40u);
  return (u16)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

constexpr int kLiftThreads = 256;
constexpr long kLiftMaxBlocks = 65536;

// Xt[t][2 v + q] = w[v] X[t][2 src[v] + q] (zero where src[v] < 0), t < T, v < dvc.
template <bool BF16>
__global__ void __launch_bounds__(kLiftThreads) lift_up(const void* __restrict__ X, long ldx, float* __restrict__ Xt,
                                                        long ldt, long T, int dvc, const int* __restrict__ src,
                                                        const float* __restrict__ w) {
  const long n = T * dvc;
  for (long e = (long)blockIdx.x * kLiftThreads + threadIdx.x; e < n; e += (long)gridDim.x * kLiftThreads) {
    const long t = e / dvc;
    const int v = (int)(e - t * dvc);
    const int j = src[v];
    float2 r = make_float2(0.f, 0.f);
    if (j >= 0) {
      const float a = w[v];
      if constexpr (BF16) {
        const u16* x = static_cast<const u16*>(X) + t * ldx + 2 * (long)j;
        r = make_float2(a * bf16_to_f(x[0]), a * bf16_to_f(x[1]));
      } else {
        const float* x = static_cast<const float*>(X) + t * ldx + 2 * (long)j;
        r = make_float2(a * x[0], a * x[1]);
      }
    }
    *reinterpret_cast<float2*>(Xt + t * ldt + 2 * (long)v) = r;
  }
}

// Y[t][2 j + q] = beta Y[t][2 j + q] + w0 Yt[t][2 v0 + q] + w1 Yt[t][2 v1 + q] over the (one or two)
// virtual coordinates v0, v1 of user coordinate j; Y is not read when beta == 0.
template <bool BF16>
__global__ void __launch_bounds__(kLiftThreads) lift_down(const float* __restrict__ Yt, long ldt, void* __restrict__ Y,
                                                          long ldy, long T, int dc, const int2* __restrict__ vv,
                                                          const float2* __restrict__ ww, float beta) {
  const long n = T * dc;
  for (long e = (long)blockIdx.x * kLiftThreads + threadIdx.x; e < n; e += (long)gridDim.x * kLiftThreads) {
    const long t = e / dc;
    const int j = (int)(e - t * dc);
    const int2 v = vv[j];
    const float2 w = ww[j];
    const float2 a = *reinterpret_cast<const float2*>(Yt + t * ldt + 2 * (long)v.x);
    float r0 = w.x * a.x, r1 = w.x * a.y;
    if (v.y >= 0) {
      const float2 b = *reinterpret_cast<const float2*>(Yt + t * ldt + 2 * (long)v.y);
      r0 = fmaf(w.y, b.x, r0);
      r1 = fmaf(w.y, b.y, r1);
    }
    if constexpr (BF16) {
      u16* y = static_cast<u16*>(Y) + t * ldy + 2 * (long)j;
      if (beta != 0.f) {
        r0 = fmaf(beta, bf16_to_f(y[0]), r0);
        r1 = fmaf(beta, bf16_to_f(y[1]), r1);
      }
      y[0] = f_to_bf16(r0);
      y[1] = f_to_bf16(r1);
    } else {
      float* y = static_cast<float*>(Y) + t * ldy + 2 * (long)j;
      if (beta != 0.f) {
        r0 = fmaf(beta, y[0], r0);
        r1 = fmaf(beta, y[1], r1);
      }
      y[0] = r0;
      y[1] = r1;
    }
  }
}

// Row `row` of Gt = the lift of the unit vector e_(row0 + row) of the output space: entry 2 v + q
// is w[v] where virtual coordinate v is fed by the unit's complex coordinate and q is its part.
__global__ void __launch_bounds__(kLiftThreads) lift_units(float* __restrict__ Gt, int rows, int row0, int dvc,
                                                           const int* __restrict__ src, const float* __restrict__ w) {
  const long n = (long)rows * dvc;
  for (long e = (long)blockIdx.x * kLiftThreads + threadIdx.x; e < n; e += (long)gridDim.x * kLiftThreads) {
    const int row = (int)(e / dvc), v = (int)(e - (long)row * dvc);
    const int i = row0 + row, j = src[v];
    float2 r = make_float2(0.f, 0.f);
    if (j == (i >> 1)) {
      if (i & 1)
        r.y = w[v];
      else
        r.x = w[v];
    }
    *reinterpret_cast<float2*>(Gt + (long)row * 2 * dvc + 2 * (long)v) = r;
  }
}

unsigned blocks_for(long n) {
  return (unsigned)std::max<long>(1, std::min<long>((n + kLiftThreads - 1) / kLiftThreads, kLiftMaxBlocks));
}

hipError_t up(const ff_frame* f, int bf16, long T, const void* X, int64_t ldx, float* Xt, hipStream_t s) {
  const LiftDev& L = f->lift;
  const unsigned nb = blocks_for(T * L.dvc);
  if (bf16)
    hipLaunchKernelGGL(lift_up<true>, dim3(nb), dim3(kLiftThreads), 0, s, X, (long)ldx, Xt, (long)f->dv, T, L.dvc,
                       L.up_src, L.up_w);
  else
    hipLaunchKernelGGL(lift_up<false>, dim3(nb), dim3(kLiftThreads), 0, s, X, (long)ldx, Xt, (long)f->dv, T, L.dvc,
                       L.up_src, L.up_w);
  return hipGetLastError();
}

hipError_t down(const ff_frame* f, int bf16, long T, const float* Yt, void* Y, int64_t ldy, float beta,
                hipStream_t s) {
  const LiftDev& L = f->lift;
  const unsigned nb = blocks_for(T * L.dc);
  if (bf16)
    hipLaunchKernelGGL(lift_down<true>, dim3(nb), dim3(kLiftThreads), 0, s, Yt, (long)f->dv, Y, (long)ldy, T, L.dc,
                       L.dn_v, L.dn_w, beta);
  else
    hipLaunchKernelGGL(lift_down<false>, dim3(nb), dim3(kLiftThreads), 0, s, Yt, (long)f->dv, Y, (long)ldy, T, L.dc,
                       L.dn_v, L.dn_w, beta);
  return hipGetLastError();
}

void record(hipEvent_t ev, hipStream_t s) {
  if (ev) (void)hipEventRecord(ev, s);
}

}  // namespace

hipError_t launch_fwd_lifted(const ff_plan* p, int bf16, int T, const void* X, int64_t ldx, const float* c,
                             float scale, float beta, void* Y, int64_t ldy, hipStream_t s) {
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  hipError_t e = up(p->fin, bf16, T, X, ldx, p->lift_x, s);
  if (e == hipSuccess)
    e = launch_fwd(p, 0, 1, T, {p->lift_x, nullptr}, p->fin->dv, c, nullptr, scale, 0.f, {p->lift_g, nullptr},
                   p->fout->dv, nullptr, s);
  if (e == hipSuccess) e = down(p->fout, bf16, T, p->lift_g, Y, ldy, beta, s);
  record(e1, s);
  return e;
}

hipError_t launch_bwd_lifted(const ff_plan* p, int bf16, int T, const void* X, int64_t ldx, const void* G,
                             int64_t ldg, const float* c, float scale, float beta_dx, void* dX, int64_t lddx,
                             bool want_dx, int accumulate_dc, float* dC, bool want_dc, hipStream_t s,
                             const BwdScratch* ws) {
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  hipError_t e = hipSuccess;
  if (T > 0 && (want_dx || want_dc)) {
    e = up(p->fout, bf16, T, G, ldg, p->lift_g, s);
    if (e == hipSuccess && want_dc) e = up(p->fin, bf16, T, X, ldx, p->lift_x, s);
  }
  if (e == hipSuccess)
    e = launch_bwd(p, 0, 1, T, {want_dc ? p->lift_x : nullptr, nullptr}, p->fin->dv, {p->lift_g, nullptr},
                   p->fout->dv, c, nullptr, scale, 0.f, {p->lift_dx, nullptr}, p->fin->dv, want_dx, accumulate_dc, dC,
                   nullptr, want_dc, nullptr, s, ws);
  if (e == hipSuccess && T > 0 && want_dx) e = down(p->fin, bf16, T, p->lift_dx, dX, lddx, beta_dx, s);
  record(e1, s);
  return e;
}

// Row i of P_out C P_in^T is (P_in C^T P_out^T e_i)^T: the backward (dX only) of the unit vectors
// of the output space, mrg_rows at a time, each lifted directly into the staging rows.
hipError_t launch_merge_lifted(const ff_plan* p, const float* c, float scale, int w_bf16, float beta, void* W,
                               int64_t ldw, hipStream_t s) {
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  const int m = (int)p->fout->d, R = p->mrg_rows;
  const size_t esz = w_bf16 ? 2 : 4;
  hipError_t e = hipSuccess;
  for (int row0 = 0; row0 < m && e == hipSuccess; row0 += R) {
    const int rows = std::min(R, m - row0);
    const LiftDev& Lo = p->fout->lift;
    hipLaunchKernelGGL(lift_units, dim3(blocks_for((long)rows * Lo.dvc)), dim3(kLiftThreads), 0, s, p->mrg_g, rows,
                       row0, Lo.dvc, Lo.up_src, Lo.up_w);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = launch_bwd(p, 0, 1, rows, {nullptr, nullptr}, p->fin->dv, {p->mrg_g, nullptr}, p->fout->dv, c, nullptr,
                     scale, 0.f, {p->mrg_out, nullptr}, p->fin->dv, true, 0, nullptr, nullptr, false, nullptr, s);
    if (e == hipSuccess)
      e = down(p->fin, w_bf16, rows, p->mrg_out, static_cast<char*>(W) + (size_t)row0 * (size_t)ldw * esz, ldw, beta,
               s);
  }
  record(e1, s);
  return e;
}

}  // namespace ff
