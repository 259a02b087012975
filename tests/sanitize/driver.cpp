// Host-code driver for the sanitizer build (test infrastructure): frame construction, plan
// building, plan groups and the argument checks of the C entry points, against the CPU stand-in
// of hip_host_stub.cpp.  It checks status codes, then runs the whole creation sequence once more
// for every device allocation in it, with that allocation failing: each such run must report
// FF_ENOMEM, leave its output handle NULL and free what it allocated (LeakSanitizer, at exit,
// reports anything left behind, device memory included).  Exit status: the number of failed
// checks (0: all passed).
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <vector>

#include "frameft.h"

extern "C" void stub_fail_malloc_at(long n);
extern "C" long stub_malloc_calls();

static int g_failed = 0;
#define CHECK(cond)                                                                        \
  do {                                                                                     \
    if (!(cond)) {                                                                         \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, ff_last_error()); \
      ++g_failed;                                                                          \
    }                                                                                      \
  } while (0)

namespace {

struct Support {
  std::vector<int32_t> rows, cols;
};

// nnz distinct (row, col) pairs in an m x n grid
Support random_support(int64_t m, int64_t n, int64_t nnz, unsigned seed) {
  std::mt19937_64 g(seed);
  std::set<int64_t> seen;
  Support s;
  while ((int64_t)seen.size() < nnz) {
    const int64_t key = (int64_t)(g() % (uint64_t)(m * n));
    if (seen.insert(key).second) {
      s.rows.push_back((int32_t)(key / n));
      s.cols.push_back((int32_t)(key % n));
    }
  }
  return s;
}

void* dev_buf(size_t bytes) {   // "device" buffers: 256-byte aligned host memory
  void* p = std::aligned_alloc(256, (bytes + 255) / 256 * 256);
  std::memset(p, 0, (bytes + 255) / 256 * 256);
  return p;
}

// (d, k, rho): the 128-wide fused path; a radix-4 single stage; two radix-4 stages; a redundant
// frame with T(x) blocks (the appendix's (6, 3, 11) in real terms); a Llama-width frame with
// d / rho = 42.67
const int64_t kFrames[][3] = {{4096, 64, 64}, {688, 172, 4}, {1024, 512, 2}, {22, 6, 6}, {4096, 48, 96}};

// One frame, a plan on it, calls through the entry points, destruction.  Returns the first
// failing status of a creation call (FF_OK when everything was created).
ff_status run_case(const int64_t* fr, int64_t nnz, bool group) {
  const int64_t d = fr[0], k = fr[1], rho = fr[2], dv = k * rho;
  ff_frame* f = nullptr;
  ff_status st = ff_framegen(d, k, rho, &f);
  if (st != FF_OK) {
    CHECK(f == nullptr);
    return st;
  }
  int64_t qd = 0, qk = 0, qr = 0;
  CHECK(ff_frame_info(f, &qd, &qk, &qr) == FF_OK && qd == d && qk == k && qr == rho);
  std::vector<double> col((size_t)d * 3);
  CHECK(ff_frame_export(f, dv - 3, 3, col.data()) == FF_OK);
  CHECK(ff_frame_export(f, dv - 2, 3, col.data()) == FF_EINVAL);
  const Support s = random_support(dv, dv, nnz, (unsigned)(d + nnz));
  const int64_t T = 40;
  ff_plan* p = nullptr;
  st = ff_plan_create(f, f, nnz, s.rows.data(), s.cols.data(), T, 2, &p);
  if (st != FF_OK) {
    CHECK(p == nullptr);
    ff_frame_destroy(f);
    return st;
  }
  int64_t L = 0;
  CHECK(ff_plan_query(p, FF_Q_COEF_SLOTS, &L) == FF_OK && L >= nnz);
  std::vector<int64_t> order((size_t)L);
  CHECK(ff_plan_order(p, order.data()) == FF_OK);
  std::vector<int> hits((size_t)nnz, 0);
  for (int64_t j = 0; j < L; ++j)
    if (order[j] >= 0 && order[j] < nnz) ++hits[order[j]];
  for (int64_t e = 0; e < nnz; ++e) CHECK(hits[e] == 1);

  // entry points: valid calls succeed; bad arguments are refused before any launch
  const int64_t ld = (d + 7) / 8 * 8;
  float* X = (float*)dev_buf((size_t)T * ld * 4);
  float* Y = (float*)dev_buf((size_t)T * ld * 4);
  float* c = (float*)dev_buf((size_t)L * 4);
  float* dC = (float*)dev_buf((size_t)L * 4);
  CHECK(ff_adapter_fwd(p, T, FF_F32, X, ld, c, 1.f, 0.f, Y, ld, nullptr) == FF_OK);
  CHECK(ff_adapter_fwd(p, T, FF_BF16, X, ld, c, 1.f, 0.f, Y, ld, nullptr) == FF_OK);
  CHECK(ff_adapter_fwd(p, T + 1, FF_F32, X, ld, c, 1.f, 0.f, Y, ld, nullptr) == FF_EINVAL);
  CHECK(ff_adapter_fwd(p, T, FF_F32, X, d - 1, c, 1.f, 0.f, Y, ld, nullptr) == FF_EINVAL);
  CHECK(ff_adapter_fwd(p, T, 7, X, ld, c, 1.f, 0.f, Y, ld, nullptr) == FF_EINVAL);
  CHECK(ff_adapter_bwd(p, T, FF_F32, X, ld, Y, ld, c, 1.f, 0.f, X, ld, 0, dC, nullptr) == FF_OK);
  CHECK(ff_adapter_bwd(p, T, FF_F32, X, ld, Y, ld, nullptr, 1.f, 0.f, nullptr, ld, 0, dC, nullptr) == FF_OK);
  CHECK(ff_adapter_bwd(p, T, FF_F32, X, ld, Y, ld, nullptr, 1.f, 0.f, X, ld, 0, dC, nullptr) == FF_EINVAL);
  CHECK(ff_adapter_bwd(p, 0, FF_F32, nullptr, ld, nullptr, ld, nullptr, 1.f, 0.f, nullptr, ld, 0, dC, nullptr) ==
        FF_OK);
  CHECK(ff_adapter_bwd_noalloc(p, T, FF_BF16, X, ld, Y, ld, c, 1.f, 0.f, X, ld, 0, dC, nullptr) == FF_OK);
  CHECK(ff_merge_delta(p, c, 1.f, FF_BF16, 1.f, Y, d, nullptr) == FF_OK);
  CHECK(ff_merge_delta(p, c, 1.f, FF_F32, 1.f, Y, d - 1, nullptr) == FF_EINVAL);
  CHECK(ff_coef_to_plan(p, dC, c, nullptr) == FF_OK);
  CHECK(ff_coef_to_user(p, c, dC, 1, nullptr) == FF_OK);
  CHECK(ff_coef_to_plan(p, c, c, nullptr) == FF_EINVAL);   // overlapping arrays
  const bool lifted = dv != d;
  const void* const* ptrs = (const void* const*)dev_buf(64);
  CHECK(ff_adapter_fwd_batched(p, 2, T, FF_F32, ptrs, ld, (const float* const*)ptrs, 1.f, 0.f, (void* const*)ptrs,
                               ld, nullptr) == (lifted ? FF_EUNSUPPORTED : FF_OK));
  CHECK(ff_adapter_fwd_batched(p, 3, T, FF_F32, ptrs, ld, (const float* const*)ptrs, 1.f, 0.f, (void* const*)ptrs,
                               ld, nullptr) == FF_EINVAL);

  if (group) {   // two supports over the frame pair
    const Support s2 = random_support(dv, dv, nnz, (unsigned)(d + nnz + 1));
    ff_plan* p2 = nullptr;
    st = ff_plan_create(f, f, nnz, s2.rows.data(), s2.cols.data(), T, 1, &p2);
    if (st == FF_OK) {
      const ff_plan* plans[2] = {p, p2};
      ff_plan_group* g = nullptr;
      st = ff_plan_group_create(2, plans, &g);
      if (st == FF_OK) {
        CHECK(!lifted);
        CHECK(ff_adapter_fwd_group(g, T, nullptr, FF_BF16, ptrs, ld, (const float* const*)ptrs, 1.f, 0.f,
                                   (void* const*)ptrs, ld, nullptr) == FF_OK);
        CHECK(ff_adapter_fwd_group(g, T + 1, nullptr, FF_BF16, ptrs, ld, (const float* const*)ptrs, 1.f, 0.f,
                                   (void* const*)ptrs, ld, nullptr) == FF_EINVAL);
        ff_plan_group_destroy(g);
      } else {
        CHECK(g == nullptr);
        if (lifted && st == FF_EUNSUPPORTED) st = FF_OK;   // groups do not take lifted frames
      }
      const ff_plan* twice[2] = {p, p};
      ff_plan_group* g2 = nullptr;
      CHECK(ff_plan_group_create(2, twice, &g2) != FF_OK && g2 == nullptr);
      ff_plan_destroy(p2);
    } else {
      CHECK(p2 == nullptr);
    }
  }
  std::free(X);
  std::free(Y);
  std::free(c);
  std::free(dC);
  std::free((void*)ptrs);
  ff_plan_destroy(p);
  ff_frame_destroy(f);
  return st;
}

}  // namespace

int main() {
  // host frames: values of a redundant frame, invalid requests
  std::vector<double> P(22 * 36);
  CHECK(ff_tff_host(22, 6, 6, 0, 36, P.data()) == FF_OK);
  double norm2 = 0;
  for (double x : P) norm2 += x * x;
  CHECK(std::abs(norm2 - 22.0) < 1e-9);   // Parseval: ||P||_F^2 = trace(P P^T) = d
  CHECK(ff_tff_host(22, 4, 6, 0, 1, P.data()) == FF_ENOTFF);
  CHECK(ff_tff_host(21, 6, 6, 0, 1, P.data()) == FF_EINVAL);
  CHECK(ff_tff_host(22, 6, 6, 30, 7, P.data()) == FF_EINVAL);
  CHECK(ff_tff_host(22, 6, 6, 0, 1, nullptr) == FF_EINVAL);

  // frame and plan argument checks
  ff_frame* f = reinterpret_cast<ff_frame*>(1);
  CHECK(ff_framegen(22, 7, 6, &f) == FF_EUNSUPPORTED && f == nullptr);
  CHECK(ff_framegen(10, 2, 4, &f) == FF_ENOTFF && f == nullptr);
  CHECK(ff_framegen(256, 16, 16, nullptr) == FF_EINVAL);
  CHECK(ff_framegen(256, 16, 16, &f) == FF_OK);
  {
    ff_plan* p = reinterpret_cast<ff_plan*>(1);
    const int32_t r2[2] = {3, 3}, c2[2] = {5, 5}, rb[1] = {256}, cb[1] = {0};
    CHECK(ff_plan_create(f, f, 2, r2, c2, 8, 1, &p) == FF_EINVAL && p == nullptr);   // duplicate entry
    CHECK(ff_plan_create(f, f, 1, rb, cb, 8, 1, &p) == FF_EINVAL && p == nullptr);   // row out of range
    CHECK(ff_plan_create(f, f, 1, nullptr, cb, 8, 1, &p) == FF_EINVAL);
    CHECK(ff_plan_create(f, f, 0, nullptr, nullptr, 8, 0, &p) == FF_EINVAL);        // max_batch 0
    CHECK(ff_plan_create(f, f, 0, nullptr, nullptr, 8, 1, &p) == FF_OK);            // empty support
    ff_plan_destroy(p);
  }
  ff_frame_destroy(f);

  // every frame kind, with and without groups
  for (const auto& fr : kFrames) CHECK(run_case(fr, 300, true) == FF_OK);

  // each device allocation of each sequence, failing in turn
  long injected = 0;
  for (const auto& fr : kFrames) {
    stub_fail_malloc_at(0);
    CHECK(run_case(fr, 300, true) == FF_OK);
    const long n = stub_malloc_calls();
    CHECK(n >= 2);
    for (long i = 1; i <= n; ++i) {
      stub_fail_malloc_at(i);
      CHECK(run_case(fr, 300, true) == FF_ENOMEM);
      ++injected;
    }
  }
  stub_fail_malloc_at(0);
  std::printf("allocation failures injected: %ld\n", injected);
  std::printf("host driver: %d failed checks\n", g_failed);
  return g_failed;
}
