// Frame generation (Algorithm 1, step 2): the real (k, rho, d) tight fusion
// frame of Sec. 3.2, built on the host in fp64 and placed on the device as
// MFMA fragments of its diagonal block.
//
// Construction (appendix "Fusion Frames Construction: an example"):
//   1. Spectral Tetris: a unit-norm tight frame F of d_c = d/2 vectors in
//      C^{rho_c}, rho_c = rho/2.  Each row must reach squared norm d_c/rho_c;
//      it is filled with ones while a whole unit is missing, and a leftover x in
//      (0,1) is placed by the 2x2 block T(x) = [[sqrt(x/2), sqrt(x/2)],
//      [sqrt((2-x)/2), -sqrt((2-x)/2)]] whose lower row starts the next row.
//      Norms are kept as integer multiples of 1/rho_c, so every comparison is
//      exact.
//   2. Modulation: vector (i, r) = row r of F times (e^{2 pi i i j / k})_j,
//      scaled by 1/sqrt(k) (Parseval normalisation).
//   3. Real extension x + iy -> [[x, -y], [y, x]].
// Column order is canonical: i*rho + 2r + s.
//
// When k*rho = d every row of F is k consecutive ones, so P is block diagonal
// with rho/2 identical square blocks B (2k x 2k): B[2 tau + t][2 i + s] is the
// entry of column (i, r, s) at real row 2(r k + tau) + t.  The device works on
// B alone.  Any other tight (k, rho, d) -- redundant frames, k rho > d, and
// those with a non-integer d / rho -- factors as P = L^T Pv: Pv is the block
// frame of dimension k rho, and the sparse lift L places each row of F at the
// positions j mod k of its block with the row's weights (modulation depends on
// j only mod k, and tightness keeps a row's columns distinct mod k).
#include <algorithm>
#include <cmath>
#include <complex>
#include <cstring>
#include <map>
#include <utility>

#include "ff_internal.h"

namespace {

struct TetrisEntry {
  int64_t r;   // row of F
  int64_t j;   // column of F
  double v;
};

// Spectral Tetris F (rho_c x d_c) as a list of nonzeros in column order.
ff_status spectral_tetris(int64_t rho_c, int64_t d_c, std::vector<TetrisEntry>& F) {
  if (rho_c < 1 || d_c < rho_c)
    return ff::fail(FF_ENOTFF, "Spectral Tetris needs d/2 >= rho/2 >= 1 (rho_c=%lld, d_c=%lld)",
                    (long long)rho_c, (long long)d_c);
  F.clear();
  const int64_t unit = rho_c;      // one unit of squared norm, in units of 1/rho_c
  const int64_t target = d_c;      // squared row norm d_c/rho_c, in units of 1/rho_c
  int64_t col = 0, carried = 0;
  for (int64_t r = 0; r < rho_c; ++r) {
    int64_t missing = target - carried;
    if (missing < 0)
      return ff::fail(FF_ENOTFF, "Spectral Tetris: row %lld overfilled", (long long)r);
    while (missing >= unit) {
      if (col >= d_c) return ff::fail(FF_ENOTFF, "Spectral Tetris ran out of columns");
      F.push_back({r, col, 1.0});
      ++col;
      missing -= unit;
    }
    if (missing > 0) {
      if (r + 1 >= rho_c || col + 2 > d_c)
        return ff::fail(FF_ENOTFF, "Spectral Tetris: leftover norm in the last row");
      // x = missing/rho_c; entries sqrt(x/2) and sqrt((2-x)/2), each ratio rounded once.
      const double a = std::sqrt((double)missing / (double)(2 * rho_c));
      const double b = std::sqrt((double)(2 * unit - missing) / (double)(2 * rho_c));
      F.push_back({r, col, a});
      F.push_back({r + 1, col, b});
      F.push_back({r, col + 1, a});
      F.push_back({r + 1, col + 1, -b});
      col += 2;
      carried = 2 * unit - missing;
    } else {
      carried = 0;
    }
  }
  if (col != d_c) return ff::fail(FF_ENOTFF, "Spectral Tetris filled %lld of %lld columns",
                                  (long long)col, (long long)d_c);
  return FF_OK;
}

// Tightness of the modulated frame: F's columns j != j' with j = j' (mod k)
// must be orthogonal (the roots-of-unity sum removes every other pair).
ff_status check_tight(const std::vector<TetrisEntry>& F, int64_t k) {
  std::map<int64_t, std::vector<std::pair<int64_t, double>>> by_row;
  for (const auto& e : F) by_row[e.r].push_back({e.j, e.v});
  std::map<std::pair<int64_t, int64_t>, double> ip;
  for (const auto& kv : by_row) {
    const auto& cols = kv.second;
    for (size_t a = 0; a < cols.size(); ++a)
      for (size_t b = a + 1; b < cols.size(); ++b)
        if ((cols[a].first - cols[b].first) % k == 0)
          ip[{cols[a].first, cols[b].first}] += cols[a].second * cols[b].second;
  }
  for (const auto& kv : ip)
    if (std::fabs(kv.second) > 1e-12)
      return ff::fail(FF_ENOTFF, "columns %lld and %lld of F are not orthogonal: not a tight frame",
                      (long long)kv.first.first, (long long)kv.first.second);
  return FF_OK;
}

// Nonzeros of real column c (canonical index) of P: (real row, value).
void real_column(const std::vector<std::vector<std::pair<int64_t, double>>>& Frows, int64_t k,
                 int64_t rho, int64_t c, std::vector<std::pair<int64_t, double>>& out) {
  out.clear();
  const int64_t i = c / rho, rem = c % rho, r = rem / 2, s = rem % 2;
  const double sqrt_k = std::sqrt((double)k);
  for (const auto& jv : Frows[r]) {
    const int64_t j = jv.first;
    const int64_t m = (i * j) % k;                    // exponent reduced mod k
    const double theta = (2.0 * M_PI * (double)m) / (double)k;
    const double re = (jv.second * std::cos(theta)) / sqrt_k;
    const double im = (jv.second * std::sin(theta)) / sqrt_k;
    if (s == 0) {          // [Re; Im]
      out.push_back({2 * j, re});
      out.push_back({2 * j + 1, im});
    } else {               // [-Im; Re]
      out.push_back({2 * j, -im});
      out.push_back({2 * j + 1, re});
    }
  }
}

ff_status build_host(int64_t d, int64_t k, int64_t rho,
                     std::vector<std::vector<std::pair<int64_t, double>>>& Frows) {
  if (d < 2 || rho < 2 || k < 1 || (d % 2) || (rho % 2))
    return ff::fail(FF_EINVAL, "need k >= 1 and even d, rho >= 2 (d=%lld, k=%lld, rho=%lld)",
                    (long long)d, (long long)k, (long long)rho);
  if (d > (int64_t)1 << 24 || k * rho > (int64_t)1 << 26)
    return ff::fail(FF_EINVAL, "frame too large");
  std::vector<TetrisEntry> F;
  ff_status st = spectral_tetris(rho / 2, d / 2, F);
  if (st != FF_OK) return st;
  st = check_tight(F, k);
  if (st != FF_OK) return st;
  Frows.assign(rho / 2, {});
  for (const auto& e : F) Frows[e.r].push_back({e.j, e.v});
  return FF_OK;
}

// S-stage radix-4 factorization (S >= 2) of the realified DFT block of size k = 4^S k2, as the
// generic kernels apply it: the input index is b + sum_t a_t K_t (K_t = k / 4^t, b < k2), the
// stages are decimation in frequency (stage t: y_a' = w_k^(-a' n 4^(t-1)) sum_a v_a (-i)^(a a'),
// n the index left in the parent sequence), and the 4^S sequences of length k2 then get the dense
// k2-point DFT (M2, with the 1/sqrt(k) of the unitary transform).  Frequency
// i = a_1' + 4 a_2' + ... + 4^(S-1) a_S' + 4^S l.  twk holds (cos, sin) of 2 pi j / k, j < k.
// Checked against B on every unit vector, both directions (a unit input reaches one residue b).
bool factor_multistage(const std::vector<double>& B, int64_t k, int S, std::vector<double>& M2,
                       std::vector<double>& twk) {
  int64_t n4 = 1;
  for (int t = 0; t < S; ++t) n4 *= 4;
  if (k % n4 != 0) return false;
  const int64_t k2 = k / n4, W = 2 * k, W2 = 2 * k2;
  const double isk = 1.0 / std::sqrt((double)k);
  M2.assign((size_t)(W2 * W2), 0.0);
  for (int64_t l = 0; l < k2; ++l)
    for (int64_t b = 0; b < k2; ++b) {
      const double th = 2.0 * M_PI * (double)((b * l) % k2) / (double)k2;
      const double re = std::cos(th) * isk, im = -std::sin(th) * isk;
      M2[(2 * l) * W2 + 2 * b] = re;
      M2[(2 * l) * W2 + 2 * b + 1] = -im;
      M2[(2 * l + 1) * W2 + 2 * b] = im;
      M2[(2 * l + 1) * W2 + 2 * b + 1] = re;
    }
  twk.assign((size_t)(2 * k), 0.0);
  for (int64_t j = 0; j < k; ++j) {
    const double ph = 2.0 * M_PI * (double)j / (double)k;
    twk[2 * j] = std::cos(ph);
    twk[2 * j + 1] = std::sin(ph);
  }
  typedef std::complex<double> cx;
  const cx mpow[4] = {cx(1, 0), cx(0, -1), cx(-1, 0), cx(0, 1)};   // (-i)^e
  const cx ppow[4] = {cx(1, 0), cx(0, 1), cx(-1, 0), cx(0, -1)};    // i^e
  // the stages on one residue's 4^S values, forward (analysis) or adjoint (synthesis)
  auto stages = [&](std::vector<cx>& v, int64_t b, bool adjoint) {
    for (int tt = 0; tt < S; ++tt) {
      const int t = adjoint ? S - tt : tt + 1;
      int64_t st = 1;
      for (int q = t; q < S; ++q) st *= 4;
      int64_t tws = 1;
      for (int q = 1; q < t; ++q) tws *= 4;
      for (int64_t hi = 0; hi < n4 / (4 * st); ++hi)
        for (int64_t lo = 0; lo < st; ++lo) {
          const int64_t base = hi * 4 * st + lo, n = b + k2 * lo;
          cx in[4], out[4];
          for (int a = 0; a < 4; ++a) in[a] = v[base + a * st];
          auto w = [&](int64_t a) {   // w_k^(a n 4^(t-1))
            const int64_t j = (a * n * tws) % k;
            return cx(twk[2 * j], twk[2 * j + 1]);
          };
          for (int o = 0; o < 4; ++o) {
            cx acc(0.0, 0.0);
            if (!adjoint) {   // out_a' = conj(w^a') sum_a (-i)^(a a') in_a
              for (int a = 0; a < 4; ++a) acc += in[a] * mpow[(a * o) % 4];
              acc *= std::conj(w(o));
            } else {          // out_a = sum_a' i^(a a') w^a' in_a'
              for (int a = 0; a < 4; ++a) acc += in[a] * w(a) * ppow[(a * o) % 4];
            }
            out[o] = acc;
          }
          for (int a = 0; a < 4; ++a) v[base + a * st] = out[a];
        }
    }
  };
  auto col_of = [&](int64_t i) {   // base-4 digit reversal of i mod 4^S
    int64_t r = i, col = 0;
    for (int t = 0; t < S; ++t) {
      col = 4 * col + (r & 3);
      r >>= 2;
    }
    return std::make_pair(col, r);
  };
  std::vector<cx> v((size_t)n4);
  // analysis of every unit vector e_u against row u of B
  for (int64_t u = 0; u < W; ++u) {
    const int64_t tau = u / 2, b = tau % k2, j0 = tau / k2;
    std::fill(v.begin(), v.end(), cx(0.0, 0.0));
    v[(size_t)j0] = (u & 1) ? cx(0.0, 1.0) : cx(1.0, 0.0);
    stages(v, b, false);
    double err = 0.0;
    for (int64_t c = 0; c < W; ++c) {
      const auto cl = col_of(c >> 1);
      const int64_t o = 2 * cl.second + (c & 1);
      const cx y = v[(size_t)cl.first];
      const double z = M2[o * W2 + 2 * b] * y.real() + M2[o * W2 + 2 * b + 1] * y.imag();
      err = std::max(err, std::fabs(z - B[u * W + c]));
    }
    if (err > 1e-12) return false;
  }
  // synthesis of every unit coefficient e_c against column c of B
  for (int64_t c = 0; c < W; ++c) {
    const auto cl = col_of(c >> 1);
    const int64_t o = 2 * cl.second + (c & 1);
    double err = 0.0;
    for (int64_t b = 0; b < k2; ++b) {
      std::fill(v.begin(), v.end(), cx(0.0, 0.0));
      v[(size_t)cl.first] = cx(M2[o * W2 + 2 * b], M2[o * W2 + 2 * b + 1]);   // row o of M2 = column of M2^T
      stages(v, b, true);
      for (int64_t j = 0; j < n4; ++j) {
        const int64_t u = 2 * (b + k2 * j);
        err = std::max(err, std::fabs(v[(size_t)j].real() - B[u * W + c]));
        err = std::max(err, std::fabs(v[(size_t)j].imag() - B[(u + 1) * W + c]));
      }
    }
    if (err > 1e-12) return false;
  }
  return true;
}

// Radix-4 factorization of the block (Sec. 3.2 modulation: with k*rho = d the block B is the
// realified unitary DFT of size k, analysis z = B^T x being the forward transform with 1/sqrt(k)).
// For k = 4 k2 and input index tau = a k2 + b, frequency i = a' + 4 l:
//   analysis   Y_a'[b] = w^(-a' b) sum_a X[a k2 + b] (-i)^(a a'),   w = e^(2 pi i / k)
//              Z[a' + 4 l] = (1/sqrt(k)) sum_b e^(-2 pi i b l / k2) Y_a'[b]
//   synthesis  Y'_a'[b] = (1/sqrt(k)) sum_l e^(+2 pi i b l / k2) Z[a' + 4 l]
//              X[a k2 + b] = sum_a' i^(a a') w^(a' b) Y'_a'[b]
// M2 is the realified k2-point matrix of the analysis (W2 x W2, rows 2 l + s, columns 2 b + t);
// synthesis uses its transpose.  tw holds (cos, sin) of 2 pi (a' b mod k) / k.  The factored
// operator is checked against B on every unit vector, in both directions, before it is used.
bool factor_radix4(const std::vector<double>& B, int64_t k, std::vector<double>& M2, std::vector<double>& tw) {
  if (k % 4 != 0 || k < 8) return false;
  const int64_t k2 = k / 4, W = 2 * k, W2 = 2 * k2;
  const double isk = 1.0 / std::sqrt((double)k);
  M2.assign((size_t)(W2 * W2), 0.0);
  for (int64_t l = 0; l < k2; ++l)
    for (int64_t b = 0; b < k2; ++b) {
      const double th = 2.0 * M_PI * (double)((b * l) % k2) / (double)k2;
      const double re = std::cos(th) * isk, im = -std::sin(th) * isk;   // e^(-i th) / sqrt(k)
      M2[(2 * l) * W2 + 2 * b] = re;
      M2[(2 * l) * W2 + 2 * b + 1] = -im;
      M2[(2 * l + 1) * W2 + 2 * b] = im;
      M2[(2 * l + 1) * W2 + 2 * b + 1] = re;
    }
  tw.assign((size_t)(3 * k2 * 2), 0.0);
  for (int64_t a = 1; a < 4; ++a)
    for (int64_t b = 0; b < k2; ++b) {
      const double ph = 2.0 * M_PI * (double)((a * b) % k) / (double)k;
      tw[((a - 1) * k2 + b) * 2] = std::cos(ph);
      tw[((a - 1) * k2 + b) * 2 + 1] = std::sin(ph);
    }
  typedef std::pair<double, double> cx;
  auto mul = [](cx p, cx q) { return cx(p.first * q.first - p.second * q.second, p.first * q.second + p.second * q.first); };
  auto twid = [&](int64_t a, int64_t b, bool conj) {
    if (a == 0) return cx(1.0, 0.0);
    const double c = tw[((a - 1) * k2 + b) * 2], sn = tw[((a - 1) * k2 + b) * 2 + 1];
    return cx(c, conj ? -sn : sn);
  };
  // (-i)^e and i^e
  auto ipow = [](int64_t e, bool neg) {
    static const cx t[4] = {cx(1, 0), cx(0, 1), cx(-1, 0), cx(0, -1)};
    const int64_t r = ((neg ? -e : e) % 4 + 4) % 4;
    return t[r];
  };
  std::vector<double> x((size_t)W), y((size_t)W), z((size_t)W);
  for (int64_t u = 0; u < W; ++u) {
    // analysis of the unit vector e_u against column u of B^T (row u of B)
    std::fill(x.begin(), x.end(), 0.0);
    x[u] = 1.0;
    for (int64_t a2 = 0; a2 < 4; ++a2)
      for (int64_t b = 0; b < k2; ++b) {
        cx acc(0.0, 0.0);
        for (int64_t a = 0; a < 4; ++a) {
          const cx X(x[2 * (a * k2 + b)], x[2 * (a * k2 + b) + 1]);
          const cx t = mul(X, ipow(a * a2, true));
          acc.first += t.first;
          acc.second += t.second;
        }
        acc = mul(acc, twid(a2, b, true));
        y[a2 * W2 + 2 * b] = acc.first;
        y[a2 * W2 + 2 * b + 1] = acc.second;
      }
    double err = 0.0;
    for (int64_t a2 = 0; a2 < 4; ++a2)
      for (int64_t o = 0; o < W2; ++o) {
        double v = 0.0;
        for (int64_t i = 0; i < W2; ++i) v += M2[o * W2 + i] * y[a2 * W2 + i];
        const int64_t freq = a2 + 4 * (o >> 1), c = 2 * freq + (o & 1);
        err = std::max(err, std::fabs(v - B[u * W + c]));
      }
    if (err > 1e-12) return false;
  }
  for (int64_t c = 0; c < W; ++c) {
    // synthesis of the unit coefficient e_c against column c of B
    std::fill(z.begin(), z.end(), 0.0);
    const int64_t freq = c >> 1, a2 = freq & 3, l = freq >> 2;
    z[a2 * W2 + 2 * l + (c & 1)] = 1.0;   // coefficient c at its factored position
    for (int64_t q = 0; q < 4; ++q)
      for (int64_t o = 0; o < W2; ++o) {
        double v = 0.0;
        for (int64_t i = 0; i < W2; ++i) v += M2[i * W2 + o] * z[q * W2 + i];
        y[q * W2 + o] = v;
      }
    double err = 0.0;
    for (int64_t a = 0; a < 4; ++a)
      for (int64_t b = 0; b < k2; ++b) {
        cx acc(0.0, 0.0);
        for (int64_t q = 0; q < 4; ++q) {
          const cx Y = mul(cx(y[q * W2 + 2 * b], y[q * W2 + 2 * b + 1]), twid(q, b, false));
          const cx t = mul(Y, ipow(a * q, false));
          acc.first += t.first;
          acc.second += t.second;
        }
        const int64_t u = 2 * (a * k2 + b);
        err = std::max(err, std::fabs(acc.first - B[u * W + c]));
        err = std::max(err, std::fabs(acc.second - B[(u + 1) * W + c]));
      }
    if (err > 1e-12) return false;
  }
  return true;
}

// The lift of the frame with rows Frows (see LiftDev): row r's entry (j, F[r][j]) goes to virtual
// complex coordinate r k + (j mod k).  Two entries of one row that agree mod k would share a virtual
// coordinate; tightness (check_tight) already excludes that, and it is checked again here.
ff_status build_lift(const std::vector<std::vector<std::pair<int64_t, double>>>& Frows, int64_t k, int64_t d_c,
                     std::vector<int>& up_src, std::vector<float>& up_w, std::vector<int>& dn_v,
                     std::vector<float>& dn_w) {
  const int64_t rho_c = (int64_t)Frows.size(), dvc = rho_c * k;
  up_src.assign((size_t)dvc, -1);
  up_w.assign((size_t)dvc, 0.f);
  dn_v.assign((size_t)(2 * d_c), -1);
  dn_w.assign((size_t)(2 * d_c), 0.f);
  for (int64_t r = 0; r < rho_c; ++r)
    for (const auto& jv : Frows[r]) {
      const int64_t j = jv.first, v = r * k + j % k;
      if (up_src[v] >= 0)
        return ff::fail(FF_ENOTFF, "row %lld of F holds columns %d and %lld, equal mod k=%lld: not a tight frame",
                        (long long)r, up_src[v], (long long)j, (long long)k);
      up_src[v] = (int)j;
      up_w[v] = (float)jv.second;
      const int slot = dn_v[2 * j] < 0 ? 0 : 1;
      if (slot == 1 && dn_v[2 * j + 1] >= 0)
        return ff::fail(FF_ENOTFF, "column %lld of F lies in more than two rows", (long long)j);
      dn_v[2 * j + slot] = (int)v;
      dn_w[2 * j + slot] = (float)jv.second;
    }
  for (int64_t j = 0; j < d_c; ++j)
    if (dn_v[2 * j] < 0) return ff::fail(FF_ENOTFF, "column %lld of F is empty", (long long)j);
  return FF_OK;
}

uint16_t bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;   // NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

}  // namespace

extern "C" ff_status ff_tff_host(int64_t d, int64_t k, int64_t rho, int64_t col0, int64_t ncols,
                                 double* out) {
  ff::clear_error();
  if (!out) return ff::fail(FF_EINVAL, "out is NULL");
  std::vector<std::vector<std::pair<int64_t, double>>> Frows;
  ff_status st = build_host(d, k, rho, Frows);
  if (st != FF_OK) return st;
  if (col0 < 0 || ncols < 0 || col0 + ncols > k * rho)
    return ff::fail(FF_EINVAL, "column range [%lld, %lld) outside [0, %lld)", (long long)col0,
                    (long long)(col0 + ncols), (long long)(k * rho));
  std::memset(out, 0, sizeof(double) * (size_t)d * (size_t)ncols);
  std::vector<std::pair<int64_t, double>> colv;
  for (int64_t c = 0; c < ncols; ++c) {
    real_column(Frows, k, rho, col0 + c, colv);
    for (const auto& rv : colv) out[rv.first * ncols + c] = rv.second;
  }
  return FF_OK;
}

extern "C" ff_status ff_framegen(int64_t d, int64_t k, int64_t rho, ff_frame** out) {
  ff::clear_error();
  if (!out) return ff::fail(FF_EINVAL, "out is NULL");
  *out = nullptr;
  std::vector<std::vector<std::pair<int64_t, double>>> Frows;
  ff_status st = build_host(d, k, rho, Frows);
  if (st != FF_OK) return st;
  // The kernels apply the block-diagonal frame Pv of dimension dv = k rho; a frame with k rho != d
  // (a redundant one, or a non-integer d / rho) is P = L^T Pv with the lift L of its own rows.
  const int64_t dv = k * rho;
  const bool lifted = dv != d;
  std::vector<int> up_src, dn_v;
  std::vector<float> up_w, dn_w;
  std::vector<std::vector<std::pair<int64_t, double>>> Fvrows;
  if (lifted) {
    if (dv > (int64_t)1 << 24) return ff::fail(FF_EUNSUPPORTED, "k rho = %lld too large", (long long)dv);
    if ((st = build_lift(Frows, k, d / 2, up_src, up_w, dn_v, dn_w)) != FF_OK) return st;
    if ((st = build_host(dv, k, rho, Fvrows)) != FF_OK) return st;
  } else {   // the identity lift
    up_src.resize((size_t)(d / 2));
    up_w.assign((size_t)(d / 2), 1.f);
    dn_v.resize((size_t)d);
    dn_w.assign((size_t)d, 0.f);
    for (int64_t j = 0; j < d / 2; ++j) {
      up_src[j] = (int)j;
      dn_v[2 * j] = (int)j;
      dn_v[2 * j + 1] = -1;
      dn_w[2 * j] = 1.f;
    }
  }
  const auto& Fb = lifted ? Fvrows : Frows;
  const int64_t W = 2 * k;
  // Lifted frames run the kernels in fp32, whose 4-element accesses need 2k to be a multiple of 4
  // only (bf16 accesses are of 8); the dense path serves those up to 128 wide.
  const bool narrow_ok = lifted && W % 4 == 0 && W <= 128;
  if (W % 8 != 0 && !narrow_ok)
    return ff::fail(FF_EUNSUPPORTED, "GPU path needs 2k to be a multiple of 8 (or of 4 for k rho != d, 2k <= 128; k=%lld)",
                    (long long)k);
  if (W > 4096) return ff::fail(FF_EUNSUPPORTED, "frame block 2k=%lld too wide (at most 4096)", (long long)W);

  // Extract the diagonal block and confirm that P is block diagonal with identical blocks.
  std::vector<double> B((size_t)(W * W), 0.0);
  std::vector<std::pair<int64_t, double>> colv;
  for (int64_t c = 0; c < k * rho; ++c) {
    const int64_t i = c / rho, rem = c % rho, r = rem / 2, s = rem % 2;
    const int64_t lc = 2 * i + s;
    real_column(Fb, k, rho, c, colv);
    for (const auto& rv : colv) {
      const int64_t u = rv.first - r * W;
      if (u < 0 || u >= W)
        return ff::fail(FF_EUNSUPPORTED, "frame is not block diagonal (column %lld)", (long long)c);
      if (r == 0) {
        B[u * W + lc] = rv.second;
      } else if (B[u * W + lc] != rv.second) {
        return ff::fail(FF_EUNSUPPORTED, "frame blocks differ (column %lld)", (long long)c);
      }
    }
  }

  // The realified DFT block satisfies B^T = D B D (D flips odd coordinates); the 128-wide
  // kernels rely on it to apply P^T with the fragments of P.  Checked exactly here.
  bool sign_flip = true;
  for (int64_t r = 0; r < W && sign_flip; ++r)
    for (int64_t c = 0; c < W; ++c)
      if (B[c * W + r] != (((r + c) & 1) ? -B[r * W + c] : B[r * W + c])) {
        sign_flip = false;
        break;
      }

  // The modulation by roots of unity makes the lower half of the block the upper half with
  // the odd complex columns negated: B[u + W/2][c] = (-1)^(c/2) B[u][c] (the row-wise radix-2
  // symmetry of the DFT).  The 128-wide kernels hold only the upper half.  Checked to within
  // the rounding of the cosines, far below bf16 resolution.
  bool half_shift = W % 4 == 0;
  for (int64_t u = 0; u < W / 2 && half_shift; ++u)
    for (int64_t c = 0; c < W; ++c) {
      const double top = B[u * W + c], bot = B[(u + W / 2) * W + c];
      if (std::fabs(bot - (((c >> 1) & 1) ? -top : top)) > 1e-12) {
        half_shift = false;
        break;
      }
    }

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ff::fail(FF_EDEVICE, "no HIP device");
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return ff::fail(FF_EDEVICE, "no HIP device");

  // Blocks wider than 128 are applied in factored form when the radix-4 split reproduces them:
  // one stage up to 512 wide, beyond that 2 or 3 stages leaving a DFT of at most 64 points.
  std::vector<double> M2, tw, twk;
  int nst = 0;
  if (W > 128 && W / 4 <= 128 && factor_radix4(B, k, M2, tw)) {
    nst = 1;
  } else if (W > 512) {
    for (int S = 2; S <= 3 && nst == 0; ++S) {
      const int64_t n4 = (int64_t)1 << (2 * S);
      if (k % n4 == 0 && k / n4 <= 64 && factor_multistage(B, k, S, M2, twk)) nst = S;
    }
    if (nst == 0)
      return ff::fail(FF_EUNSUPPORTED, "frame block 2k=%lld: k is not 4^S k2 with S <= 3 and k2 <= 64",
                      (long long)W);
  }
  const bool factored = nst > 0;
  const int64_t n4 = factored ? (int64_t)1 << (2 * nst) : 1;

  ff::FrameDev fd{};
  fd.d = (int)dv;
  fd.W = (int)W;
  fd.nblk = (int)(rho / 2);
  fd.radix = factored ? 4 : 1;
  fd.nst = nst;
  fd.ncol = (int)n4;
  fd.k2 = factored ? (int)(k / n4) : (int)k;
  fd.W2 = factored ? (int)(W / n4) : (int)W;
  fd.cs = (fd.W2 + 7) / 8 * 8;
  const int64_t W2 = fd.W2;
  fd.MT = (int)((W2 + 15) / 16);
  fd.KT = (int)((W2 + 31) / 32);
  fd.KT4 = (int)((W2 + 15) / 16);
  const size_t n16 = (size_t)fd.MT * fd.KT * 64 * 8;     // bf16 elements per fragment set
  const size_t n32 = (size_t)fd.MT * fd.KT4 * 64 * 4;    // fp32 elements per fragment set
  std::vector<uint16_t> fa16(n16, 0), fs16(n16, 0);
  std::vector<float> fa32(n32, 0.f), fs32(n32, 0.f), B32((size_t)(W * W));
  // analysis computes out[c] = sum_u B[u][c] in[u]  (matrix M_a[o][i] = B[i][o]);
  // synthesis computes out[u] = sum_c B[u][c] in[c] (matrix M_s[o][i] = B[o][i]).
  // Factored: M_a = M2 and M_s = M2^T.
  auto Ma = [&](int64_t o, int64_t i) {
    if (o >= W2 || i >= W2) return 0.0;
    return factored ? M2[o * W2 + i] : B[i * W + o];
  };
  auto Ms = [&](int64_t o, int64_t i) {
    if (o >= W2 || i >= W2) return 0.0;
    return factored ? M2[i * W2 + o] : B[o * W + i];
  };
  for (int mt = 0; mt < fd.MT; ++mt)
    for (int lane = 0; lane < 64; ++lane) {
      const int64_t o = 16 * mt + (lane & 15), q = lane >> 4;
      for (int ks = 0; ks < fd.KT; ++ks)
        for (int j = 0; j < 8; ++j) {
          const size_t idx = (((size_t)mt * fd.KT + ks) * 64 + lane) * 8 + j;
          const int64_t i = 32 * ks + 8 * q + j;
          fa16[idx] = bf16_rne((float)Ma(o, i));
          fs16[idx] = bf16_rne((float)Ms(o, i));
        }
      for (int ks = 0; ks < fd.KT4; ++ks)
        for (int j = 0; j < 4; ++j) {
          const size_t idx = (((size_t)mt * fd.KT4 + ks) * 64 + lane) * 4 + j;
          const int64_t i = 16 * ks + 4 * q + j;
          fa32[idx] = (float)Ma(o, i);
          fs32[idx] = (float)Ms(o, i);
        }
    }
  for (size_t e = 0; e < B32.size(); ++e) B32[e] = (float)B[e];
  // the transposed block for the merge (a column of B is then a contiguous row)
  std::vector<float> Bt32((size_t)(W * W));
  for (int64_t u = 0; u < W; ++u)
    for (int64_t c = 0; c < W; ++c) Bt32[c * W + u] = (float)B[u * W + c];

  std::vector<float> tw32(std::max<size_t>(tw.size(), 2)), twk32(std::max<size_t>(twk.size(), 2));
  for (size_t e = 0; e < tw.size(); ++e) tw32[e] = (float)tw[e];
  for (size_t e = 0; e < twk.size(); ++e) twk32[e] = (float)twk[e];

  const size_t b16 = n16 * 2, b32 = n32 * 4, bB = B32.size() * 4, bT = tw32.size() * 4, bK = twk32.size() * 4;
  const size_t bU = up_src.size() * 4, bD = dn_v.size() * 4, bBt = Bt32.size() * 4;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t total = 2 * up(b16) + 2 * up(b32) + up(bB) + up(bBt) + up(bT) + up(bK) + 2 * up(bU) + 2 * up(bD);
  void* mem = nullptr;
  if (hipMalloc(&mem, total) != hipSuccess) {
    (void)hipGetLastError();
    return ff::fail(FF_ENOMEM, "hipMalloc of %zu bytes for frame failed", total);
  }
  char* p = (char*)mem;
  size_t off = 0;
  auto put = [&](const void* src, size_t bytes) -> const void* {
    void* dst = p + off;
    off += up(bytes);
    return hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice) == hipSuccess ? dst : nullptr;
  };
  fd.fa16 = put(fa16.data(), b16);
  fd.fs16 = put(fs16.data(), b16);
  fd.fa32 = put(fa32.data(), b32);
  fd.fs32 = put(fs32.data(), b32);
  fd.B32 = (const float*)put(B32.data(), bB);
  fd.Bt32 = (const float*)put(Bt32.data(), bBt);
  fd.tw = (const float2*)put(tw32.data(), bT);
  fd.twk = (const float2*)put(twk32.data(), bK);
  ff::LiftDev lift{};
  lift.dc = (int)(d / 2);
  lift.dvc = (int)(dv / 2);
  lift.up_src = (const int*)put(up_src.data(), bU);
  lift.up_w = (const float*)put(up_w.data(), bU);
  lift.dn_v = (const int2*)put(dn_v.data(), bD);
  lift.dn_w = (const float2*)put(dn_w.data(), bD);
  if (!fd.fa16 || !fd.fs16 || !fd.fa32 || !fd.fs32 || !fd.B32 || !fd.Bt32 || !fd.tw || !fd.twk || !lift.up_src ||
      !lift.up_w || !lift.dn_v || !lift.dn_w) {
    (void)hipFree(mem);
    return ff::fail(FF_EDEVICE, "copying frame to the device failed");
  }
  if (ff::configure_kernels() != hipSuccess || ff::configure_fast128() != hipSuccess) {
    (void)hipFree(mem);
    return ff::fail(FF_EDEVICE, "configuring kernels failed");
  }
  ff_frame* f = new ff_frame();
  f->d = d;
  f->k = k;
  f->rho = rho;
  f->dv = dv;
  f->lifted = lifted;
  f->lift = lift;
  f->device = dev;
  f->B = std::move(B);
  f->transpose_is_sign_flip = sign_flip;
  f->half_shift_sign = half_shift;
  f->dev_mem = mem;
  f->dev = fd;
  *out = f;
  return FF_OK;
}

extern "C" ff_status ff_frame_export(const ff_frame* f, int64_t col0, int64_t ncols, double* out) {
  ff::clear_error();
  if (!f || !out) return ff::fail(FF_EINVAL, "NULL argument");
  const int64_t d = f->d, k = f->k, rho = f->rho, W = 2 * k;
  if (col0 < 0 || ncols < 0 || col0 + ncols > k * rho)
    return ff::fail(FF_EINVAL, "column range outside [0, %lld)", (long long)(k * rho));
  std::vector<float> B32((size_t)(W * W)), up_w((size_t)f->lift.dvc);
  std::vector<int> up_src((size_t)f->lift.dvc);
  if (hipMemcpy(B32.data(), f->dev.B32, B32.size() * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(up_src.data(), f->lift.up_src, up_src.size() * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(up_w.data(), f->lift.up_w, up_w.size() * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return ff::fail(FF_EDEVICE, "reading the frame back failed");
  std::memset(out, 0, sizeof(double) * (size_t)d * (size_t)ncols);
  // column c of P = L^T Pv: its block entries B[u][2 i + s] at virtual coordinate r k + u / 2,
  // carried to the user coordinate that feeds it, with that coordinate's weight
  for (int64_t cc = 0; cc < ncols; ++cc) {
    const int64_t c = col0 + cc;
    const int64_t i = c / rho, rem = c % rho, r = rem / 2, s = rem % 2;
    for (int64_t u = 0; u < W; ++u) {
      const int64_t v = r * k + u / 2;
      const int j = up_src[v];
      if (j < 0) continue;
      out[(2 * (int64_t)j + u % 2) * ncols + cc] += (double)up_w[v] * (double)B32[u * W + 2 * i + s];
    }
  }
  return FF_OK;
}

extern "C" ff_status ff_frame_info(const ff_frame* f, int64_t* d, int64_t* k, int64_t* rho) {
  ff::clear_error();
  if (!f) return ff::fail(FF_EINVAL, "frame is NULL");
  if (d) *d = f->d;
  if (k) *k = f->k;
  if (rho) *rho = f->rho;
  return FF_OK;
}

extern "C" void ff_frame_destroy(ff_frame* f) {
  if (!f) return;
  if (f->refs.fetch_sub(1) == 1) {
    if (f->dev_mem) (void)hipFree(f->dev_mem);
    delete f;
  }
}
