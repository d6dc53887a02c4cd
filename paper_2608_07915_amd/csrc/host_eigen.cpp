// Symmetric eigendecomposition on the host (fp64): Householder reduction to
// tridiagonal form followed by implicit symmetric QR steps with a Wilkinson
// shift (the textbook method; e.g. Golub & Van Loan, Sec. 8.3), accumulating
// every transformation into the eigenvector matrix. Used by the fit, which is
// off the per-token path; 128 x 128 takes a few milliseconds. The eigenvector matrix is
// held transposed (row k = eigenvector column k), so that every reflection and rotation
// updates whole contiguous rows.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "host_common.hpp"

namespace spectra {

namespace {

// Reduce symmetric A (n x n, row-major, overwritten) to tridiagonal T = Q^T A Q; Qt holds
// Q transposed.
void householder_tridiagonal(std::vector<double>& A, std::vector<double>& Qt, int n) {
  auto a = [&](int i, int j) -> double& { return A[(size_t)i * n + j]; };
  std::vector<double> v(n), pv(n), qv(n), sr(n);
  for (int k = 0; k + 2 < n; ++k) {
    const int m = n - k - 1;  // length of the column below the diagonal
    double norm2 = 0.0;
    for (int i = 0; i < m; ++i) norm2 += a(k + 1 + i, k) * a(k + 1 + i, k);
    if (norm2 == 0.0) continue;
    const double x0 = a(k + 1, k);
    const double alpha = x0 >= 0 ? -std::sqrt(norm2) : std::sqrt(norm2);
    for (int i = 0; i < m; ++i) v[i] = a(k + 1 + i, k);
    v[0] -= alpha;
    double vtv = 0.0;
    for (int i = 0; i < m; ++i) vtv += v[i] * v[i];
    if (vtv == 0.0) continue;
    const double beta = 2.0 / vtv;  // H = I - beta v v^T on indices k+1..n-1
    // p = beta * A_sub v ; K = beta/2 * v^T p ; w = p - K v ; A_sub -= v w^T + w v^T
    // (A_sub symmetric: row j of A_sub is its column j, so the sums run as row updates;
    // each pv[i] still adds its terms in ascending j)
    std::fill(pv.begin(), pv.begin() + m, 0.0);
    for (int j = 0; j < m; ++j) {
      const double vj = v[j];
      const double* row = &a(k + 1 + j, k + 1);
      for (int i = 0; i < m; ++i) pv[i] += row[i] * vj;
    }
    for (int i = 0; i < m; ++i) pv[i] *= beta;
    double vp = 0.0;
    for (int i = 0; i < m; ++i) vp += v[i] * pv[i];
    const double K = 0.5 * beta * vp;
    for (int i = 0; i < m; ++i) qv[i] = pv[i] - K * v[i];
    for (int i = 0; i < m; ++i)
      for (int j = 0; j < m; ++j) a(k + 1 + i, k + 1 + j) -= v[i] * qv[j] + qv[i] * v[j];
    a(k + 1, k) = alpha;
    a(k, k + 1) = alpha;
    for (int i = 1; i < m; ++i) {
      a(k + 1 + i, k) = 0.0;
      a(k, k + 1 + i) = 0.0;
    }
    // Q <- Q H, i.e. rows k+1.. of Qt: s_r = sum_j v_j Qt[k+1+j][r] (ascending j), then
    // Qt[k+1+j][r] -= (beta s_r) v_j
    std::fill(sr.begin(), sr.end(), 0.0);
    for (int j = 0; j < m; ++j) {
      const double vj = v[j];
      const double* row = &Qt[(size_t)(k + 1 + j) * n];
      for (int r = 0; r < n; ++r) sr[r] += row[r] * vj;
    }
    for (int r = 0; r < n; ++r) sr[r] *= beta;
    for (int j = 0; j < m; ++j) {
      const double vj = v[j];
      double* row = &Qt[(size_t)(k + 1 + j) * n];
      for (int r = 0; r < n; ++r) row[r] -= sr[r] * vj;
    }
  }
}

}  // namespace

spectra_status eigh_sym(const double* a_in, int n, double* w, double* v_out) {
  if (n <= 0 || n > 1024) return fail(SPECTRA_EINVAL, "eigh: n=%d out of range", n);
  std::vector<double> T((size_t)n * n), Qt((size_t)n * n, 0.0);
  double fro = 0.0;
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < n; ++j) {
      const double x = 0.5 * (a_in[(size_t)i * n + j] + a_in[(size_t)j * n + i]);
      if (!std::isfinite(x)) return fail(SPECTRA_ENUMERIC, "eigh: non-finite input");
      T[(size_t)i * n + j] = x;
      fro += x * x;
    }
  for (int i = 0; i < n; ++i) Qt[(size_t)i * n + i] = 1.0;
  householder_tridiagonal(T, Qt, n);
  auto t = [&](int i, int j) -> double& { return T[(size_t)i * n + j]; };
  const double eps = 2.220446049250313e-16;
  const double tiny = 1e-300 + eps * std::sqrt(fro) * 1e-3;

  // Apply P = [[c, s], [-s, c]] on rows/cols (k, k+1): T <- P T P^T, Q <- Q P^T (rows k
  // and k+1 of Qt).
  auto rotate = [&](int k, double c, double s, int lo, int hi) {
    const int j0 = std::max(lo, k - 1), j1 = std::min(hi, k + 2);
    for (int j = j0; j <= j1; ++j) {
      const double r1 = t(k, j), r2 = t(k + 1, j);
      t(k, j) = c * r1 + s * r2;
      t(k + 1, j) = -s * r1 + c * r2;
    }
    for (int i = j0; i <= j1; ++i) {
      const double c1 = t(i, k), c2 = t(i, k + 1);
      t(i, k) = c * c1 + s * c2;
      t(i, k + 1) = -s * c1 + c * c2;
    }
    double* r1 = &Qt[(size_t)k * n];
    double* r2 = &Qt[(size_t)(k + 1) * n];
    for (int r = 0; r < n; ++r) {
      const double q1 = r1[r], q2 = r2[r];
      r1[r] = c * q1 + s * q2;
      r2[r] = -s * q1 + c * q2;
    }
  };

  int hi = n - 1;
  long iters = 0;
  const long max_iters = 60L * n;
  while (hi > 0) {
    for (int i = 0; i < hi; ++i) {
      if (std::fabs(t(i + 1, i)) <= eps * (std::fabs(t(i, i)) + std::fabs(t(i + 1, i + 1))) ||
          std::fabs(t(i + 1, i)) < tiny) {
        t(i + 1, i) = 0.0;
        t(i, i + 1) = 0.0;
      }
    }
    while (hi > 0 && t(hi, hi - 1) == 0.0) --hi;
    if (hi == 0) break;
    int lo = hi - 1;
    while (lo > 0 && t(lo, lo - 1) != 0.0) --lo;
    if (++iters > max_iters) return fail(SPECTRA_ENUMERIC, "eigh: QR iteration did not converge");
    // Wilkinson shift from the trailing 2x2 of the unreduced block [lo, hi]
    const double an = t(hi, hi), bn = t(hi, hi - 1);
    const double delta = 0.5 * (t(hi - 1, hi - 1) - an);
    const double sgn = delta >= 0 ? 1.0 : -1.0;
    const double mu = an - bn * bn / (delta + sgn * std::hypot(delta, bn));
    double x = t(lo, lo) - mu, z = t(lo + 1, lo);
    for (int k = lo; k < hi; ++k) {
      const double r = std::hypot(x, z);
      const double c = r == 0.0 ? 1.0 : x / r, s = r == 0.0 ? 0.0 : z / r;
      rotate(k, c, s, lo, hi);
      if (k + 1 < hi) {
        x = t(k + 1, k);
        z = t(k + 2, k);
      }
    }
  }
  // Sort descending (stable by position), sign-normalise, write out.
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int i, int j) { return t(i, i) > t(j, j); });
  for (int jo = 0; jo < n; ++jo) {
    const int j = order[jo];
    w[jo] = t(j, j);
    int imax = 0;
    double vmax = -1.0;
    const double* qj = &Qt[(size_t)j * n];
    for (int i = 0; i < n; ++i) {
      const double x = std::fabs(qj[i]);
      if (x > vmax) {
        vmax = x;
        imax = i;
      }
    }
    const double sg = qj[imax] < 0 ? -1.0 : 1.0;
    for (int i = 0; i < n; ++i) v_out[(size_t)i * n + jo] = sg * qj[i];
  }
  return SPECTRA_OK;
}

}  // namespace spectra
