// host_linalg.hpp -- the r x r steps of the PCA fit, in fp64 on the host (no GPU code, so the
// CPU tests can build them alone): the Cholesky factor behind CholeskyQR with the inverse of
// its transpose, and a symmetric eigensolver.
#pragma once

#include <math.h>

#include <thread>
#include <vector>

namespace hmoe {

inline double dot_f64(const double* a, const double* b, int n) {
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  int k = 0;
  for (; k + 4 <= n; k += 4) {
    s0 += a[k] * b[k];
    s1 += a[k + 1] * b[k + 1];
    s2 += a[k + 2] * b[k + 2];
    s3 += a[k + 3] * b[k + 3];
  }
  for (; k < n; ++k) s0 += a[k] * b[k];
  return (s0 + s1) + (s2 + s3);
}

// S = L L^T (L lower triangular, row-major, built row by row from contiguous dot products);
// returns R^{-1} for R = L^T in Ri (upper triangular, row-major): row j of R^{-1} is column j of
// L^{-1}, the forward solve of L x = e_j.  False when S is not positive definite even after a
// tiny diagonal shift, or when a pivot (before its square root) is at most min_rel_pivot times
// the largest diagonal entry of S (the columns behind S have lost rank to that precision).
inline bool chol_inverse(const std::vector<double>& S, int r, std::vector<double>& Ri,
                         double min_rel_pivot = 0.0) {
  double tr = 0.0, dmax = 0.0;
  for (int i = 0; i < r; ++i) {
    tr += S[(size_t)i * r + i];
    dmax = S[(size_t)i * r + i] > dmax ? S[(size_t)i * r + i] : dmax;
  }
  const double shift = 1e-12 * tr / r;
  std::vector<double> L((size_t)r * r, 0.0);
  for (int i = 0; i < r; ++i) {
    double* Li = &L[(size_t)i * r];
    for (int j = 0; j <= i; ++j) {
      const double* Lj = &L[(size_t)j * r];
      const double v = S[(size_t)i * r + j] + (i == j ? shift : 0.0) - dot_f64(Li, Lj, j);
      if (i == j) {
        if (!(v > 0.0) || !(v > min_rel_pivot * dmax)) return false;
        Li[i] = sqrt(v);
      } else {
        Li[j] = v / Lj[j];
      }
    }
  }
  // the columns of L^{-1} are independent solves: spread over a few threads (column j costs
  // ~(r - j)^2 / 2, so thread t takes j = t, t + T, ... to balance them); each result is the
  // same as the serial solve's
  Ri.assign((size_t)r * r, 0.0);
  auto solve = [&](int t, int T) {
    std::vector<double> x(r);
    for (int j = t; j < r; j += T) {
      x[j] = 1.0 / L[(size_t)j * r + j];
      for (int i = j + 1; i < r; ++i) x[i] = -dot_f64(&L[(size_t)i * r + j], &x[j], i - j) / L[(size_t)i * r + i];
      for (int i = j; i < r; ++i) Ri[(size_t)j * r + i] = x[i];
    }
  };
  const unsigned hw = std::thread::hardware_concurrency();
  const int T = r >= 64 ? (int)(hw < 2 ? 1 : (hw > 8 ? 8 : hw)) : 1;
  std::vector<std::thread> pool;
  for (int t = 1; t < T; ++t) pool.emplace_back(solve, t, T);
  solve(0, T);
  for (std::thread& th : pool) th.join();
  return true;
}

// Eigenpairs of the symmetric A (n x n, row-major; destroyed): Householder reflections reduce A
// to tridiagonal form T = Q^T A Q, then implicit symmetric QR steps with the Wilkinson shift
// (bulge chasing with Givens rotations, deflating negligible off-diagonal entries) diagonalise
// T.  Both transformations are accumulated into the rows of VT, so on return row j of VT is the
// unit eigenvector of eigenvalue w[j] (unsorted).  All updates run along contiguous rows.
// Returns false when the QR steps have not deflated every off-diagonal entry within max_steps
// (default 60 n, about 30 times what the shift needs in practice); w and VT are then not
// eigenpairs.
inline bool sym_eigen(std::vector<double>& A, int n, std::vector<double>& w, std::vector<double>& VT,
                      int max_steps = -1) {
  if (max_steps < 0) max_steps = 60 * n;
  VT.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) VT[(size_t)i * n + i] = 1.0;
  std::vector<double> d(n), e(n, 0.0), u(n), p(n), acc(n);
  for (int k = 0; k + 2 < n; ++k) {
    const int m = n - k - 1;
    const double* x = &A[(size_t)k * n + k + 1];  // the column below the diagonal, read as row k
    const double xn = sqrt(dot_f64(x, x, m));
    if (xn == 0.0) continue;  // already reduced: e[k] stays 0
    const double alpha = x[0] > 0.0 ? -xn : xn;
    for (int i = 0; i < m; ++i) u[i] = x[i];
    u[0] -= alpha;
    e[k] = alpha;
    const double sc = sqrt(2.0 / dot_f64(u.data(), u.data(), m));
    for (int i = 0; i < m; ++i) u[i] *= sc;  // the reflection is I - u u^T
    // trailing block B <- H B H = B - u q^T - q u^T with p = B u, q = p - (u^T p / 2) u
    for (int i = 0; i < m; ++i) p[i] = dot_f64(&A[(size_t)(k + 1 + i) * n + k + 1], u.data(), m);
    const double half = 0.5 * dot_f64(u.data(), p.data(), m);
    for (int i = 0; i < m; ++i) p[i] -= half * u[i];
    for (int i = 0; i < m; ++i) {
      double* row = &A[(size_t)(k + 1 + i) * n + k + 1];
      const double ui = u[i], qi = p[i];
      for (int j = 0; j < m; ++j) row[j] -= ui * p[j] + qi * u[j];
    }
    // VT <- H VT on rows k+1 ..
    for (int j = 0; j < n; ++j) acc[j] = 0.0;
    for (int i = 0; i < m; ++i) {
      const double* row = &VT[(size_t)(k + 1 + i) * n];
      const double ui = u[i];
      for (int j = 0; j < n; ++j) acc[j] += ui * row[j];
    }
    for (int i = 0; i < m; ++i) {
      double* row = &VT[(size_t)(k + 1 + i) * n];
      const double ui = u[i];
      for (int j = 0; j < n; ++j) row[j] -= ui * acc[j];
    }
  }
  for (int i = 0; i < n; ++i) d[i] = A[(size_t)i * n + i];
  if (n >= 2) e[n - 2] = A[(size_t)(n - 2) * n + n - 1];
  const double eps = 2.220446049250313e-16;
  int hi = n - 1;
  for (int guard = 0; hi > 0 && guard < max_steps;) {
    if (fabs(e[hi - 1]) <= eps * (fabs(d[hi - 1]) + fabs(d[hi]))) {  // d[hi] has converged
      e[hi - 1] = 0.0;
      --hi;
      continue;
    }
    int lo = hi - 1;  // the unreduced block [lo, hi]
    while (lo > 0 && fabs(e[lo - 1]) > eps * (fabs(d[lo - 1]) + fabs(d[lo]))) --lo;
    ++guard;
    // Wilkinson shift: the eigenvalue of the trailing 2 x 2 block nearer to its last diagonal
    const double half = 0.5 * (d[hi - 1] - d[hi]);
    const double eb = e[hi - 1];
    const double mu = d[hi] - eb * eb / (half + (half >= 0.0 ? 1.0 : -1.0) * hypot(half, eb));
    double x = d[lo] - mu, z = e[lo];
    for (int k = lo; k < hi; ++k) {
      // rotation of coordinates (k, k+1) that zeroes z against x (the bulge from step k-1)
      const double r = hypot(x, z);
      const double c = r == 0.0 ? 1.0 : x / r, s = r == 0.0 ? 0.0 : -z / r;
      if (k > lo) e[k - 1] = r;
      const double ak = d[k], bk = d[k + 1], f = e[k];
      d[k] = c * c * ak - 2.0 * c * s * f + s * s * bk;
      d[k + 1] = s * s * ak + 2.0 * c * s * f + c * c * bk;
      e[k] = c * s * (ak - bk) + (c * c - s * s) * f;
      if (k + 1 < hi) {
        const double g = e[k + 1];
        z = -s * g;  // the new bulge at (k, k + 2)
        e[k + 1] = c * g;
      }
      x = e[k];
      double* r0 = &VT[(size_t)k * n];
      double* r1 = &VT[(size_t)(k + 1) * n];
      for (int j = 0; j < n; ++j) {
        const double v0 = r0[j], v1 = r1[j];
        r0[j] = c * v0 - s * v1;
        r1[j] = s * v0 + c * v1;
      }
    }
  }
  w = d;
  return hi <= 0;
}

}  // namespace hmoe
