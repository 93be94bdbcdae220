// pca.hip -- the projection before the K-means (Section 4.2: the trunk's features are projected
// to their first 256 principal directions before the clustering).
//
// Fit: the sample mean (fp64 column sums), the covariance C = (X^T X - n m m^T) / (n - 1) with
// X^T X on the tile engines (fp32 accumulation, the correction in fp64), and the r leading
// eigenpairs of C by subspace iteration: Q <- orth(C Q), n_iter times from a seeded start, then
// Rayleigh-Ritz (the eigenpairs of Q^T C Q, rotated back by Q).  The d x d x r and d x r x r
// products run on the GPU; the r x r steps -- the Cholesky factor behind each orthonormalisation
// (CholeskyQR) and the final symmetric eigensolve (Householder tridiagonalisation and implicit
// QR steps) -- run on the host in fp64, so a fit synchronises its stream.
// Projection: Z = (X - m) U^T on the tile engine, the mean folded into an fp32 column bias.
#include <math.h>

#include <algorithm>
#include <vector>

#include "gemm.hpp"
#include "host_linalg.hpp"
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

static __global__ void k_pca_seg(int32_t* __restrict__ seg, int64_t rows) {
  if (threadIdx.x == 0) {
    seg[0] = 0;
    seg[1] = (int32_t)rows;
  }
}

// C = (C - s s^T / n) / (n - 1) in place (C holds X^T X, s the fp64 column sums), mean = s / n.
static __global__ void __launch_bounds__(256) k_cov_finalize(float* __restrict__ C, const double* __restrict__ s,
                                                             int64_t n, int d, float* __restrict__ mean) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q < d) mean[q] = (float)(s[q] / (double)n);
  if (q >= (int64_t)d * d) return;
  const int i = (int)(q / d), j = (int)(q % d);
  C[q] = (float)(((double)C[q] - s[i] * s[j] / (double)n) / (double)(n - 1));
}

// A seeded start for the subspace iteration: uniform in [-1, 1) from SplitMix64 of seed + index.
static __global__ void __launch_bounds__(256) k_pca_start(float* __restrict__ Q, int64_t count, uint64_t seed) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= count) return;
  uint64_t z = seed + (uint64_t)q + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  Q[q] = (float)((double)(z >> 11) * (1.0 / 9007199254740992.0) * 2.0 - 1.0);
}

// Fresh directions for the columns of Z [d][r] that flags[] marks (rank lost): uniform in
// [-1, 1) from SplitMix64 of seed + index, as k_pca_start.
static __global__ void __launch_bounds__(256) k_pca_refill(float* __restrict__ Z, int d, int r,
                                                           const int32_t* __restrict__ flags, uint64_t seed) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= (int64_t)d * r || !flags[q % r]) return;
  uint64_t z = seed + (uint64_t)q + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  Z[q] = (float)((double)(z >> 11) * (1.0 / 9007199254740992.0) * 2.0 - 1.0);
}

// comps[j][:] = sign_j U[:, j], sign_j making the largest-magnitude entry of the column positive
// (lowest index on ties).  One block per column.
static __global__ void __launch_bounds__(256) k_pca_comps(const float* __restrict__ U, int d, int r,
                                                          float* __restrict__ comps) {
  __shared__ float sv[256];
  __shared__ int si[256];
  const int j = blockIdx.x;
  float bv = -1.f;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float a = fabsf(U[(int64_t)i * r + j]);
    if (a > bv) {  // i increases: ties keep the lower index
      bv = a;
      bi = i;
    }
  }
  sv[threadIdx.x] = bv;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (threadIdx.x < w) {
      const float ov = sv[threadIdx.x + w];
      const int oi = si[threadIdx.x + w];
      if (ov > sv[threadIdx.x] || (ov == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = ov;
        si[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  const float sign = U[(int64_t)si[0] * r + j] < 0.f ? -1.f : 1.f;
  for (int i = threadIdx.x; i < d; i += 256) comps[(int64_t)j * d + i] = sign * U[(int64_t)i * r + j];
}

// b[j] = mean . comps[j] (fp32, fixed-order block sum) and the components in the data dtype.
template <typename T>
__global__ void __launch_bounds__(256) k_pca_bias(const float* __restrict__ mean, const float* __restrict__ comps,
                                                  int d, float* __restrict__ b, T* __restrict__ comps_lo) {
  __shared__ double sh[256];
  const int j = blockIdx.x;
  double s = 0.0;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float c = comps[(int64_t)j * d + i];
    s += (double)mean[i] * (double)c;
    comps_lo[(int64_t)j * d + i] = from_f32<T>(c);
  }
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (threadIdx.x < w) sh[threadIdx.x] += sh[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) b[j] = (float)sh[0];
}

// Z [n][r] = X comps_lo^T - b (the centred projection), in the data dtype.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_pca_project(const typename C::type* __restrict__ X, const typename C::type* __restrict__ W,
                  const float* __restrict__ b, int64_t n, int d, int r, typename C::type* __restrict__ Z) {
  using T = typename C::type;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_plain<C>(n, r, d);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, true>(X + tc.m0 * d, d, tc.m_rows, W + (int64_t)tc.n0 * d, d, tc.n_cols, d, smem, acc);
  using F = Frag<C>;
  const F f;
  float bb[F::NCOL];
#pragma unroll
  for (int q = 0; q < F::NCOL; ++q) {
    const int col = f.colq(q);
    bb[q] = col < tc.n_cols ? b[tc.n0 + col] : 0.f;
  }
  store_out<C, T>(tc, acc, smem, Z, r, [&](int, int j, int rr, float v) { return v - bb[F::qidx(j, rr)]; },
                  RowId{tc.m0}, NoVec{});
}

// ------------------------------------------------------------------ host side of the fit (the r x r steps: host_linalg.hpp)

static int d2h(void* dst, const void* src, size_t bytes, hipStream_t st) {
  HMOE_TRY(hip_check(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, st), "pca: copy to host"));
  return hip_check(hipStreamSynchronize(st), "pca: synchronise");
}
static int h2d(void* dst, const void* src, size_t bytes, hipStream_t st) {
  HMOE_TRY(hip_check(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, st), "pca: copy to device"));
  return hip_check(hipStreamSynchronize(st), "pca: synchronise");
}

// Q <- Q R^{-1} with Q^T Q = R^T R (CholeskyQR), `passes` times (the second pass restores the
// orthonormality the fp32 Gram matrix loses on an ill-conditioned Q); Z is scratch of Q's size.
// Rank-revealing: when a pivot falls below 1e-9 of the largest diagonal of Q^T Q (the fp32
// Gram matrix's noise; a covariance of rank below r does this), Q is rebuilt from the
// eigenpairs (w_j, v_j) of Q^T Q -- column j = Q v_j / sqrt(w_j) where w_j stays above that
// level, a fresh seeded random column where it does not -- and the passes start again.  The
// kept columns span what Q determined; the fresh ones lie outside it with probability 1.
static int orthonormalise(float*& Q, float*& Z, int d, int r, float* S, float* Rinv, int passes, uint64_t seed,
                          Workspace& ws, hipStream_t st) {
  constexpr double kRank = 1e-9;
  std::vector<float> hs((size_t)r * r);
  std::vector<double> Sd((size_t)r * r), Ri;
  int refills = 0;
  for (int pass = 0; pass < passes; ++pass) {
    const size_t mark = ws.off;
    HMOE_TRY(launch_gemm_tn<float>(Q, Q, d, r, r, S, ws, st));
    HMOE_TRY(d2h(hs.data(), S, hs.size() * sizeof(float), st));
    for (size_t i = 0; i < hs.size(); ++i) Sd[i] = hs[i];
    if (!chol_inverse(Sd, r, Ri, kRank)) {
      if (++refills > 4) {
        set_error("pca: could not complete an orthonormal basis of %d columns", r);
        return HMOE_EINVAL;
      }
      std::vector<double> A = Sd, w, VT;
      if (!sym_eigen(A, r, w, VT)) {
        set_error("pca: the eigensolve of the %d x %d Gram matrix did not converge", r, r);
        return HMOE_ENUMERIC;
      }
      double wmax = 0.0;
      for (double x : w) wmax = x > wmax ? x : wmax;
      std::vector<int32_t> flags(r, 0);
      for (int j = 0; j < r; ++j) {
        const bool keep = wmax > 0.0 && w[j] > kRank * wmax;
        const double sc = keep ? 1.0 / sqrt(w[j]) : 0.0;
        for (int i = 0; i < r; ++i) hs[(size_t)i * r + j] = (float)(VT[(size_t)j * r + i] * sc);
        flags[j] = keep ? 0 : 1;
      }
      HMOE_TRY(h2d(Rinv, hs.data(), hs.size() * sizeof(float), st));
      HMOE_TRY(launch_gemm_nn<float>(Q, Rinv, d, r, r, Z, ws, st));
      ws.off = mark;
      HMOE_TRY(h2d(S, flags.data(), flags.size() * sizeof(int32_t), st));  // S is free until the next pass
      HMOE_LAUNCH("pca refill", k_pca_refill, dim3((unsigned)cdiv((int64_t)d * r, 256)), dim3(256), 0, st, Z, d, r,
                  (const int32_t*)S, seed + 0x5851F42D4C957F2Dull * (uint64_t)refills);
      std::swap(Q, Z);
      pass = -1;  // orthonormalise the rebuilt block from scratch
      continue;
    }
    for (size_t i = 0; i < hs.size(); ++i) hs[i] = (float)Ri[i];
    HMOE_TRY(h2d(Rinv, hs.data(), hs.size() * sizeof(float), st));
    HMOE_TRY(launch_gemm_nn<float>(Q, Rinv, d, r, r, Z, ws, st));
    ws.off = mark;
    std::swap(Q, Z);
  }
  return HMOE_OK;
}

size_t pca_fit_ws(int64_t n, int d, int r, hmoe_dtype_t dt) {
  Workspace ws(nullptr, 0);
  ws.take<double>(d);
  ws.take<int32_t>(2);
  ws.take<float>((size_t)d * d);
  ws.take<float>((size_t)d * r);
  ws.take<float>((size_t)d * r);
  ws.take<float>((size_t)r * r);
  ws.take<float>((size_t)r * r);
  const size_t g = dt == HMOE_BF16 ? gemm_tn_ws<bf16>() : gemm_tn_ws<float>();
  const size_t sg = segsum_ws(n, 1, d);
  return ws.off + (g > sg ? g : sg) + 4096;
}

template <typename T>
static int pca_fit_t(const T* X, int64_t n, int d, int r, int n_iter, uint64_t seed, float* mean, float* comps,
                     float* eigvals, Workspace& ws, hipStream_t st) {
  double* msum = ws.take<double>(d);
  int32_t* seg = ws.take<int32_t>(2);
  float* Cv = ws.take<float>((size_t)d * d);
  float* Q = ws.take<float>((size_t)d * r);
  float* Z = ws.take<float>((size_t)d * r);
  float* S = ws.take<float>((size_t)r * r);
  float* Rinv = ws.take<float>((size_t)r * r);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const size_t mark = ws.off;
  HMOE_LAUNCH("pca segment", k_pca_seg, dim3(1), dim3(64), 0, st, seg, n);
  HMOE_TRY(launch_segsum<T, double>(X, d, nullptr, seg, 1, d, n, msum, 0, ws, st));
  ws.off = mark;
  HMOE_TRY(launch_gemm_tn<T>(X, X, n, d, d, Cv, ws, st, "pca X^T X"));
  ws.off = mark;
  HMOE_LAUNCH("pca covariance", k_cov_finalize, dim3((unsigned)cdiv((int64_t)d * d, 256)), dim3(256), 0, st, Cv, msum,
              n, d, mean);
  HMOE_LAUNCH("pca start", k_pca_start, dim3((unsigned)cdiv((int64_t)d * r, 256)), dim3(256), 0, st, Q,
              (int64_t)d * r, seed);
  // one CholeskyQR pass per iteration keeps the subspace; the basis that enters Rayleigh-Ritz
  // gets two
  HMOE_TRY(orthonormalise(Q, Z, d, r, S, Rinv, n_iter == 0 ? 2 : 1, seed ^ 0xA5A5A5A5u, ws, st));
  for (int it = 0; it < n_iter; ++it) {
    HMOE_TRY(launch_gemm_nn<float>(Cv, Q, d, d, r, Z, ws, st));
    ws.off = mark;
    std::swap(Q, Z);
    HMOE_TRY(orthonormalise(Q, Z, d, r, S, Rinv, it == n_iter - 1 ? 2 : 1, seed + 0x9E3779B9u * (uint64_t)(it + 1), ws,
                            st));
  }
  // Rayleigh-Ritz: the eigenpairs of Q^T C Q, sorted by decreasing eigenvalue
  HMOE_TRY(launch_gemm_nn<float>(Cv, Q, d, d, r, Z, ws, st));
  ws.off = mark;
  HMOE_TRY(launch_gemm_tn<float>(Q, Z, d, r, r, S, ws, st));
  ws.off = mark;
  std::vector<float> hs((size_t)r * r);
  HMOE_TRY(d2h(hs.data(), S, hs.size() * sizeof(float), st));
  std::vector<double> Tm((size_t)r * r), w, VT;
  for (int i = 0; i < r; ++i)
    for (int j = 0; j < r; ++j) Tm[(size_t)i * r + j] = 0.5 * ((double)hs[(size_t)i * r + j] + hs[(size_t)j * r + i]);
  if (!sym_eigen(Tm, r, w, VT)) {
    set_error("pca: the eigensolve of the %d x %d Rayleigh-Ritz matrix did not converge", r, r);
    return HMOE_ENUMERIC;
  }
  std::vector<int> ord(r);
  for (int i = 0; i < r; ++i) ord[i] = i;
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return w[a] > w[b]; });
  std::vector<float> hw(r);
  for (int i = 0; i < r; ++i)
    for (int j = 0; j < r; ++j) hs[(size_t)i * r + j] = (float)VT[(size_t)ord[j] * r + i];
  for (int j = 0; j < r; ++j) hw[j] = (float)w[ord[j]];
  HMOE_TRY(h2d(Rinv, hs.data(), hs.size() * sizeof(float), st));
  HMOE_TRY(h2d(eigvals, hw.data(), hw.size() * sizeof(float), st));
  HMOE_TRY(launch_gemm_nn<float>(Q, Rinv, d, r, r, Z, ws, st));
  ws.off = mark;
  HMOE_LAUNCH("pca components", k_pca_comps, dim3((unsigned)r), dim3(256), 0, st, (const float*)Z, d, r, comps);
  return HMOE_OK;
}

int launch_pca_fit(const void* X, hmoe_dtype_t dt, int64_t n, int d, int r, int n_iter, uint64_t seed, float* mean,
                   float* comps, float* eigvals, Workspace& ws, hipStream_t st) {
  if (dt == HMOE_BF16) return pca_fit_t<bf16>((const bf16*)X, n, d, r, n_iter, seed, mean, comps, eigvals, ws, st);
  return pca_fit_t<float>((const float*)X, n, d, r, n_iter, seed, mean, comps, eigvals, ws, st);
}

size_t pca_project_ws(int d, int r, hmoe_dtype_t dt) {
  Workspace ws(nullptr, 0);
  ws.take<float>(r);
  ws.take<char>((size_t)r * d * (dt == HMOE_BF16 ? 2 : 4));
  return ws.off;
}

template <typename T>
static int pca_project_t(const T* X, int64_t n, int d, const float* mean, const float* comps, int r, T* Zo,
                         Workspace& ws, hipStream_t st) {
  // both operands K-contiguous: the direct-to-LDS engine in either dtype
  using C = typename std::conditional<sizeof(T) == 2, CfgDma, CfgDmaF32>::type;
  float* b = ws.take<float>(r);
  T* W = ws.take<T>((size_t)r * d);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  HMOE_LAUNCH("pca bias", k_pca_bias<T>, dim3((unsigned)r), dim3(256), 0, st, mean, comps, d, b, W);
  HMOE_LAUNCH("pca project", k_pca_project<C>, dim3((unsigned)(cdiv(n, C::BM) * cdiv(r, C::BN))), dim3(C::THREADS),
              C::LDS, st, X, (const T*)W, (const float*)b, n, d, r, Zo);
  return HMOE_OK;
}

int launch_pca_project(const void* X, hmoe_dtype_t dt, int64_t n, int d, const float* mean, const float* comps,
                       int r, void* Z, Workspace& ws, hipStream_t st) {
  if (dt == HMOE_BF16) return pca_project_t<bf16>((const bf16*)X, n, d, mean, comps, r, (bf16*)Z, ws, st);
  return pca_project_t<float>((const float*)X, n, d, mean, comps, r, (float*)Z, ws, st);
}

}  // namespace hmoe
