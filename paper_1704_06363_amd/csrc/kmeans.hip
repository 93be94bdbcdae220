// kmeans.hip -- the K-means gater of Section 2: nearest-centroid assignment (Eq. 2) as a fused
// distance GEMM + argmin on MFMA, k-means++ seeding, and the Lloyd centre update as a
// deterministic segmented reduction with farthest-point reseeding of empty clusters.
#include <float.h>
#include <limits.h>

#include "gemm.hpp"
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

// ------------------------------------------------------------------ centre norms

template <typename T>
__global__ void __launch_bounds__(256) k_cnorm(const T* __restrict__ C, int K, int d, float* __restrict__ cn) {
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (k >= K) return;
  float s = 0.f;
  for (int j = l; j < d; j += 64) {
    const float c = to_f32(C[(int64_t)k * d + j]);
    s += c * c;
  }
  s = wave_sum(s);
  if (l == 0) cn[k] = s;
}

// ------------------------------------------------------------------ distance GEMM + argmin

// One BM-row x BN-centre tile: dist'(i, k) = |c_k|^2 - 2 x_i . c_k (the |x_i|^2 term is
// common to the row); the tile's minimum per row (lowest k on ties) goes either straight to
// assign / min_dist (all centres in one tile) or to per-tile partials merged afterwards.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_assign(const typename C::type* __restrict__ X, int64_t n, int d, const typename C::type* __restrict__ Cn, int K,
             const float* __restrict__ cn, int32_t* __restrict__ assign, float* __restrict__ min_dist,
             float* __restrict__ part_v, int32_t* __restrict__ part_i, float* __restrict__ xnorm) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  constexpr int NV = C::BM * 8 / C::THREADS;  // staged A vectors per thread
  const TileCoord tc = tile_plain<C>(n, K, d);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  float xs[NV];
  gemm_tile<C, true, true, true>(X + tc.m0 * d, d, tc.m_rows, Cn + (int64_t)tc.n0 * d, d, tc.n_cols, d, smem, acc,
                                 xs);
  lds<float>* xn = reinterpret_cast<lds<float>*>(smem);  // [BM]
  lds<float>* rv = xn + C::BM;                       // [WAVES_N][BM]
  lds<int32_t>* ri = reinterpret_cast<lds<int32_t>*>(rv + C::WAVES_N * C::BM);
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    float s = xs[q];
    s += shfl_xor(s, 1);
    s += shfl_xor(s, 2);
    s += shfl_xor(s, 4);
    if ((t & 7) == 0) xn[(t + C::THREADS * q) >> 3] = s;
  }
  const Frag<C> f;
#pragma unroll
  for (int i = 0; i < C::MI; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float best = FLT_MAX;
      int bi = INT_MAX;
#pragma unroll
      for (int j = 0; j < C::NJ; ++j) {
        const int col = f.col(j, 0);
        if (col < tc.n_cols) argmin_merge(best, bi, cn[tc.n0 + col] - 2.f * acc[i][j][r], tc.n0 + col);
      }
#pragma unroll
      for (int m = 1; m < 16; m <<= 1) {
        const float v2 = shfl_xor(best, m);
        const int i2 = shfl_xor(bi, m);
        argmin_merge(best, bi, v2, i2);
      }
      if (f.lr == 0) {
        rv[f.wn * C::BM + f.row(i, r)] = best;
        ri[f.wn * C::BM + f.row(i, r)] = bi;
      }
    }
  }
  __syncthreads();
  const int nt = (int)cdiv(K, C::BN);
  for (int q = t; q < tc.m_rows; q += C::THREADS) {
    float v = rv[q];
    int bi = ri[q];
#pragma unroll
    for (int w = 1; w < C::WAVES_N; ++w) argmin_merge(v, bi, rv[w * C::BM + q], ri[w * C::BM + q]);
    const int64_t row = tc.m0 + q;
    if (nt == 1) {
      assign[row] = bi;
      if (min_dist) min_dist[row] = fmaxf(v + xn[q], 0.f);
    } else {
      const int ti = tc.n0 / C::BN;
      part_v[(int64_t)ti * n + row] = v;
      part_i[(int64_t)ti * n + row] = bi;
      if (ti == 0) xnorm[row] = xn[q];
    }
  }
}

// The same tile on the direct-to-LDS engine (bf16 with many centres, and fp32).  Each lane
// holds four consecutive centres of one row per fragment; the row norms come from the A
// fragments the engine already reads (fragment i summed by wave i mod WAVES_N).  fp32 rows are
// staged as 16-bit units (U per element).
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_assign_dma(const typename C::type* __restrict__ X, int64_t n, int d, const typename C::type* __restrict__ Cn,
                 int K,
                 const float* __restrict__ cn, int32_t* __restrict__ assign, float* __restrict__ min_dist,
                 float* __restrict__ part_v, int32_t* __restrict__ part_i, float* __restrict__ xnorm) {
  static_assert(C::DMA && C::TRANS, "direct-to-LDS configuration expected");
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_plain<C>(n, K, d);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  float xs[C::MI];
  // only the first centre tile of a row block needs the row norms (min_dist = min + |x|^2)
  constexpr int U = C::F32 ? 2 : 1;
  const bf16* Xu = reinterpret_cast<const bf16*>(X);
  const bf16* Cu = reinterpret_cast<const bf16*>(Cn);
  DmaTile<C, true, true> pipe;
  pipe.prime(Xu + tc.m0 * d * U, (int64_t)d * U, tc.m_rows, Cu + (int64_t)tc.n0 * d * U, (int64_t)d * U, tc.n_cols,
             d * U, smem);
  if (tc.n0 == 0)
    pipe.template run<true>(smem, acc, xs);
  else
    pipe.template run<false>(smem, acc);
  using F = Frag<C>;
  const F f;
  lds<float>* xn = reinterpret_cast<lds<float>*>(smem);  // [BM]
  lds<float>* rv = xn + C::BM;                           // [WAVES_N][BM]
  lds<int32_t>* ri = reinterpret_cast<lds<int32_t>*>(rv + C::WAVES_N * C::BM);
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
    if (tc.n0 == 0 && (i % C::WAVES_N) == f.wn) {
      float s = xs[i];
      s += shfl_xor(s, 16);
      s += shfl_xor(s, 32);
      if (f.lg == 0) xn[f.row(i, 0)] = s;
    }
  float cv[F::NCOL];
#pragma unroll
  for (int q = 0; q < F::NCOL; ++q) {
    const int col = f.colq(q);
    cv[q] = col < tc.n_cols ? cn[tc.n0 + col] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < C::MI; ++i) {
    float best = FLT_MAX;
    int bi = INT_MAX;
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int col = f.col(j, r);
        if (col < tc.n_cols) argmin_merge(best, bi, cv[F::qidx(j, r)] - 2.f * acc[i][j][r], tc.n0 + col);
      }
#pragma unroll
    for (int m = 16; m < 64; m <<= 1) {
      const float v2 = shfl_xor(best, m);
      const int i2 = shfl_xor(bi, m);
      argmin_merge(best, bi, v2, i2);
    }
    if (f.lg == 0) {
      rv[f.wn * C::BM + f.row(i, 0)] = best;
      ri[f.wn * C::BM + f.row(i, 0)] = bi;
    }
  }
  __syncthreads();
  const int nt = (int)cdiv(K, C::BN);
  for (int q = threadIdx.x; q < tc.m_rows; q += C::THREADS) {
    float v = rv[q];
    int bi = ri[q];
#pragma unroll
    for (int w = 1; w < C::WAVES_N; ++w) argmin_merge(v, bi, rv[w * C::BM + q], ri[w * C::BM + q]);
    const int64_t row = tc.m0 + q;
    if (nt == 1) {
      assign[row] = bi;
      if (min_dist) min_dist[row] = fmaxf(v + xn[q], 0.f);
    } else {
      const int ti = tc.n0 / C::BN;
      part_v[(int64_t)ti * n + row] = v;
      part_i[(int64_t)ti * n + row] = bi;
      if (ti == 0) xnorm[row] = xn[q];
    }
  }
}

__global__ void __launch_bounds__(256) k_assign_merge(const float* __restrict__ part_v,
                                                      const int32_t* __restrict__ part_i,
                                                      const float* __restrict__ xnorm, int64_t n, int nt,
                                                      int32_t* __restrict__ assign, float* __restrict__ min_dist) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= n) return;
  float v = FLT_MAX;
  int bi = INT_MAX;
  for (int t = 0; t < nt; ++t) argmin_merge(v, bi, part_v[(int64_t)t * n + row], part_i[(int64_t)t * n + row]);
  assign[row] = bi;
  if (min_dist) min_dist[row] = fmaxf(v + xnorm[row], 0.f);
}

// Centre-tile width of the assignment: up to 64 centres run the narrow 128 x 64 tiles of the
// direct-to-LDS engine, fp32 above that and bf16 above 128 centres its 256 x 256 tiles, bf16
// with 65 .. 128 centres the register-staged 128 x 128 tiles.
// bf16 with more than 128 centres
typedef CfgDma CfgAssignWide;

static int assign_bn(hmoe_dtype_t dt, int32_t K) {
  if (K <= 64) return 64;
  if (dt != HMOE_BF16) return CfgDmaF32::BN;
  return K > 128 ? CfgAssignWide::BN : 128;
}

static size_t assign_ws_bytes(int64_t n, int32_t K, hmoe_dtype_t dt) {
  Workspace ws(nullptr, 0);
  const int nt = (int)cdiv(K, assign_bn(dt, K));
  ws.take<float>(K);
  if (nt > 1) {
    ws.take<float>((size_t)nt * n);
    ws.take<int32_t>((size_t)nt * n);
    ws.take<float>(n);
  }
  return ws.off;
}

template <class C>
static int assign_t(const typename C::type* X, int64_t n, int32_t d, const typename C::type* Cn, int32_t K,
                    int32_t* assign, float* min_dist, Workspace& ws, hipStream_t st) {
  using T = typename C::type;
  const int nt = (int)cdiv(K, C::BN);
  float* cn = ws.take<float>(K);
  float *pv = nullptr, *xn = nullptr;
  int32_t* pi = nullptr;
  if (nt > 1) {
    pv = ws.take<float>((size_t)nt * n);
    pi = ws.take<int32_t>((size_t)nt * n);
    xn = ws.take<float>(n);
  }
  if (!ws.fits()) return HMOE_EWORKSPACE;
  HMOE_LAUNCH("centre norms", k_cnorm<T>, dim3((unsigned)cdiv(K, 4)), dim3(256), 0, st, Cn, K, d, cn);
  if (n == 0) return HMOE_OK;
  const int64_t tiles = cdiv(n, C::BM) * nt;
  if constexpr (C::DMA)
    HMOE_LAUNCH("assign", k_assign_dma<C>, dim3((unsigned)tiles), dim3(C::THREADS), C::LDS, st, X, n, d, Cn, K, cn,
                assign, min_dist, pv, pi, xn);
  else
    HMOE_LAUNCH("assign", k_assign<C>, dim3((unsigned)tiles), dim3(C::THREADS), C::LDS, st, X, n, d, Cn, K, cn,
                assign, min_dist, pv, pi, xn);
  if (nt > 1)
    HMOE_LAUNCH("assign merge", k_assign_merge, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, pv, pi, xn, n, nt,
                assign, min_dist);
  return HMOE_OK;
}

int launch_assign(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const void* C, int32_t K, int32_t* assign,
                  float* min_dist, Workspace& ws, hipStream_t st) {
  const int bn = assign_bn(dt, K);
  if (dt == HMOE_BF16) {
    if (bn == 64) return assign_t<CfgDmaNarrow>((const bf16*)X, n, d, (const bf16*)C, K, assign, min_dist, ws, st);
    if (K > 128)
      return assign_t<CfgAssignWide>((const bf16*)X, n, d, (const bf16*)C, K, assign, min_dist, ws, st);
    return assign_t<CfgSmall<bf16>>((const bf16*)X, n, d, (const bf16*)C, K, assign, min_dist, ws, st);
  }
  if (bn == 64)
    return assign_t<CfgDmaF32Narrow>((const float*)X, n, d, (const float*)C, K, assign, min_dist, ws, st);
  return assign_t<CfgDmaF32>((const float*)X, n, d, (const float*)C, K, assign, min_dist, ws, st);
}

// ------------------------------------------------------------------ k-means++ seeding

constexpr int kKppRows = 256;  // rows per block of the D^2 pass

__global__ void k_kpp_first(const double* __restrict__ u, int64_t n, int32_t* __restrict__ idx) {
  if (threadIdx.x == 0) {
    int64_t f = (int64_t)floor(u[0] * (double)n);
    idx[0] = (int32_t)(f > n - 1 ? n - 1 : f);
  }
}

// D2[i] = min(D2[i], |x_i - X[idx[t]]|^2) (fp64 direct differences; t == 0 initialises) and
// bsum[b] = sum of D2 over the block's kKppRows rows, in a fixed order.  16 lanes share a row
// (16-byte loads, fp64 partial sums reduced over the 16 lanes), so each wave streams 4 rows at
// once and the block 16.
template <typename T>
__global__ void __launch_bounds__(256) k_kpp_update(const T* __restrict__ X, int64_t n, int d,
                                                    const int32_t* __restrict__ idx, int t,
                                                    double* __restrict__ D2, double* __restrict__ bsum) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int G = 16;  // lanes per row
  __shared__ double rowv[kKppRows];
  const int lane = threadIdx.x % G;         // position inside the row group
  const int grp = threadIdx.x / G;          // 16 row groups per block
  const T* c = X + (int64_t)idx[t] * d;
  const int64_t r0 = (int64_t)blockIdx.x * kKppRows;
  const int vpr = d / EPV;                  // 16-byte vectors per row
  for (int q = 0; q < kKppRows / 16; ++q) {
    const int lr = q * 16 + grp;
    const int64_t i = r0 + lr;
    double s = 0.0;
    if (i < n) {
      const T* x = X + i * d;
      for (int v = lane; v < vpr; v += G) {
        const i32x4 xr = *reinterpret_cast<const i32x4*>(x + v * EPV);
        const i32x4 cr = *reinterpret_cast<const i32x4*>(c + v * EPV);
        const T* xe = reinterpret_cast<const T*>(&xr);
        const T* ce = reinterpret_cast<const T*>(&cr);
#pragma unroll
        for (int z = 0; z < EPV; ++z) {
          const double df = (double)to_f32(xe[z]) - (double)to_f32(ce[z]);
          s += df * df;
        }
      }
    }
#pragma unroll
    for (int m = 1; m < G; m <<= 1) s += shfl_xor(s, m);
    if (lane == 0) {
      double v = 0.0;
      if (i < n) {
        v = s;
        if (t > 0) {
          const double old = D2[i];
          v = old < s ? old : s;
        }
        D2[i] = v;
      }
      rowv[lr] = v;
    }
  }
  __syncthreads();
  // block sum in row order, split over the first wave: lane l adds rows 4l..4l+3, then the
  // lanes are combined by the wave's fixed butterfly
  if (threadIdx.x < 64) {
    double s = ((rowv[4 * threadIdx.x] + rowv[4 * threadIdx.x + 1]) + rowv[4 * threadIdx.x + 2]) +
               rowv[4 * threadIdx.x + 3];
    s = wave_sum(s);
    if (threadIdx.x == 0) bsum[blockIdx.x] = s;
  }
}

// Picks centre t: the first row whose running D^2 sum exceeds u[t] * total (lowest unchosen row
// if the total is zero).  One block of 1024 threads.
__global__ void __launch_bounds__(1024) k_kpp_select(const double* __restrict__ D2, int64_t n,
                                                     const double* __restrict__ bsum, int nb,
                                                     const double* __restrict__ u, int t,
                                                     int32_t* __restrict__ idx) {
  __shared__ double sh[17];
  __shared__ int32_t pick;
  const int per = (nb + 1023) / 1024;
  const int b0 = threadIdx.x * per;
  double s = 0.0;
  for (int q = 0; q < per; ++q)
    if (b0 + q < nb) s += bsum[b0 + q];
  double S;
  const double ex = block_excl_scan<double>(s, sh, &S);
  if (threadIdx.x == 0) pick = -1;
  __syncthreads();
  if (S > 0.0) {
    const double target = u[t] * S;
    // the thread whose run of blocks crosses the target walks its rows in order
    if (ex <= target && target < ex + s) {
      double P = ex;
      int32_t found = -1;
      for (int q = 0; q < per && found < 0; ++q) {
        const int b = b0 + q;
        if (b >= nb) break;
        if (P + bsum[b] <= target) {
          P += bsum[b];
          continue;
        }
        const int64_t r1 = ((int64_t)b + 1) * kKppRows < n ? ((int64_t)b + 1) * kKppRows : n;
        for (int64_t i = (int64_t)b * kKppRows; i < r1; ++i) {
          P += D2[i];
          if (P > target) {
            found = (int32_t)i;
            break;
          }
        }
        if (found < 0) {  // rounding left the crossing just past this block: take its last
          for (int64_t i = r1 - 1; i >= (int64_t)b * kKppRows; --i)  // row with D2 > 0
            if (D2[i] > 0.0) { found = (int32_t)i; break; }
        }
      }
      pick = found;
    }
    __syncthreads();
    if (threadIdx.x == 0 && pick < 0) {  // target beyond the rounded total: last row with D2 > 0
      for (int64_t i = n - 1; i >= 0; --i)
        if (D2[i] > 0.0) { pick = (int32_t)i; break; }
    }
    __syncthreads();
  }
  if (pick < 0) {
    // every D^2 is zero: the lowest row not chosen yet (one of 0..t)
    __shared__ int32_t low;
    if (threadIdx.x == 0) low = INT_MAX;
    __syncthreads();
    for (int i = threadIdx.x; i <= t; i += 1024) {
      bool used = false;
      for (int q = 0; q < t; ++q) used |= (idx[q] == i);
      if (!used) atomicMin(&low, i);
    }
    __syncthreads();
    if (threadIdx.x == 0) pick = low;
    __syncthreads();
  }
  if (threadIdx.x == 0) idx[t] = pick;
}

// C[k][:] = X[idx[k]][:] as fp32, and Cd (the data-precision copy) when given.
template <typename T>
__global__ void __launch_bounds__(256) k_gather_centres(const T* __restrict__ X, int d,
                                                        const int32_t* __restrict__ idx, int K,
                                                        float* __restrict__ C, T* __restrict__ Cd) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= (int64_t)K * d) return;
  const int k = (int)(q / d), j = (int)(q % d);
  const T v = X[(int64_t)idx[k] * d + j];
  C[q] = to_f32(v);
  if (Cd) Cd[q] = v;
}

// ------------------------------------------------------------------ Lloyd update

// The farthest-row search of the first reseed, spread over the grid: block b takes rows
// [b chunk, (b + 1) chunk) and writes its largest min_dist among rows whose cluster has more
// than one member (lowest index on ties; -1 / INT64_MAX when it has none) to pv[b], pi[b].
// Every block returns at once when no cluster is empty.
constexpr int kReseedBlocks = 512;

__global__ void __launch_bounds__(1024) k_reseed_scan(const int32_t* __restrict__ assign,
                                                      const float* __restrict__ d1, int64_t n, int K,
                                                      const int32_t* __restrict__ counts32, float* __restrict__ pv,
                                                      int64_t* __restrict__ pi) {
  __shared__ int any_empty;
  __shared__ float bv[16];
  __shared__ int64_t bix[16];
  if (threadIdx.x == 0) any_empty = 0;
  __syncthreads();
  for (int k = threadIdx.x; k < K; k += 1024)
    if (counts32[k] == 0) any_empty = 1;
  __syncthreads();
  if (!any_empty) return;
  const int64_t chunk = cdiv(n, (int64_t)gridDim.x);
  const int64_t i0 = (int64_t)blockIdx.x * chunk;
  const int64_t i1 = i0 + chunk < n ? i0 + chunk : n;
  float best = -1.f;
  int64_t bi = INT64_MAX;
  for (int64_t i = i0 + threadIdx.x; i < i1; i += 1024) {
    const int32_t a = assign[i];
    if ((unsigned)a >= (unsigned)K || counts32[a] <= 1) continue;  // out-of-range ids are never donors
    const float v = d1[i];
    if (v > best || (v == best && i < bi)) {
      best = v;
      bi = i;
    }
  }
  for (int m = 1; m < 64; m <<= 1) {
    const float v2 = __shfl_xor(best, m, 64);
    const int64_t i2 = __shfl_xor(bi, m, 64);
    if (v2 > best || (v2 == best && i2 < bi)) {
      best = v2;
      bi = i2;
    }
  }
  if ((threadIdx.x & 63) == 0) {
    bv[threadIdx.x >> 6] = best;
    bix[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w)
      if (bv[w] > best || (bv[w] == best && bix[w] < bi)) {
        best = bv[w];
        bi = bix[w];
      }
    pv[blockIdx.x] = best;
    pi[blockIdx.x] = bi;
  }
}

// Loads counts into shared memory, reseeds empty clusters (ascending ids; each takes the
// farthest row -- largest min_dist, lowest index on ties -- whose cluster has more than one
// member, moves it and its vector between the fp64 sums), then writes counts back.  The first
// reseed takes its row from the np partials of k_reseed_scan (the same counts and assignment,
// so the same row); later ones scan the rows here.  One block of 1024 threads; K <= 4096.
template <typename T>
__global__ void __launch_bounds__(1024) k_reseed(const T* __restrict__ X, int64_t n, int d, int K,
                                                 int32_t* __restrict__ assign, const float* __restrict__ d1,
                                                 int32_t* __restrict__ counts32, int64_t* __restrict__ counts64,
                                                 double* __restrict__ sums, int reseed, const float* __restrict__ pv,
                                                 const int64_t* __restrict__ pi, int np) {
  __shared__ int32_t cnt[4096];
  __shared__ float bv[16];
  __shared__ int64_t bix[16];
  __shared__ int64_t chosen;
  for (int k = threadIdx.x; k < K; k += 1024) cnt[k] = counts32[k];
  __syncthreads();
  if (reseed && n > 0) {
    bool first = true;
    for (int k = 0; k < K; ++k) {
      if (cnt[k] != 0) continue;
      float best = -1.f;
      int64_t bi = INT64_MAX;
      if (first && np > 0) {
        for (int q = threadIdx.x; q < np; q += 1024) {
          const float v = pv[q];
          const int64_t i = pi[q];
          if (v > best || (v == best && i < bi)) {
            best = v;
            bi = i;
          }
        }
      } else {
        for (int64_t i = threadIdx.x; i < n; i += 1024) {
          const int32_t a = __hip_atomic_load(assign + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if ((unsigned)a >= (unsigned)K || cnt[a] <= 1) continue;
          const float v = d1[i];
          if (v > best || (v == best && i < bi)) {
            best = v;
            bi = i;
          }
        }
      }
      first = false;
      for (int m = 1; m < 64; m <<= 1) {
        const float v2 = __shfl_xor(best, m, 64);
        const int64_t i2 = __shfl_xor(bi, m, 64);
        if (v2 > best || (v2 == best && i2 < bi)) {
          best = v2;
          bi = i2;
        }
      }
      if ((threadIdx.x & 63) == 0) {
        bv[threadIdx.x >> 6] = best;
        bix[threadIdx.x >> 6] = bi;
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        float b = bv[0];
        int64_t c = bix[0];
        for (int w = 1; w < 16; ++w)
          if (bv[w] > b || (bv[w] == b && bix[w] < c)) {
            b = bv[w];
            c = bix[w];
          }
        chosen = (c == INT64_MAX) ? -1 : c;
      }
      __syncthreads();
      const int64_t i = chosen;
      if (i < 0) break;  // no donor left; eligibility only shrinks, so later empties stay empty
      const int32_t donor = __hip_atomic_load(assign + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      for (int j = threadIdx.x; j < d; j += 1024) {
        const double x = (double)to_f32(X[i * d + j]);
        sums[(int64_t)donor * d + j] -= x;
        sums[(int64_t)k * d + j] = x;
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        cnt[donor] -= 1;
        cnt[k] = 1;
        __hip_atomic_store(assign + i, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
    }
  }
  for (int k = threadIdx.x; k < K; k += 1024) {
    counts32[k] = cnt[k];
    if (counts64) counts64[k] = cnt[k];
  }
}

__global__ void __launch_bounds__(256) k_add_counts(const int32_t* __restrict__ c32, int K, int64_t* __restrict__ c64) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k < K) c64[k] += c32[k];
}

// Cd = C rounded to the data precision.
template <typename T>
__global__ void __launch_bounds__(256) k_convert_centres(const float* __restrict__ C, int64_t count,
                                                         T* __restrict__ Cd) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q < count) Cd[q] = from_f32<T>(C[q]);
}

// C = sums / counts for non-empty clusters (others keep C); Cd = data-precision copy of C.
template <typename T, typename CNT>
__global__ void __launch_bounds__(256) k_finalize(const double* __restrict__ sums, const CNT* __restrict__ counts,
                                                  int K, int d, float* __restrict__ C, T* __restrict__ Cd) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= (int64_t)K * d) return;
  const int k = (int)(q / d);
  float c = C[q];
  if (counts[k] > 0) c = (float)(sums[q] / (double)counts[k]);
  C[q] = c;
  if (Cd) Cd[q] = from_f32<T>(c);
}

// ------------------------------------------------------------------ fit / update drivers

struct UpdateBufs {
  int32_t *counts32, *offsets, *perm, *inv;
};

template <typename T>
static int update_core(const T* X, int64_t n, int32_t d, int32_t K, int32_t* assign, const float* d1,
                       double* sums, int64_t* counts64, int accumulate, int reseed, const UpdateBufs& b,
                       Workspace& ws, hipStream_t st) {
  HMOE_TRY(launch_dispatch(assign, n, K, b.counts32, b.offsets, b.perm, b.inv, ws, st));
  HMOE_TRY(launch_segsum<T, double>(X, d, b.perm, b.offsets, K, d, n, sums, accumulate, ws, st));
  if (accumulate) {
    HMOE_LAUNCH("add counts", k_add_counts, dim3((unsigned)cdiv(K, 256)), dim3(256), 0, st, b.counts32, K, counts64);
    return HMOE_OK;
  }
  float* pv = nullptr;
  int64_t* pi = nullptr;
  int np = 0;
  if (reseed && n > 0) {
    np = (int)(cdiv(n, (int64_t)4096) < kReseedBlocks ? cdiv(n, (int64_t)4096) : kReseedBlocks);
    pv = ws.take<float>(np);
    pi = ws.take<int64_t>(np);
    if (!ws.fits()) return HMOE_EWORKSPACE;
    HMOE_LAUNCH("reseed scan", k_reseed_scan, dim3((unsigned)np), dim3(1024), 0, st, (const int32_t*)assign, d1, n, K,
                (const int32_t*)b.counts32, pv, pi);
  }
  HMOE_LAUNCH("reseed", k_reseed<T>, dim3(1), dim3(1024), 0, st, X, n, d, K, assign, d1, b.counts32, counts64, sums,
                     reseed, (const float*)pv, (const int64_t*)pi, np);
  return HMOE_OK;
}

static size_t update_scratch(int64_t n, int32_t d, int32_t K) {
  Workspace ws(nullptr, 0);
  ws.take<int32_t>(K);
  ws.take<int32_t>(K + 1);
  ws.take<int32_t>(n);
  ws.take<int32_t>(n);
  size_t s = ws.off + dispatch_ws(n, K) + segsum_ws(n, K, d) +
             (size_t)kReseedBlocks * (sizeof(float) + sizeof(int64_t)) + 4096;
  return s;
}

template <typename T>
static int update_t(const T* X, int64_t n, int32_t d, int32_t K, int32_t* assign, const float* d1, double* sums,
                    int64_t* counts64, float* C, int32_t mode, int32_t reseed, Workspace& ws, hipStream_t st) {
  UpdateBufs b;
  b.counts32 = ws.take<int32_t>(K);
  b.offsets = ws.take<int32_t>(K + 1);
  b.perm = ws.take<int32_t>(n);
  b.inv = ws.take<int32_t>(n);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  if (mode != HMOE_UPDATE_FINALIZE) {
    HMOE_TRY(update_core<T>(X, n, d, K, assign, d1, sums, counts64, mode == HMOE_UPDATE_ACCUMULATE,
                            mode == HMOE_UPDATE_FULL ? reseed : 0, b, ws, st));
  }
  if (mode != HMOE_UPDATE_ACCUMULATE) {
    HMOE_LAUNCH("finalize centres", (k_finalize<T, int64_t>), dim3((unsigned)cdiv((int64_t)K * d, 256)), dim3(256), 0, st, sums,
                       counts64, K, d, C, (T*)nullptr);
  }
  return HMOE_OK;
}

int launch_update(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t* assign,
                  const float* min_dist, double* sums, int64_t* counts, float* C, int32_t mode, int32_t reseed,
                  Workspace& ws, hipStream_t st) {
  if (dt == HMOE_BF16)
    return update_t<bf16>((const bf16*)X, n, d, K, assign, min_dist, sums, counts, C, mode, reseed, ws, st);
  return update_t<float>((const float*)X, n, d, K, assign, min_dist, sums, counts, C, mode, reseed, ws, st);
}

size_t update_ws_bytes(int64_t n, int32_t d, int32_t K) { return update_scratch(n, d, K); }

size_t fit_ws_bytes(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt) {
  Workspace ws(nullptr, 0);
  ws.take<double>((size_t)K * d);           // sums
  ws.take<int64_t>(K);                      // counts64
  ws.take<char>((size_t)K * d * dtype_size(dt));  // data-precision centres
  ws.take<float>(n);                        // min distances when the caller passes none
  ws.take<double>(n);                       // D^2 for k-means++
  ws.take<double>(cdiv(n, kKppRows));       // block sums
  ws.take<int32_t>(K);                      // picks when the caller passes none
  size_t s = ws.off + update_scratch(n, d, K) + assign_ws_bytes(n, K, dt) + 4096;
  return s;
}

size_t assign_ws(int64_t n, int32_t K, hmoe_dtype_t dt) { return assign_ws_bytes(n, K, dt) + 256; }

template <typename T>
static int fit_t(const T* X, int64_t n, int32_t d, int32_t K, int32_t n_iter, const double* u, int32_t reseed,
                 float* C, int32_t* assign, float* min_dist, int32_t* counts, double* objective, int32_t* init_idx,
                 Workspace& ws, hipStream_t st) {
  double* sums = ws.take<double>((size_t)K * d);
  int64_t* c64 = ws.take<int64_t>(K);
  T* Cd = reinterpret_cast<T*>(ws.take<char>((size_t)K * d * sizeof(T)));
  float* d1 = min_dist ? min_dist : ws.take<float>(n);
  double* D2 = ws.take<double>(n);
  const int nb = (int)cdiv(n, kKppRows);
  double* bsum = ws.take<double>(nb);
  int32_t* idx = init_idx ? init_idx : ws.take<int32_t>(K);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const int64_t Kd = (int64_t)K * d;
  const bool same = sizeof(T) == sizeof(float);  // fp32 data assigns against C itself
  const T* Cuse = same ? reinterpret_cast<const T*>(C) : Cd;
  if (u) {
    HMOE_LAUNCH("kmeans++ first", k_kpp_first, dim3(1), dim3(64), 0, st, u, n, idx);
    for (int t = 0; t < K; ++t) {
      HMOE_LAUNCH("kmeans++ D2", k_kpp_update<T>, dim3((unsigned)nb), dim3(256), 0, st, X, n, d, idx, t, D2, bsum);
      if (t + 1 < K) {
        HMOE_LAUNCH("kmeans++ select", k_kpp_select, dim3(1), dim3(1024), 0, st, D2, n, bsum, nb, u, t + 1, idx);
      }
    }
    HMOE_LAUNCH("gather centres", k_gather_centres<T>, dim3((unsigned)cdiv(Kd, 256)), dim3(256), 0, st, X, d, idx, K, C,
                       same ? (T*)nullptr : Cd);
  }
  if (!u && !same) {
    // data-precision copy of the given centres
    HMOE_LAUNCH("convert centres", (k_convert_centres<T>), dim3((unsigned)cdiv(Kd, 256)), dim3(256), 0, st, C, Kd, Cd);
  }
  UpdateBufs b;
  Workspace* wsp = &ws;
  b.counts32 = wsp->take<int32_t>(K);
  b.offsets = wsp->take<int32_t>(K + 1);
  b.perm = wsp->take<int32_t>(n);
  b.inv = wsp->take<int32_t>(n);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const size_t mark = ws.off;
  for (int t = 0; t <= n_iter; ++t) {
    ws.off = mark;
    HMOE_TRY(launch_assign(X, DT<T>::id, n, d, Cuse, K, assign, d1, ws, st));
    if (objective) HMOE_TRY(launch_sum_f32(d1, n, 1.0, objective + t, nullptr, ws, st));
    if (t == n_iter) break;
    HMOE_TRY(update_core<T>(X, n, d, K, assign, d1, sums, c64, 0, reseed, b, ws, st));
    HMOE_LAUNCH("finalize centres", (k_finalize<T, int64_t>), dim3((unsigned)cdiv(Kd, 256)), dim3(256), 0, st, sums, c64, K, d,
                       C, same ? (T*)nullptr : Cd);
  }
  if (counts) {
    ws.off = mark;
    HMOE_TRY(launch_dispatch(assign, n, K, counts, b.offsets, b.perm, b.inv, ws, st));
  }
  return HMOE_OK;
}

int launch_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t n_iter, const double* u,
               int32_t reseed, float* C, int32_t* assign, float* min_dist, int32_t* counts, double* objective,
               int32_t* init_idx, Workspace& ws, hipStream_t st) {
  if (dt == HMOE_BF16)
    return fit_t<bf16>((const bf16*)X, n, d, K, n_iter, u, reseed, C, assign, min_dist, counts, objective, init_idx,
                       ws, st);
  return fit_t<float>((const float*)X, n, d, K, n_iter, u, reseed, C, assign, min_dist, counts, objective, init_idx,
                      ws, st);
}

}  // namespace hmoe
