// primitives.hpp -- small device building blocks used by several launchers: block scans,
// segment tiling, deterministic segmented column sums, row permutation, fixed-order sums.
#pragma once
#include "common.hpp"

namespace hmoe {

// Inclusive scan across one wavefront.
template <typename V>
__device__ __forceinline__ V wave_incl_scan(V v) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    V t = __shfl_up(v, o, 64);
    if (l >= o) v += t;
  }
  return v;
}

// Exclusive scan across the block (blockDim.x a multiple of 64, <= 1024); returns the
// exclusive prefix of v and writes the block total to *total.  `sh` holds >= 16 V.
template <typename V>
__device__ __forceinline__ V block_excl_scan(V v, V* sh, V* total) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  V inc = wave_incl_scan(v);
  if (l == 63) sh[w] = inc;
  __syncthreads();
  if (w == 0) {
    V s = (l < nw) ? sh[l] : V(0);
    V si = wave_incl_scan(s);
    if (l < nw) sh[l] = si - s;  // exclusive wave offsets
    if (l == nw - 1) sh[16] = si;
  }
  __syncthreads();
  V res = sh[w] + inc - v;
  *total = sh[16];
  __syncthreads();
  return res;
}

// tile_start[e] = sum_{e' < e} ceil((seg[e'+1] - seg[e']) / tile), e = 0..G.  One block of
// 1024 threads; G <= 4096.
static __global__ void __launch_bounds__(1024) k_seg_tiles(const int32_t* __restrict__ seg, int G, int tile,
                                                    int32_t* __restrict__ tile_start) {
  __shared__ int32_t sh[17];
  const int per = (G + 1023) / 1024;
  const int e0 = threadIdx.x * per;
  int32_t loc[4];
  int32_t s = 0;
  for (int q = 0; q < per && q < 4; ++q) {
    const int e = e0 + q;
    int32_t c = 0;
    if (e < G) c = (seg[e + 1] - seg[e] + tile - 1) / tile;
    loc[q] = c;
    s += c;
  }
  int32_t total;
  int32_t ex = block_excl_scan<int32_t>(s, sh, &total);
  for (int q = 0; q < per && q < 4; ++q) {
    const int e = e0 + q;
    if (e < G) tile_start[e] = ex;
    ex += loc[q];
  }
  if (threadIdx.x == 0) tile_start[G] = total;
}

// order[r] = the segment of rank r when segments are ranked by length, longest first, equal
// lengths by lower index (a stable descending sort, so `order` is a permutation of 0..G-1).
// Each thread ranks one segment against all G lengths, staged through LDS 256 at a time.
static __global__ void __launch_bounds__(256) k_seg_order(const int32_t* __restrict__ seg, int G,
                                                        int32_t* __restrict__ order) {
  __shared__ int32_t len_s[256];
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int32_t mine = e < G ? seg[e + 1] - seg[e] : 0;
  int rank = 0;
  for (int f0 = 0; f0 < G; f0 += 256) {
    const int f = f0 + threadIdx.x;
    __syncthreads();
    len_s[threadIdx.x] = f < G ? seg[f + 1] - seg[f] : 0;
    __syncthreads();
    const int m = (G - f0) < 256 ? (G - f0) : 256;
    for (int q = 0; q < m; ++q) {
      const int32_t c = len_s[q];
      rank += (c > mine) || (c == mine && f0 + q < e);
    }
  }
  if (e < G) order[rank] = e;
}

// Finds the segment owning global piece b: last e with tile_start[e] <= b (e < G).
__device__ __forceinline__ int find_segment(const int32_t* __restrict__ tile_start, int G, int64_t b) {
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (tile_start[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// ------------------------------------------------------------------ segmented column sums
//
// out[e][j] = sum over rows p in [seg[e], seg[e+1]) of X[rowmap ? rowmap[p] : p][j], computed
// deterministically: pieces of at most kSegPiece rows are summed in fp64 in row order, then
// the pieces of each segment are added in a fixed order (k_segsum_final).

constexpr int kSegPiece = 256;
constexpr int kSegMaxVec = 4;  // vectors per thread: w <= 1024 * 16 / sizeof(T)

template <typename T>
__global__ void __launch_bounds__(256) k_segsum_partial(const T* __restrict__ X, int64_t ld,
                                                        const int32_t* __restrict__ rowmap,
                                                        const int32_t* __restrict__ seg,
                                                        const int32_t* __restrict__ tile_start, int G,
                                                        int w, double* __restrict__ part) {
  constexpr int EPV = 16 / sizeof(T);
  __shared__ double red[256 * EPV];
  const int64_t b = blockIdx.x;
  if (b >= tile_start[G]) return;
  const int e = find_segment(tile_start, G, b);
  const int64_t r0 = seg[e] + (b - tile_start[e]) * kSegPiece;
  const int64_t r1 = (r0 + kSegPiece < seg[e + 1]) ? r0 + kSegPiece : seg[e + 1];
  const int VPR = w / EPV;
  const int t = threadIdx.x;
  const int RG = VPR >= 256 ? 1 : 256 / VPR;
  const int rg = VPR >= 256 ? 0 : t / VPR;
  const int v0 = VPR >= 256 ? t : t % VPR;
  __shared__ int64_t rows_s[kSegPiece];  // the piece's source rows, staged once
  for (int64_t p = r0 + t; p < r1; p += 256) rows_s[p - r0] = rowmap ? rowmap[p] : p;
  __syncthreads();
  double acc[kSegMaxVec][EPV];
#pragma unroll
  for (int q = 0; q < kSegMaxVec; ++q)
#pragma unroll
    for (int z = 0; z < EPV; ++z) acc[q][z] = 0.0;
  if (rg < RG) {
    // rows in groups of U (loads of the group in flight together), added in row order
    constexpr int U = 4;
    const int cnt = (int)(r1 - r0);
    for (int p0 = rg; p0 < cnt; p0 += U * RG) {
#pragma unroll
      for (int q = 0; q < kSegMaxVec; ++q) {
        const int v = v0 + q * 256;
        if (!(v < VPR && (q == 0 || VPR > 256))) continue;
        i32x4 raw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int p = p0 + u * RG;
          if (p < cnt) raw[u] = *reinterpret_cast<const i32x4*>(X + rows_s[p] * ld + v * EPV);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (p0 + u * RG >= cnt) break;
          const T* e8 = reinterpret_cast<const T*>(&raw[u]);
#pragma unroll
          for (int z = 0; z < EPV; ++z) acc[q][z] += (double)to_f32(e8[z]);
        }
      }
    }
  }
  double* dst = part + b * (int64_t)w;
  if (RG == 1) {
#pragma unroll
    for (int q = 0; q < kSegMaxVec; ++q) {
      const int v = v0 + q * 256;
      if (v < VPR && (q == 0 || VPR > 256))
#pragma unroll
        for (int z = 0; z < EPV; ++z) dst[v * EPV + z] = acc[q][z];
    }
    return;
  }
  // Row groups hold partial sums of the same columns: add them in group order.
  if (rg < RG)
#pragma unroll
    for (int z = 0; z < EPV; ++z) red[t * EPV + z] = acc[0][z];
  __syncthreads();
  if (t < VPR) {
    for (int z = 0; z < EPV; ++z) {
      double s = 0.0;
      for (int g = 0; g < RG; ++g) s += red[(g * VPR + t) * EPV + z];
      dst[t * EPV + z] = s;
    }
  }
}

// out[e][j] (=, or += when accumulate) sum of the pieces of segment e in a fixed order: the
// segment's piece number m goes to partial sum m % 8 (each summed in piece order), then the 8
// partials are added pairwise -- 8 independent chains keep the loads in flight.
template <typename O>
__global__ void __launch_bounds__(256) k_segsum_final(const double* __restrict__ part,
                                                      const int32_t* __restrict__ tile_start, int G,
                                                      int w, O* __restrict__ out, int accumulate) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)G * w) return;
  const int e = (int)(idx / w), j = (int)(idx % w);
  const int32_t q0 = tile_start[e], q1 = tile_start[e + 1];
  double p[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int32_t q = q0;
  for (; q + 8 <= q1; q += 8)
#pragma unroll
    for (int u = 0; u < 8; ++u) p[u] += part[(int64_t)(q + u) * w + j];
#pragma unroll
  for (int u = 0; u < 8; ++u)
    if (q + u < q1) p[u] += part[(int64_t)(q + u) * w + j];
  const double s = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
  if (accumulate) out[idx] = (O)((double)out[idx] + s);
  else out[idx] = (O)s;
}

// ------------------------------------------------------------------ row permutation

// out[r] = in[index[r]] for rows of `vpr` 16-byte vectors; a negative index writes zeros.
static __global__ void __launch_bounds__(256) k_permute_rows(const i32x4* __restrict__ in,
                                                      i32x4* __restrict__ out,
                                                      const int32_t* __restrict__ index, int64_t n,
                                                      int vpr) {
  const int64_t total = n * vpr;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += stride) {
    const int64_t r = q / vpr;
    const int v = (int)(q - r * vpr);
    const int32_t s = index[r];
    // in has n rows too; an index outside [0, n) gives a zero row instead of a stray read
    out[q] = (uint32_t)s < (uint64_t)n ? in[(int64_t)s * vpr + v] : i32x4{0, 0, 0, 0};
  }
}

// ------------------------------------------------------------------ fill

// x[0 .. n) = 0 (fp32).  A kernel rather than a memset so that calls stay graph-capturable.
static __global__ void __launch_bounds__(256) k_zero_f32(float* __restrict__ x, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) x[i] = 0.f;
}

// ------------------------------------------------------------------ fixed-order sums

constexpr int kSumBlocks = 256;

// part[b] = sum of x over the contiguous slice b of kSumBlocks equal slices (fp64).
template <typename S>
__global__ void __launch_bounds__(256) k_sum_partial(const S* __restrict__ x, int64_t n,
                                                     double* __restrict__ part) {
  __shared__ double sh[4];
  const int64_t per = (n + kSumBlocks - 1) / kSumBlocks;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  double s = 0.0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256) s += (double)x[i];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = sh[0] + sh[1] + sh[2] + sh[3];
}

// *out = scale * sum of part[0 .. kSumBlocks) (as fp64 or fp32 per O).
template <typename O>
__global__ void __launch_bounds__(64) k_sum_final(const double* __restrict__ part, double scale,
                                                  O* __restrict__ out) {
  double s = 0.0;
  for (int i = threadIdx.x; i < kSumBlocks; i += 64) s += part[i];
  s = wave_sum(s);
  if (threadIdx.x == 0) *out = (O)(s * scale);
}

}  // namespace hmoe
