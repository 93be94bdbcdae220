// dispatch.hip -- hard routing: a stable counting sort of the batch by expert id (Section 2:
// each expert gets its own share of the data), and row gathers for dispatch / combine.
//
// Three passes over the int32 ids, all fixed-size blocks of 1024 ids (4 waves x 4 chunks of
// 64 lanes):
//   hist    per-wave bucket counts via ballot-built peer masks (lanes with the same id),
//           summed into block_counts[k][b];
//   colscan per expert (one wave each), exclusive prefix of block_counts[k][*] over blocks
//           -> counts[k];
//   offsets exclusive scan of counts (one block);
//           (for small problems colscan and offsets run as one single-workgroup kernel);
//   scatter recomputes the peer masks and writes each id's slot = offsets[k] + earlier blocks
//           + earlier waves + earlier chunks + rank among earlier peer lanes: the order of
//           equal ids is the sample order, so the permutation is unique.
// Ids outside [0, K) (an error of the caller's, which the device cannot report synchronously)
// go to one more bucket, K, after every expert: counts exclude them, offsets[K] stops before
// them, and perm / inv stay permutations of all n rows, so nothing downstream indexes outside
// its buffers.
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

constexpr int kIdsPerBlock = 1024;

// Peer mask: the valid lanes whose id equals this lane's id (ids < 2^bits).
__device__ __forceinline__ uint64_t peer_mask(int id, bool valid, int bits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < bits; ++b) {
    const bool bit = (id >> b) & 1;
    const uint64_t on = __ballot(valid && bit);
    m &= bit ? on : ~on;
  }
  return m;
}

__device__ __forceinline__ int lane_rank(uint64_t peers) {
  const int l = threadIdx.x & 63;
  const uint64_t lt = l == 0 ? 0ull : (~0ull >> (64 - l));
  return __popcll(peers & lt);
}

__device__ __forceinline__ void wave_hist(const int32_t* __restrict__ e, int64_t n, int K, int bits,
                                          int32_t* __restrict__ hist_w, int32_t* __restrict__ err) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int c = 0; c < 4; ++c) {
    const int64_t i = (int64_t)blockIdx.x * kIdsPerBlock + w * 256 + c * 64 + l;
    int id = i < n ? e[i] : -1;
    const bool valid = i < n;
    if (valid && (id < 0 || id >= K)) {
      if (err) atomicOr(err, 1);
      id = K;  // the bucket after every expert
    }
    const uint64_t peers = peer_mask(valid ? id : 0, valid, bits);
    if (valid && lane_rank(peers) == 0) atomicAdd(&hist_w[id], (int32_t)__popcll(peers));
  }
}

__global__ void __launch_bounds__(256) k_dispatch_hist(const int32_t* __restrict__ e, int64_t n, int K,
                                                       int bits, int32_t* __restrict__ block_counts,
                                                       int32_t* __restrict__ err) {
  extern __shared__ int32_t hist[];  // [4][K + 1]
  const int KB = K + 1;
  for (int k = threadIdx.x; k < 4 * KB; k += 256) hist[k] = 0;
  __syncthreads();
  wave_hist(e, n, K, bits, hist + (threadIdx.x >> 6) * KB, err);
  __syncthreads();
  for (int k = threadIdx.x; k < KB; k += 256)
    block_counts[(int64_t)k * gridDim.x + blockIdx.x] =
        hist[k] + hist[KB + k] + hist[2 * KB + k] + hist[3 * KB + k];
}

// Exclusive prefix over the blocks of block_counts[k][*] (in place) by one wave; returns the
// column's total (in every lane).  Lane l scans a contiguous run of the blocks, the runs are
// combined by a wave scan.
__device__ __forceinline__ int32_t wave_colscan(int32_t* __restrict__ col, int nb) {
  const int l = threadIdx.x & 63;
  const int per = (nb + 63) / 64;
  const int b0 = l * per;
  int32_t loc = 0;
  for (int q = 0; q < per; ++q)
    if (b0 + q < nb) loc += col[b0 + q];
  // wave exclusive scan of loc
  int32_t inc = loc;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const int32_t o = __shfl_up(inc, m, 64);
    if (l >= m) inc += o;
  }
  int32_t run = inc - loc;
  for (int q = 0; q < per; ++q)
    if (b0 + q < nb) {
      const int32_t t = col[b0 + q];
      col[b0 + q] = run;
      run += t;
    }
  return __shfl(inc, 63, 64);
}

// One wave per expert k: the column scan of block_counts[k][*] and counts[k] = its total.
// Buckets 0 .. K (K: the out-of-range ids); counts[k] is written for the K experts only.
__global__ void __launch_bounds__(256) k_dispatch_colscan(int32_t* __restrict__ block_counts, int nb, int K,
                                                          int32_t* __restrict__ counts) {
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (k > K) return;
  const int32_t total = wave_colscan(block_counts + (int64_t)k * nb, nb);
  if ((threadIdx.x & 63) == 0 && k < K) counts[k] = total;
}

__global__ void __launch_bounds__(1024) k_dispatch_offsets(const int32_t* __restrict__ counts, int K,
                                                           int32_t* __restrict__ offsets) {
  __shared__ int32_t sh[17];
  const int per = (K + 1023) / 1024;
  const int k0 = threadIdx.x * per;
  int32_t s = 0;
  for (int q = 0; q < per; ++q)
    if (k0 + q < K) s += counts[k0 + q];
  int32_t total;
  int32_t ex = block_excl_scan<int32_t>(s, sh, &total);
  for (int q = 0; q < per; ++q)
    if (k0 + q < K) {
      offsets[k0 + q] = ex;
      ex += counts[k0 + q];
    }
  if (threadIdx.x == 0) offsets[K] = total;
}

// The column scans and the offsets in one workgroup, for small problems ((K + 1) nb <=
// kScanSmall): wave j scans the columns k = j, j + 16, ..., the totals meet in LDS, and the
// workgroup's exclusive scan of them gives the offsets -- one launch instead of two.
constexpr int64_t kScanSmall = 1 << 16;
__global__ void __launch_bounds__(1024) k_dispatch_scan_small(int32_t* __restrict__ block_counts, int nb, int K,
                                                              int32_t* __restrict__ counts,
                                                              int32_t* __restrict__ offsets) {
  __shared__ int32_t s_cnt[4096];
  __shared__ int32_t sh[17];
  for (int k = threadIdx.x >> 6; k < K; k += 16) {
    const int32_t total = wave_colscan(block_counts + (int64_t)k * nb, nb);
    if ((threadIdx.x & 63) == 0) {
      counts[k] = total;
      s_cnt[k] = total;
    }
  }
  if ((threadIdx.x >> 6) == K % 16) wave_colscan(block_counts + (int64_t)K * nb, nb);  // the out-of-range bucket
  __syncthreads();
  const int per = (K + 1023) / 1024;
  const int k0 = threadIdx.x * per;
  int32_t s = 0;
  for (int q = 0; q < per; ++q)
    if (k0 + q < K) s += s_cnt[k0 + q];
  int32_t total;
  int32_t ex = block_excl_scan<int32_t>(s, sh, &total);
  for (int q = 0; q < per; ++q)
    if (k0 + q < K) {
      offsets[k0 + q] = ex;
      ex += s_cnt[k0 + q];
    }
  if (threadIdx.x == 0) offsets[K] = total;
}

__global__ void __launch_bounds__(256) k_dispatch_scatter(const int32_t* __restrict__ e, int64_t n, int K,
                                                          int bits, const int32_t* __restrict__ block_base,
                                                          const int32_t* __restrict__ offsets,
                                                          int32_t* __restrict__ perm,
                                                          int32_t* __restrict__ inv) {
  extern __shared__ int32_t hist[];  // [4][K + 1] -> per-wave running slot
  const int KB = K + 1;
  for (int k = threadIdx.x; k < 4 * KB; k += 256) hist[k] = 0;
  __syncthreads();
  const int w = threadIdx.x >> 6;
  wave_hist(e, n, K, bits, hist + w * KB, nullptr);
  __syncthreads();
  for (int k = threadIdx.x; k < KB; k += 256) {
    int32_t run = offsets[k] + block_base[(int64_t)k * gridDim.x + blockIdx.x];  // offsets[K]: past the experts
    for (int q = 0; q < 4; ++q) {
      const int32_t t = hist[q * KB + k];
      hist[q * KB + k] = run;
      run += t;
    }
  }
  __syncthreads();
  int32_t* slot_w = hist + w * KB;
  const int l = threadIdx.x & 63;
  for (int c = 0; c < 4; ++c) {
    const int64_t i = (int64_t)blockIdx.x * kIdsPerBlock + w * 256 + c * 64 + l;
    int id = i < n ? e[i] : -1;
    const bool valid = i < n;
    if (valid && (id < 0 || id >= K)) id = K;
    const uint64_t peers = peer_mask(valid ? id : 0, valid, bits);
    if (valid) {
      const int rank = lane_rank(peers);
      const int32_t slot = slot_w[id] + rank;
      perm[slot] = (int32_t)i;
      inv[i] = slot;
      // every peer has read slot_w[id] above (same wave, program order) before the leader
      // advances it for the next chunk
      if (rank == 0) atomicAdd(&slot_w[id], (int32_t)__popcll(peers));
    }
  }
}

static int id_bits(int K) {
  int b = 0;
  while ((1 << b) < K) ++b;
  return b;
}

size_t dispatch_ws(int64_t n, int32_t K) {
  Workspace ws(nullptr, 0);
  const int64_t nb = cdiv(n, kIdsPerBlock);
  ws.take<int32_t>((size_t)(nb > 0 ? nb : 1) * (K + 1));
  return ws.off;
}

int launch_dispatch(const int32_t* e, int64_t n, int32_t K, int32_t* counts, int32_t* offsets,
                    int32_t* perm, int32_t* inv, Workspace& ws, hipStream_t st) {
  const int64_t nb = cdiv(n, kIdsPerBlock);
  int32_t* bc = ws.take<int32_t>((size_t)(nb > 0 ? nb : 1) * (K + 1));
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const int bits = id_bits(K + 1);  // ids 0 .. K (K: out of range)
  const size_t lds = 4 * (size_t)(K + 1) * sizeof(int32_t);
  if (nb > 0) {
    HMOE_LAUNCH("dispatch hist", k_dispatch_hist, dim3((unsigned)nb), dim3(256), lds, st, e, n, K, bits, bc,
                       (int32_t*)nullptr);
  }
  if ((int64_t)(K + 1) * nb <= kScanSmall) {
    HMOE_LAUNCH("dispatch scan", k_dispatch_scan_small, dim3(1), dim3(1024), 0, st, bc, (int)nb, K, counts, offsets);
  } else {
    HMOE_LAUNCH("dispatch colscan", k_dispatch_colscan, dim3((unsigned)cdiv(K + 1, 4)), dim3(256), 0, st, bc,
                (int)nb, K, counts);
    HMOE_LAUNCH("dispatch offsets", k_dispatch_offsets, dim3(1), dim3(1024), 0, st, counts, K, offsets);
  }
  if (nb > 0) {
    HMOE_LAUNCH("dispatch scatter", k_dispatch_scatter, dim3((unsigned)nb), dim3(256), lds, st, e, n, K, bits, bc,
                       offsets, perm, inv);
  }
  return HMOE_OK;
}

int launch_permute(const void* in, void* out, const int32_t* index, int64_t n, int32_t w, hmoe_dtype_t dt,
                   hipStream_t st) {
  if (n == 0) return HMOE_OK;
  const int vpr = (int)(w * dtype_size(dt) / 16);
  const int64_t total = n * vpr;
  int64_t grid = cdiv(total, 256);
  if (grid > 8192) grid = 8192;
  HMOE_LAUNCH("permute rows", k_permute_rows, dim3((unsigned)grid), dim3(256), 0, st, (const i32x4*)in, (i32x4*)out,
                     index, n, vpr);
  return HMOE_OK;
}

int launch_seg_tiles(const int32_t* seg, int G, int tile, int32_t* tile_start, hipStream_t st) {
  HMOE_LAUNCH("segment tiles", k_seg_tiles, dim3(1), dim3(1024), 0, st, seg, G, tile, tile_start);
  return HMOE_OK;
}

int launch_seg_order(const int32_t* seg, int G, int32_t* order, hipStream_t st) {
  HMOE_LAUNCH("segment order", k_seg_order, dim3((unsigned)cdiv(G, 256)), dim3(256), 0, st, seg, G, order);
  return HMOE_OK;
}

template <typename T, typename O>
int launch_segsum(const T* X, int64_t ld, const int32_t* rowmap, const int32_t* seg, int G, int w,
                  int64_t n, O* out, int accumulate, Workspace& ws, hipStream_t st) {
  const int64_t pieces = cdiv(n, kSegPiece) + G;
  int32_t* ts = ws.take<int32_t>(G + 1);
  double* part = ws.take<double>((size_t)pieces * w);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  HMOE_TRY(launch_seg_tiles(seg, G, kSegPiece, ts, st));
  HMOE_LAUNCH("segsum partial", k_segsum_partial<T>, dim3((unsigned)pieces), dim3(256), 0, st, X, ld, rowmap, seg, ts, G,
                     w, part);
  HMOE_LAUNCH("segsum final", k_segsum_final<O>, dim3((unsigned)cdiv((int64_t)G * w, 256)), dim3(256), 0, st, part,
                     ts, G, w, out, accumulate);
  return HMOE_OK;
}

size_t segsum_ws(int64_t n, int G, int w) {
  Workspace ws(nullptr, 0);
  ws.take<int32_t>(G + 1);
  ws.take<double>((size_t)(cdiv(n, kSegPiece) + G) * w);
  return ws.off;
}

template int launch_segsum<float, double>(const float*, int64_t, const int32_t*, const int32_t*, int, int,
                                          int64_t, double*, int, Workspace&, hipStream_t);
template int launch_segsum<bf16, double>(const bf16*, int64_t, const int32_t*, const int32_t*, int, int,
                                         int64_t, double*, int, Workspace&, hipStream_t);
template int launch_segsum<float, float>(const float*, int64_t, const int32_t*, const int32_t*, int, int,
                                         int64_t, float*, int, Workspace&, hipStream_t);
template int launch_segsum<bf16, float>(const bf16*, int64_t, const int32_t*, const int32_t*, int, int,
                                        int64_t, float*, int, Workspace&, hipStream_t);

int launch_zero_f32(float* x, int64_t n, hipStream_t st) {
  if (n <= 0) return HMOE_OK;
  int64_t grid = cdiv(n, 256);
  if (grid > 4096) grid = 4096;
  HMOE_LAUNCH("zero", k_zero_f32, dim3((unsigned)grid), dim3(256), 0, st, x, n);
  return HMOE_OK;
}

int launch_sum_f32(const float* x, int64_t n, double scale, double* out_f64, float* out_f32, Workspace& ws,
                   hipStream_t st) {
  double* part = ws.take<double>(kSumBlocks);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  HMOE_LAUNCH("sum partial", k_sum_partial<float>, dim3(kSumBlocks), dim3(256), 0, st, x, n, part);
  if (out_f64) HMOE_LAUNCH("sum final", k_sum_final<double>, dim3(1), dim3(64), 0, st, part, scale, out_f64);
  if (out_f32) HMOE_LAUNCH("sum final", k_sum_final<float>, dim3(1), dim3(64), 0, st, part, scale, out_f32);
  return HMOE_OK;
}

}  // namespace hmoe
