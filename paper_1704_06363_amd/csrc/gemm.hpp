// gemm.hpp -- MFMA tile engine shared by every dense contraction of the hot path.
//
// C[m, n] = sum_k A(m, k) * B(n, k) over one 128 x 128 output tile per workgroup (256 threads,
// four 64-wide waves in a 2 x 2 grid, each wave 64 x 64).  Operands are staged through LDS
// in a "row-major, K-contiguous" layout whatever their layout in HBM:
//   K-contiguous operand  (stored [rows][K]): 16-byte vector loads go straight to LDS;
//   K-strided operand     (stored [K][rows]): each thread loads 4 K-rows of one 16-byte
//                         column chunk and transposes them in registers before the LDS store.
// bf16 uses v_mfma_f32_16x16x32_bf16 (8 consecutive k per lane); fp32 uses
// v_mfma_f32_16x16x4_f32, fed from the same 16-byte LDS reads (4 consecutive k per lane,
// consumed by 4 MFMAs).  Accumulation is fp32.  The K loop is double-buffered: the next
// stage's global loads are in flight while the current stage feeds the MFMAs.
//
// Accumulator ownership (verified layout of the 16x16 MFMA outputs): lane l of wave w holds,
// for sub-tile (i, j) and r = 0..3,
//   row = (w / 2) * 64 + 16 i + 4 (l / 16) + r,     col = (w % 2) * 64 + 16 j + (l % 16).
#pragma once
#include "common.hpp"

namespace hmoe {

constexpr int kBM = 128;
constexpr int kBN = 128;
constexpr int kThreads = 256;
constexpr int kStageRowBytes = 128;  // K extent of one stage, in bytes (64 bf16 or 32 fp32)
constexpr int kLdsStride = 144;      // padded LDS row stride (bytes): conflict-free b128 reads
constexpr int kOperandBytes = kBM * kLdsStride;
constexpr int kGemmLds = 4 * kOperandBytes;  // A and B, two stages each

template <typename T>
struct Elt {
  static constexpr int per_vec = 16 / sizeof(T);             // elements per 16-byte vector
  static constexpr int bk = kStageRowBytes / sizeof(T);      // K per stage
};

// ------------------------------------------------------------------ operand staging

// Loads one 128-row x (one stage of K) operand tile into registers.  `rows_valid` rows
// exist (others read as zero); K positions >= k_valid read as zero.
template <typename T, bool KCONTIG>
struct Stager {
  i32x4 v[4];

  // K-contiguous: element (r, k) at base + r * ld + k.  k_valid must be a multiple of the
  // vector width (checked by the host).
  // K-strided:    element (r, k) at base + k * ld + r.  rows_valid must be a multiple of the
  // vector width.
  __device__ __forceinline__ void load(const T* __restrict__ base, int64_t ld, int rows_valid,
                                       int k0, int k_valid) {
    const int t = threadIdx.x;
    constexpr int EPV = Elt<T>::per_vec;
    if constexpr (KCONTIG) {
      const int vc = t & 7;
      const int k = k0 + vc * EPV;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = (t >> 3) + 32 * q;
        if (r < rows_valid && k < k_valid)
          v[q] = *reinterpret_cast<const i32x4*>(base + (int64_t)r * ld + k);
        else
          v[q] = i32x4{0, 0, 0, 0};
      }
    } else {
      constexpr int CHUNKS = kBM / EPV;  // 16 (bf16) or 32 (fp32) column chunks
      const int rc = t % CHUNKS;
      const int kq = t / CHUNKS;         // 0..15 (bf16) or 0..7 (fp32): 4 K-rows each
      const int r = rc * EPV;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = k0 + 4 * kq + q;
        if (r < rows_valid && k < k_valid)
          v[q] = *reinterpret_cast<const i32x4*>(base + (int64_t)k * ld + r);
        else
          v[q] = i32x4{0, 0, 0, 0};
      }
    }
  }

  __device__ __forceinline__ void store(char* lds) const {
    const int t = threadIdx.x;
    if constexpr (KCONTIG) {
      const int vc = t & 7;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = (t >> 3) + 32 * q;
        *reinterpret_cast<i32x4*>(lds + r * kLdsStride + vc * 16) = v[q];
      }
    } else if constexpr (sizeof(T) == 2) {
      // v[q] holds 8 bf16 of K-row q; row r' of the tile gets (v[0][r'], .., v[3][r']).
      const int rc = t % 16, kq = t / 16;
      const uint16_t* s0 = reinterpret_cast<const uint16_t*>(&v[0]);
      const uint16_t* s1 = reinterpret_cast<const uint16_t*>(&v[1]);
      const uint16_t* s2 = reinterpret_cast<const uint16_t*>(&v[2]);
      const uint16_t* s3 = reinterpret_cast<const uint16_t*>(&v[3]);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        uint32_t lo = (uint32_t)s0[rr] | ((uint32_t)s1[rr] << 16);
        uint32_t hi = (uint32_t)s2[rr] | ((uint32_t)s3[rr] << 16);
        uint2 w = make_uint2(lo, hi);
        *reinterpret_cast<uint2*>(lds + (rc * 8 + rr) * kLdsStride + kq * 8) = w;
      }
    } else {
      const int rc = t % 32, kq = t / 32;
      const floatx4 s0 = __builtin_bit_cast(floatx4, v[0]);
      const floatx4 s1 = __builtin_bit_cast(floatx4, v[1]);
      const floatx4 s2 = __builtin_bit_cast(floatx4, v[2]);
      const floatx4 s3 = __builtin_bit_cast(floatx4, v[3]);
      const floatx4 w0 = {s0[0], s1[0], s2[0], s3[0]};
      const floatx4 w1 = {s0[1], s1[1], s2[1], s3[1]};
      const floatx4 w2 = {s0[2], s1[2], s2[2], s3[2]};
      const floatx4 w3 = {s0[3], s1[3], s2[3], s3[3]};
      char* dst = lds + (rc * 4) * kLdsStride + kq * 16;
      *reinterpret_cast<floatx4*>(dst) = w0;
      *reinterpret_cast<floatx4*>(dst + kLdsStride) = w1;
      *reinterpret_cast<floatx4*>(dst + 2 * kLdsStride) = w2;
      *reinterpret_cast<floatx4*>(dst + 3 * kLdsStride) = w3;
    }
  }
};

// ------------------------------------------------------------------ MFMA step

template <typename T>
__device__ __forceinline__ void mfma_stage(const char* ldsA, const char* ldsB,
                                           floatx4 (&acc)[4][4]) {
  const int l = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int lr = l & 15, lg = l >> 4;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    i32x4 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = *reinterpret_cast<const i32x4*>(ldsA + (wm * 64 + 16 * i + lr) * kLdsStride + c * 64 + lg * 16);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = *reinterpret_cast<const i32x4*>(ldsB + (wn * 64 + 16 * j + lr) * kLdsStride + c * 64 + lg * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (sizeof(T) == 2) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
        } else {
          const floatx4 af = __builtin_bit_cast(floatx4, a[i]);
          const floatx4 bf = __builtin_bit_cast(floatx4, b[j]);
#pragma unroll
          for (int s = 0; s < 4; ++s)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s], bf[s], acc[i][j], 0, 0, 0);
        }
      }
    }
  }
}

// Full K loop for one tile.  A rows [0, a_rows), B rows [0, b_rows), K positions [0, k_len).
// With ROWNORM (K-contiguous A only) xs[q] accumulates the squared norm of the part of A
// row (threadIdx.x >> 3) + 32 q that this thread staged; the 8 lanes sharing a row together
// hold the full norm.
template <typename T>
__device__ __forceinline__ void add_sq(const i32x4 (&v)[4], float* xs) {
  constexpr int EPV = Elt<T>::per_vec;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const T* e = reinterpret_cast<const T*>(&v[q]);
#pragma unroll
    for (int z = 0; z < EPV; ++z) {
      const float f = to_f32(e[z]);
      xs[q] += f * f;
    }
  }
}

template <typename T, bool A_KC, bool B_KC, bool ROWNORM = false>
__device__ __forceinline__ void gemm_tile(const T* __restrict__ A, int64_t lda, int a_rows,
                                          const T* __restrict__ B, int64_t ldb, int b_rows,
                                          int k_len, char* smem, floatx4 (&acc)[4][4],
                                          float* xs = nullptr) {
  static_assert(!ROWNORM || A_KC, "row norms need a K-contiguous A");
  if constexpr (ROWNORM) {
#pragma unroll
    for (int q = 0; q < 4; ++q) xs[q] = 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  constexpr int BK = Elt<T>::bk;
  const int nk = (int)cdiv(k_len, BK);
  if (nk == 0) return;
  Stager<T, A_KC> sa;
  Stager<T, B_KC> sb;
  char* bufA[2] = {smem, smem + kOperandBytes};
  char* bufB[2] = {smem + 2 * kOperandBytes, smem + 3 * kOperandBytes};
  sa.load(A, lda, a_rows, 0, k_len);
  sb.load(B, ldb, b_rows, 0, k_len);
  if constexpr (ROWNORM) add_sq<T>(sa.v, xs);
  sa.store(bufA[0]);
  sb.store(bufB[0]);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      sa.load(A, lda, a_rows, (kt + 1) * BK, k_len);
      sb.load(B, ldb, b_rows, (kt + 1) * BK, k_len);
    }
    mfma_stage<T>(bufA[cur], bufB[cur], acc);
    if (more) {
      if constexpr (ROWNORM) add_sq<T>(sa.v, xs);
      sa.store(bufA[cur ^ 1]);
      sb.store(bufB[cur ^ 1]);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ tile scheduling

// Which output tile a workgroup owns.
struct TileCoord {
  int group;      // expert id (0 for ungrouped problems)
  int64_t m0;     // first output row (global, in the row space of A / C)
  int m_rows;     // valid rows in this tile (<= 128)
  int n0;         // first output column
  int n_cols;     // valid columns (<= 128)
  int64_t k0;     // first reduction index (grouped-K problems)
  int k_len;      // reduction length
  bool valid;
};

// Plain problem: M x N tiles, bands of `band` m-tiles walked m-fastest so that concurrently
// running workgroups share both operand tiles in the caches.
__device__ __forceinline__ TileCoord tile_plain(int64_t M, int N, int K) {
  TileCoord tc;
  const int64_t mt = cdiv(M, kBM);
  const int nt = (int)cdiv(N, kBN);
  const int64_t b = blockIdx.x;
  constexpr int band = 16;
  const int64_t band_tiles = (int64_t)band * nt;
  const int64_t g = b / band_tiles;
  const int64_t in = b - g * band_tiles;
  const int64_t m_first = g * band;
  const int64_t bm = (mt - m_first < band) ? (mt - m_first) : band;
  const int64_t mi = m_first + in % bm;
  const int ni = (int)(in / bm);
  tc.group = 0;
  tc.m0 = mi * kBM;
  tc.n0 = ni * kBN;
  tc.valid = (mi < mt) && (ni < nt);
  tc.m_rows = (int)((M - tc.m0) < kBM ? (M - tc.m0) : kBM);
  tc.n_cols = (N - tc.n0) < kBN ? (N - tc.n0) : kBN;
  tc.k0 = 0;
  tc.k_len = K;
  return tc;
}

// Row-grouped problem (experts' forward / input-gradient GEMMs): group e owns rows
// [seg[e], seg[e+1]) of A and C.  tile_start[e] = number of m-tiles of groups < e (prefix,
// tile_start[G] = total).  Launched over an upper bound of m-tiles x n-tiles; the excess
// workgroups find no tile and exit.
__device__ __forceinline__ TileCoord tile_group_m(const int32_t* __restrict__ seg,
                                                  const int32_t* __restrict__ tile_start, int G,
                                                  int N, int K) {
  TileCoord tc;
  const int nt = (int)cdiv(N, kBN);
  const int64_t b = blockIdx.x;
  const int64_t mtile = b / nt;
  const int ni = (int)(b - mtile * nt);
  tc.valid = false;
  const int total = tile_start[G];
  if (mtile >= total) return tc;
  int lo = 0, hi = G - 1;  // last e with tile_start[e] <= mtile
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (tile_start[mid] <= mtile) lo = mid; else hi = mid - 1;
  }
  const int e = lo;
  const int64_t local = mtile - tile_start[e];
  const int64_t rows = seg[e + 1] - seg[e];
  tc.group = e;
  tc.m0 = seg[e] + local * kBM;
  tc.m_rows = (int)((rows - local * kBM) < kBM ? (rows - local * kBM) : kBM);
  tc.n0 = ni * kBN;
  tc.n_cols = (N - tc.n0) < kBN ? (N - tc.n0) : kBN;
  tc.k0 = 0;
  tc.k_len = K;
  tc.valid = tc.m_rows > 0;
  return tc;
}

// Reduction-grouped problem (experts' weight gradients): group e reduces over the rows
// [seg[e], seg[e+1]) of both operands; output tile (m, n) of group e.
__device__ __forceinline__ TileCoord tile_group_k(const int32_t* __restrict__ seg, int G, int M,
                                                  int N) {
  TileCoord tc;
  const int mt = (int)cdiv(M, kBM), nt = (int)cdiv(N, kBN);
  const int64_t b = blockIdx.x;
  const int per = mt * nt;
  const int e = (int)(b / per);
  const int in = (int)(b - (int64_t)e * per);
  const int mi = in / nt, ni = in % nt;
  tc.group = e;
  tc.valid = e < G;
  tc.m0 = (int64_t)mi * kBM;
  tc.m_rows = (M - mi * kBM) < kBM ? (M - mi * kBM) : kBM;
  tc.n0 = ni * kBN;
  tc.n_cols = (N - tc.n0) < kBN ? (N - tc.n0) : kBN;
  if (tc.valid) {
    tc.k0 = seg[e];
    tc.k_len = seg[e + 1] - seg[e];
  } else {
    tc.k0 = 0;
    tc.k_len = 0;
  }
  return tc;
}

// ------------------------------------------------------------------ epilogue helpers

struct Frag {
  int wm, wn, lr, lg;
  __device__ __forceinline__ Frag() {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    wm = w >> 1;
    wn = w & 1;
    lr = l & 15;
    lg = l >> 4;
  }
  __device__ __forceinline__ int row(int i, int r) const { return wm * 64 + 16 * i + 4 * lg + r; }
  __device__ __forceinline__ int col(int j) const { return wn * 64 + 16 * j + lr; }
};

}  // namespace hmoe
