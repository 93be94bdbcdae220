// metrics.hip -- the inference tail of Section 4.4: t_m, the m largest logits of every row
// (the softmax keeps their order, so these are the m most probable tags), and the counts
// behind p@m (Eq. 4) and q@m (Eq. 5) for every m' <= m.
//
// k_topm (plain logits): one wave per row; each lane keeps its own m largest entries in a
// register list sorted by (value desc, index asc), and the m results are taken in m rounds of
// a wave-wide (value desc, index asc) maximum over the lists' heads, the lane holding the
// winner dropping it.  Lane l reads the row's 16-byte vectors l, l + 64, ... (so it sees its
// entries in increasing index order, and an entry enters only when strictly greater than the
// list's last, which keeps equal values in increasing index order), and only when it is not
// below a wave-wide bound on the row's m-th value (the m-th largest of the lanes' maxima).
// The row is read once: the kernel is bound by HBM.
// k_topm_anchored (logits stored as offsets <= 0 from per-row anchors, one per 64 columns, as
// the forward writes them; an entry is anchor + offset formed in fp32), one lane per row and
// four waves per 64 rows: a block's anchor bounds all its entries, so the row's anchors (a few
// KB) are read and only the blocks whose anchor can reach the row's m-th entry -- about m
// blocks of 64 columns when every anchor is its block's maximum.
//
// k_topm_hits: one thread per row (p) and per draw (q); the rank of each matching tag in the
// top-m list adds 1 to every m' above it.  Integer counts, summed through LDS and then with
// one 64-bit atomic per block and m' -- integer sums, so the result does not depend on order.
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

// Carries entry (cv, ci) down the list ordered by (value desc, index asc): it goes before the
// first entry it ranks above, and each entry it displaces is carried on by the same order.
template <int M>
__device__ __forceinline__ void list_carry(float (&lv)[M], int (&li)[M], float cv, int ci) {
#pragma unroll
  for (int k = 0; k < M; ++k) {
    const bool gt = cv > lv[k] || (cv == lv[k] && ci < li[k]);
    const float tv = lv[k];
    const int ti = li[k];
    lv[k] = gt ? cv : tv;
    li[k] = gt ? ci : ti;
    cv = gt ? tv : cv;
    ci = gt ? ti : ci;
  }
}

// The m largest entries of the union of the lanes' lists, in (value desc, index asc) order.
template <int M>
__device__ __forceinline__ void emit_topm(float (&lv)[M], int (&li)[M], int m, int l, int64_t row,
                                          int32_t* __restrict__ idx, float* __restrict__ val) {
  for (int q = 0; q < m; ++q) {
    float bv = lv[0];
    int bi = li[0];
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
      const float ov = shfl_xor(bv, s);
      const int oi = shfl_xor(bi, s);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (li[0] == bi) {  // this lane's head won: drop it
#pragma unroll
      for (int k = 0; k < M - 1; ++k) {
        lv[k] = lv[k + 1];
        li[k] = li[k + 1];
      }
      lv[M - 1] = -INFINITY;
      li[M - 1] = 0x7fffffff;
    }
    if (l == 0) {
      idx[row * (int64_t)m + q] = bi;
      if (val) val[row * (int64_t)m + q] = bv;
    }
  }
}

template <typename T, int M>
__global__ void __launch_bounds__(256) k_topm(const T* __restrict__ L, int64_t n, int V, int m,
                                              int32_t* __restrict__ idx, float* __restrict__ val) {
  constexpr int EPV = 16 / sizeof(T);
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= n) return;
  float lv[M];
  int li[M];
#pragma unroll
  for (int k = 0; k < M; ++k) {
    lv[k] = -INFINITY;
    li[k] = 0x7fffffff;
  }
  const T* r = L + row * (int64_t)V;
  const int nvec = V / EPV;
  // Wave-wide lower bound on the row's m-th largest value (the m-th largest of the lanes'
  // maxima: m entries are at least that large), so an entry below thr is not in t_m (entries
  // equal to it may be, and stay).  It closes in on the m-th value within a few steps, which
  // keeps the insertion branch -- taken by the wave when any lane takes it -- rare.
  float thr = -INFINITY;
  constexpr int U = 4;  // vectors in flight per lane
  // the trip count is the same for every lane (the bound is a wave-wide shuffle reduction)
  int step = 0;
  for (int b0 = 0; b0 < nvec; b0 += 64 * U, ++step) {
    i32x4 raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = b0 + 64 * u + l;
      if (v < nvec) raw[u] = *reinterpret_cast<const i32x4*>(r + (int64_t)v * EPV);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = b0 + 64 * u + l;
      if (v >= nvec) break;
      const T* e = reinterpret_cast<const T*>(&raw[u]);
      float f[EPV];
      float vmax = -INFINITY;
#pragma unroll
      for (int z = 0; z < EPV; ++z) {
        f[z] = to_f32(e[z]);
        vmax = fmaxf(vmax, f[z]);
      }
      if (!(vmax >= thr && vmax > lv[M - 1])) continue;  // the common case: nothing here enters
#pragma unroll
      for (int z = 0; z < EPV; ++z)
        if (f[z] >= thr && f[z] > lv[M - 1]) list_carry(lv, li, f[z], v * EPV + z);
    }
    // the m-th largest of the lanes' maxima: m lanes each hold an entry at least that large
    // (refreshed on the first steps, then every 4th: it settles quickly, and any value it
    // took is a valid bound)
    if (step >= 4 && (step & 3) != 0) continue;
    float x = lv[0];
    float t = -INFINITY;
    for (int q = 0; q < m; ++q) {
      t = wave_max(x);
      const uint64_t hit = __ballot(x == t);
      if (l == __ffsll((unsigned long long)hit) - 1) x = -INFINITY;  // drop one holder
    }
    thr = t;
  }
  emit_topm(lv, li, m, l, row, idx, val);
}

constexpr int kTopmRows = 64;  // rows per workgroup (one per lane; four waves split the tiles)

// The first m entries, in (value desc, index asc) order, of the union of the four sorted lists
// of this lane's row held in LDS ([wave][k][lane]; si NULL: values only): the m-th value is
// returned, and with gi given the m entries are written to gi[0 .. m) (and gv).
template <int M>
__device__ __forceinline__ float merge4(const float* sv, const int32_t* si, int m, int l,
                                        int32_t* __restrict__ gi = nullptr, float* __restrict__ gv = nullptr) {
  int h[4] = {0, 0, 0, 0};
  float v = -INFINITY;
  for (int q = 0; q < m; ++q) {
    float bv = -INFINITY;
    int bi = 0x7fffffff, bw = -1;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (h[w] >= M) continue;
      const float cv = sv[(w * M + h[w]) * kTopmRows + l];
      const int ci = si ? si[(w * M + h[w]) * kTopmRows + l] : 0;
      if (bw < 0 || cv > bv || (cv == bv && ci < bi)) {
        bv = cv;
        bi = ci;
        bw = w;
      }
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) h[w] += (w == bw);
    v = bv;
    if (gi) gi[q] = bi;
    if (gv) gv[q] = bv;
  }
  return v;
}

// Reads block b of a row (64 columns from r) and offers its entries >= lo, formed as anchor a
// + stored value in fp32, to the (value desc, index asc) list; cnt counts the entries that
// enter.  Nothing is read when `take` is false.
template <typename T, int M>
__device__ __forceinline__ void topm_block(const T* __restrict__ r, int V, int b, float a, float lo, bool take,
                                           float (&lv)[M], int (&li)[M], int& cnt) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int VPB = kAnchorCols / EPV;
  const int c0 = b * kAnchorCols;
  i32x4 raw[VPB];
#pragma unroll
  for (int v = 0; v < VPB; ++v)
    if (take && c0 + v * EPV < V) raw[v] = *reinterpret_cast<const i32x4*>(r + c0 + v * EPV);
  if (!take) return;
  auto offer = [&](const i32x4& x, int cv0) {
    const T* e = reinterpret_cast<const T*>(&x);
#pragma unroll
    for (int z = 0; z < EPV; ++z) {
      const float cv = a + to_f32(e[z]);
      if (cv >= lo && (cv > lv[M - 1] || (cv == lv[M - 1] && cv0 + z < li[M - 1]))) {
        list_carry(lv, li, cv, cv0 + z);
        ++cnt;
      }
    }
  };
  if constexpr (M <= 4) {
#pragma unroll
    for (int v = 0; v < VPB; ++v)
      if (c0 + v * EPV < V) offer(raw[v], c0 + v * EPV);  // V is a multiple of 8: vectors are whole
  } else {
    // longer lists: one vector per trip, picked by selects.  Fully unrolled, the insertion code
    // of a block is (64 entries x M steps) long: it compiled for minutes per list length, and
    // past 12 entries the unroller gave up and indexed the vectors through scratch memory.
#pragma unroll 1
    for (int v = 0; v < VPB; ++v) {
      if (c0 + v * EPV >= V) break;
      i32x4 x = raw[0];
#pragma unroll
      for (int vv = 1; vv < VPB; ++vv) x = v == vv ? raw[vv] : x;
      offer(x, c0 + v * EPV);
    }
  }
}

// One pass over this lane's tiles reading every block whose anchor is >= lo when `on`.
template <typename T, int M, int TU>
__device__ __forceinline__ void topm_scan(const T* __restrict__ r, const floatx4* __restrict__ arow, int64_t n,
                                          int V, int nb, int nt, int w, float lo, bool on, float (&lv)[M],
                                          int (&li)[M], int& cnt) {
  for (int t0 = w; t0 < nt; t0 += 4 * TU) {
    floatx4 q[TU];
#pragma unroll
    for (int u = 0; u < TU; ++u)
      if (t0 + 4 * u < nt) q[u] = arow[(int64_t)(t0 + 4 * u) * n];
    uint32_t mark = 0u;
#pragma unroll
    for (int u = 0; u < TU; ++u)
#pragma unroll
      for (int sl = 0; sl < 4; ++sl)
        if (on && t0 + 4 * u < nt && (t0 + 4 * u) * 4 + sl < nb && q[u][sl] >= lo) mark |= 1u << (4 * u + sl);
    while (mark) {
      const int k = __ffs(mark) - 1;
      mark &= mark - 1u;
      float a = q[0][0];  // the block's anchor, selected without indexing the registers
#pragma unroll
      for (int kk = 1; kk < 4 * TU; ++kk) a = k == kk ? q[kk / 4][kk % 4] : a;
      topm_block<T, M>(r, V, (t0 + 4 * (k / 4)) * 4 + k % 4, a, lo, true, lv, li, cnt);
    }
  }
}

// Anchored logits.  Block b (columns [64 b, 64 b + 64)) of row i has its anchor at
// anc[((b / 4) n + i) 4 + b % 4], and every entry of it is at most that anchor; the four
// anchors of a 256-column tile are one 16-byte vector.  A workgroup takes 64 rows, one per
// lane, and its four waves split each row's tiles (wave w takes tiles w, w + 4, ...), so one
// load instruction reads 1 KB of consecutive anchors.  Each lane keeps sorted register lists
// over its share; the four shares of a row meet in LDS, where every lane merges them.
//   1. Each lane keeps its m largest anchors with their blocks; merged, a_m = the row's m-th
//      largest anchor (with multiplicity).  Every entry >= a_m lies in a block with anchor >=
//      a_m, and those blocks are in the lanes' lists -- unless a lane's list ends at a_m and
//      it dropped a block (then an anchor equal to a_m may be missing from its list, and the
//      row rescans its anchors).
//   2. The blocks with anchor >= a_m are read and their entries >= a_m enter the (value desc,
//      index asc) lists of the row.  If the row has at least m such entries, its m-th largest
//      entry is >= a_m and the lists hold t_m.  With the forward's anchors (each its block's
//      maximum, so each of the m blocks holds an entry equal to its anchor) this is always the
//      case: a row costs its anchors and about m blocks of 64 columns.
//   3. Otherwise (anchors above their blocks' entries) the row's lists start again and every
//      block is read.
// The entries counted in pass 2 are distinct, and an entry >= a_m that does not enter a full
// list ranks below m counted ones, so the count reaches m exactly when the row has m entries
// >= a_m.  Entries reach a list out of index order, so an entry enters when it ranks above the
// list's last by (value desc, index asc).
template <typename T, int M>
__global__ void __launch_bounds__(256) k_topm_anchored(const T* __restrict__ L, const float* __restrict__ anc,
                                                       int64_t n, int V, int m, int32_t* __restrict__ idx,
                                                       float* __restrict__ val) {
  constexpr int TU = 4;  // a lane's anchor tiles in flight
  static_assert(kAnchorSlots == 4 && 4 * TU <= 32, "one 16-byte anchor vector per tile, one mask bit per block");
  __shared__ float s_v[4 * M * kTopmRows];
  __shared__ int32_t s_i[4 * M * kTopmRows];
  __shared__ int32_t s_c[4 * kTopmRows];
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * kTopmRows + l;
  const bool live = row0 < n;
  const int64_t row = live ? row0 : n - 1;  // a spare lane shadows the last row, writes nothing
  const int nb = (int)cdiv(V, kAnchorCols);
  const int nt = (int)cdiv(V, kAnchorTile);
  const floatx4* arow = reinterpret_cast<const floatx4*>(anc) + row;  // tile t at arow[t n]
  const T* r = L + row * (int64_t)V;
  // pass 1
  float av[M];
  int ab[M];
#pragma unroll
  for (int k = 0; k < M; ++k) {
    av[k] = -INFINITY;
    ab[k] = -1;
  }
  int seen = 0;  // blocks in this lane's share
  for (int t0 = w; t0 < nt; t0 += 4 * TU) {
    floatx4 q[TU];
#pragma unroll
    for (int u = 0; u < TU; ++u)
      if (t0 + 4 * u < nt) q[u] = arow[(int64_t)(t0 + 4 * u) * n];
#pragma unroll
    for (int u = 0; u < TU; ++u)
#pragma unroll
      for (int sl = 0; sl < 4; ++sl) {
        const int b = (t0 + 4 * u) * 4 + sl;
        if (t0 + 4 * u < nt && b < nb) {
          ++seen;
          float cv = q[u][sl];
          int cb = b;
          if (cv > av[M - 1]) {
#pragma unroll
            for (int k = 0; k < M; ++k) {
              const bool gt = cv > av[k];
              const float tv = av[k];
              const int tb = ab[k];
              av[k] = gt ? cv : tv;
              ab[k] = gt ? cb : tb;
              cv = gt ? tv : cv;
              cb = gt ? tb : cb;
            }
          }
        }
      }
  }
#pragma unroll
  for (int k = 0; k < M; ++k) s_v[(w * M + k) * kTopmRows + l] = av[k];
  __syncthreads();
  const float a_m = merge4<M>(s_v, nullptr, m, l);  // -inf when the row has fewer than m blocks
  __syncthreads();
  s_c[w * kTopmRows + l] = (seen > M && av[M - 1] >= a_m) ? 1 : 0;  // this lane may miss a block at a_m
  __syncthreads();
  const bool rescan = s_c[l] | s_c[kTopmRows + l] | s_c[2 * kTopmRows + l] | s_c[3 * kTopmRows + l];
  __syncthreads();
  float lv[M];
  int li[M];
#pragma unroll
  for (int k = 0; k < M; ++k) {
    lv[k] = -INFINITY;
    li[k] = 0x7fffffff;
  }
  int cnt = 0;  // entries >= a_m that entered this lane's list (each entry enters at most once)
  // pass 2: the listed blocks with anchor >= a_m (a prefix of the sorted list), two at a time
  // from the head of the list, which then shifts by two (every register index stays static);
  // an unfilled slot (block -1, anchor -inf) is never read, also when a_m is -inf
  for (int k = 0; k < M; k += 2) {
    const bool t0k = !rescan && ab[0] >= 0 && av[0] >= a_m;
    const bool t1k = M > 1 && !rescan && ab[M > 1 ? 1 : 0] >= 0 && av[M > 1 ? 1 : 0] >= a_m;
    if (!__any(t0k)) break;  // wave-uniform: the lists are sorted, nothing further qualifies
    topm_block<T, M>(r, V, ab[0], av[0], a_m, t0k, lv, li, cnt);
    if (M > 1) topm_block<T, M>(r, V, ab[M > 1 ? 1 : 0], av[M > 1 ? 1 : 0], a_m, t1k, lv, li, cnt);
#pragma unroll
    for (int q = 0; q < M; ++q) {
      av[q] = q + 2 < M ? av[q + 2 < M ? q + 2 : q] : -INFINITY;
      ab[q] = q + 2 < M ? ab[q + 2 < M ? q + 2 : q] : -1;
    }
  }
  if (__any(rescan)) topm_scan<T, M, TU>(r, arow, n, V, nb, nt, w, a_m, rescan, lv, li, cnt);
  // pass 3 for the rows with fewer than m entries >= a_m
  s_c[w * kTopmRows + l] = cnt;
  __syncthreads();
  const int total = s_c[l] + s_c[kTopmRows + l] + s_c[2 * kTopmRows + l] + s_c[3 * kTopmRows + l];
  if (__any(total < m)) {
    const bool redo = total < m;
    if (redo) {
#pragma unroll
      for (int k = 0; k < M; ++k) {
        lv[k] = -INFINITY;
        li[k] = 0x7fffffff;
      }
    }
    topm_scan<T, M, TU>(r, arow, n, V, nb, nt, w, -INFINITY, redo, lv, li, cnt);
  }
  // the four shares of each row, merged by wave 0
#pragma unroll
  for (int k = 0; k < M; ++k) {
    s_v[(w * M + k) * kTopmRows + l] = lv[k];
    s_i[(w * M + k) * kTopmRows + l] = li[k];
  }
  __syncthreads();
  if (w == 0 && live) merge4<M>(s_v, s_i, m, l, idx + row * (int64_t)m, val ? val + row * (int64_t)m : nullptr);
}

// hits[0 .. m) for p, hits[m .. 2m) for q; must start at zero.
__global__ void __launch_bounds__(256) k_topm_hits(const int32_t* __restrict__ idx, int64_t n, int m,
                                                   const int32_t* __restrict__ row_ptr,
                                                   const int32_t* __restrict__ tag,
                                                   const int32_t* __restrict__ q_sample,
                                                   const int32_t* __restrict__ q_tag, int64_t S,
                                                   unsigned long long* __restrict__ hits) {
  __shared__ unsigned int cnt[2 * 16];
  if (threadIdx.x < 2 * 16) cnt[threadIdx.x] = 0u;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t < n) {
    const int32_t* top = idx + t * (int64_t)m;
    for (int32_t q = row_ptr[t]; q < row_ptr[t + 1]; ++q) {
      const int32_t tg = tag[q];
      for (int k = 0; k < m; ++k)
        if (top[k] == tg) {
          atomicAdd(&cnt[k], 1u);  // counted for every m' > k below
          break;
        }
    }
  } else if (t - n < S) {
    const int64_t s = t - n;
    const int32_t i = q_sample[s];
    if (i >= 0 && i < n) {  // a draw naming no sample counts as a miss
      const int32_t* top = idx + (int64_t)i * m;
      const int32_t tg = q_tag[s];
      for (int k = 0; k < m; ++k)
        if (top[k] == tg) {
          atomicAdd(&cnt[16 + k], 1u);
          break;
        }
    }
  }
  __syncthreads();
  if (threadIdx.x < m) {
    // the entry at rank k is in t_m' for every m' > k: prefix over the ranks
    unsigned long long p = 0, qh = 0;
    for (int k = 0; k <= (int)threadIdx.x; ++k) {
      p += cnt[k];
      qh += cnt[16 + k];
    }
    if (p) atomicAdd(&hits[threadIdx.x], p);
    if (qh) atomicAdd(&hits[m + threadIdx.x], qh);
  }
}

template <typename T, int M>
static int topm_launch(const T* L, int64_t n, int V, int m, int32_t* idx, float* val, hipStream_t st) {
  HMOE_LAUNCH("top-m", (k_topm<T, M>), dim3((unsigned)cdiv(n, 4)), dim3(256), 0, st, L, n, V, m, idx, val);
  return HMOE_OK;
}

// The anchored kernel keeps M >= m entries per list (it takes the m-th of the merged lists), so
// four list lengths cover m = 1 .. 16.
template <typename T, int M>
static int topm_launch_anchored(const T* L, const float* anc, int64_t n, int V, int m, int32_t* idx, float* val,
                                hipStream_t st) {
  HMOE_LAUNCH("top-m", (k_topm_anchored<T, M>), dim3((unsigned)cdiv(n, kTopmRows)), dim3(256), 0, st, L, anc, n, V,
              m, idx, val);
  return HMOE_OK;
}

// The plain kernel's register lists hold exactly m entries (the insertion and the registers
// scale with the list length: a 16-entry list for m = 10 ran 25% slower than a 12-entry one).
template <typename T>
static int topm_t(const T* L, const float* anc, int64_t n, int V, int m, int32_t* idx, float* val, hipStream_t st) {
  if (anc) {
    if (m <= 4) return topm_launch_anchored<T, 4>(L, anc, n, V, m, idx, val, st);
    if (m <= 8) return topm_launch_anchored<T, 8>(L, anc, n, V, m, idx, val, st);
    if (m <= 12) return topm_launch_anchored<T, 12>(L, anc, n, V, m, idx, val, st);
    return topm_launch_anchored<T, 16>(L, anc, n, V, m, idx, val, st);
  }
  switch (m) {
    case 1: return topm_launch<T, 1>(L, n, V, m, idx, val, st);
    case 2: return topm_launch<T, 2>(L, n, V, m, idx, val, st);
    case 3: return topm_launch<T, 3>(L, n, V, m, idx, val, st);
    case 4: return topm_launch<T, 4>(L, n, V, m, idx, val, st);
    case 5: return topm_launch<T, 5>(L, n, V, m, idx, val, st);
    case 6: return topm_launch<T, 6>(L, n, V, m, idx, val, st);
    case 7: return topm_launch<T, 7>(L, n, V, m, idx, val, st);
    case 8: return topm_launch<T, 8>(L, n, V, m, idx, val, st);
    case 9: return topm_launch<T, 9>(L, n, V, m, idx, val, st);
    case 10: return topm_launch<T, 10>(L, n, V, m, idx, val, st);
    case 11: return topm_launch<T, 11>(L, n, V, m, idx, val, st);
    case 12: return topm_launch<T, 12>(L, n, V, m, idx, val, st);
    case 13: return topm_launch<T, 13>(L, n, V, m, idx, val, st);
    case 14: return topm_launch<T, 14>(L, n, V, m, idx, val, st);
    case 15: return topm_launch<T, 15>(L, n, V, m, idx, val, st);
    default: return topm_launch<T, 16>(L, n, V, m, idx, val, st);
  }
}

int launch_topm(const void* L, const float* anc, hmoe_dtype_t dt, int64_t n, int V, int m, int32_t* idx, float* val,
                hipStream_t st) {
  if (dt == HMOE_BF16) return topm_t<bf16>((const bf16*)L, anc, n, V, m, idx, val, st);
  return topm_t<float>((const float*)L, anc, n, V, m, idx, val, st);
}

int launch_topm_hits(const int32_t* idx, int64_t n, int m, const hmoe_labels_t* y, const int32_t* q_sample,
                     const int32_t* q_tag, int64_t S, int64_t* hits, hipStream_t st) {
  HMOE_TRY(launch_zero_f32((float*)hits, 4 * (int64_t)m, st));  // 2m int64 = 4m zero words
  if (n + S == 0) return HMOE_OK;
  HMOE_LAUNCH("top-m hits", k_topm_hits, dim3((unsigned)cdiv(n + S, 256)), dim3(256), 0, st, idx, n, m, y->row_ptr,
              y->tag, q_sample, q_tag, S, (unsigned long long*)hits);
  return HMOE_OK;
}

}  // namespace hmoe
