// metrics.hip -- the inference tail of Section 4.4: t_m, the m largest logits of every row
// (the softmax keeps their order, so these are the m most probable tags), and the counts
// behind p@m (Eq. 4) and q@m (Eq. 5) for every m' <= m.
//
// k_topm: one wave per row.  An entry is the stored value, plus its anchor when the logits are
// stored relative to per-row anchors (the forward's layout), the sum formed in fp32.
// Lane l reads the row's 16-byte vectors l, l + 64, ... (so it sees its entries in increasing
// index order) and keeps its own M largest in a register list sorted
// by decreasing value; an entry enters only when strictly greater than the list's last, which
// with the index order keeps equal values in increasing index order, and only when it is not
// below a wave-wide bound on the row's m-th value (the m-th largest of the lanes' maxima).
// The m results are then
// taken in m rounds of a wave-wide (value desc, index asc) maximum over the lists' heads; the
// lane holding the winner drops it.  The row is read once: the kernel is bound by HBM.
//
// k_topm_hits: one thread per row (p) and per draw (q); the rank of each matching tag in the
// top-m list adds 1 to every m' above it.  Integer counts, summed through LDS and then with
// one 64-bit atomic per block and m' -- integer sums, so the result does not depend on order.
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

template <typename T, int M>
__global__ void __launch_bounds__(256) k_topm(const T* __restrict__ L, const float* __restrict__ anc, int64_t n,
                                              int V, int m, int32_t* __restrict__ idx, float* __restrict__ val) {
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
    float an[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = b0 + 64 * u + l;
      an[u] = 0.f;
      if (v < nvec) {
        raw[u] = *reinterpret_cast<const i32x4*>(r + (int64_t)v * EPV);
        // the vector's anchor (a 16-byte vector never straddles a 64-column block)
        if (anc) an[u] = anc[anchor_index(n, row, (int64_t)v * EPV)];
      }
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
        f[z] = anc ? an[u] + to_f32(e[z]) : to_f32(e[z]);
        vmax = fmaxf(vmax, f[z]);
      }
      if (!(vmax >= thr && vmax > lv[M - 1])) continue;  // the common case: nothing here enters
#pragma unroll
      for (int z = 0; z < EPV; ++z) {
        float cv = f[z];
        if (cv >= thr && cv > lv[M - 1]) {
          int ci = v * EPV + z;
          // carry the entry down the list, ordered by (value desc, index asc): the new entry has
          // the largest index the lane has seen, so it goes before the first strictly smaller
          // one; an entry it displaces is carried on by the same order, ahead of equal values
          // with higher indices
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
      }
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
static int topm_launch(const T* L, const float* anc, int64_t n, int V, int m, int32_t* idx, float* val,
                       hipStream_t st) {
  HMOE_LAUNCH("top-m", (k_topm<T, M>), dim3((unsigned)cdiv(n, 4)), dim3(256), 0, st, L, anc, n, V, m, idx, val);
  return HMOE_OK;
}

// The register lists hold exactly m entries (the insertion and the registers scale with the
// list length: a 16-entry list for m = 10 ran 25% slower than a 12-entry one).
template <typename T>
static int topm_t(const T* L, const float* anc, int64_t n, int V, int m, int32_t* idx, float* val, hipStream_t st) {
  switch (m) {
    case 1: return topm_launch<T, 1>(L, anc, n, V, m, idx, val, st);
    case 2: return topm_launch<T, 2>(L, anc, n, V, m, idx, val, st);
    case 3: return topm_launch<T, 3>(L, anc, n, V, m, idx, val, st);
    case 4: return topm_launch<T, 4>(L, anc, n, V, m, idx, val, st);
    case 5: return topm_launch<T, 5>(L, anc, n, V, m, idx, val, st);
    case 6: return topm_launch<T, 6>(L, anc, n, V, m, idx, val, st);
    case 7: return topm_launch<T, 7>(L, anc, n, V, m, idx, val, st);
    case 8: return topm_launch<T, 8>(L, anc, n, V, m, idx, val, st);
    case 9: return topm_launch<T, 9>(L, anc, n, V, m, idx, val, st);
    case 10: return topm_launch<T, 10>(L, anc, n, V, m, idx, val, st);
    case 11: return topm_launch<T, 11>(L, anc, n, V, m, idx, val, st);
    case 12: return topm_launch<T, 12>(L, anc, n, V, m, idx, val, st);
    case 13: return topm_launch<T, 13>(L, anc, n, V, m, idx, val, st);
    case 14: return topm_launch<T, 14>(L, anc, n, V, m, idx, val, st);
    case 15: return topm_launch<T, 15>(L, anc, n, V, m, idx, val, st);
    default: return topm_launch<T, 16>(L, anc, n, V, m, idx, val, st);
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
