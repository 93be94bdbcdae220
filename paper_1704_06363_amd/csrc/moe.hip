// moe.hip -- hard-routed expert evaluation with a shared decoder (Section 2, shared-decoder
// figure) and the multilabel softmax loss (Section 4.1, Eq. 3), forward and backward.
//
// Rows arrive grouped by expert (X_sorted, offsets).  Every contraction runs on the MFMA tile
// engines of gemm.hpp (bf16: the direct-to-LDS engine; fp32: the register-staged one):
//   experts, forward     row-grouped NT GEMMs (bias + ReLU epilogue; the second layer's
//                        epilogue writes rows straight back to sample order = the combine)
//   decoder, forward     NT GEMM H . D^T with a per-row (max, sum exp) epilogue and, when the
//                        caller keeps them for the backward, the logits stored in the data
//                        dtype; a merge pass forms lse and the loss
//   decoder, backward    g = (p - y)/n, formed elementwise from the stored logits (or, without
//                        them, from logits recomputed by the GEMM), stored with per-tile column
//                        sums for dbD; then dH = g D (epilogue scatters rows to expert order) and
//                        dD = g^T H (a partly filled last round of tiles split over K)
//   experts, backward    reduction-grouped TN GEMMs for dW (empty experts give exact zeros),
//                        row-grouped NN GEMMs for dH1 (ReLU mask epilogue) and dX (epilogue
//                        scatters rows back to sample order); bias gradients are deterministic
//                        segmented column sums.
#include <float.h>

#include "gemm.hpp"
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

// ------------------------------------------------------------------ expert forward

struct RowVia {  // destination row = map[m0 + r]
  const int32_t* __restrict__ map;
  int64_t m0;
  __device__ __forceinline__ int64_t operator()(int r) const { return map[m0 + r]; }
};
struct Ident {
  __device__ __forceinline__ float operator()(int, int, int, float v) const { return v; }
};

// LAYER 1: H1s[m] = relu(Xs[m] W1_e^T + b1_e).   LAYER 2: H[perm[m]] = H1s[m] W2_e^T + b2_e.
template <class C, int LAYER>
__device__ __forceinline__ void expert_fwd_tile(const TileCoord& tc, const typename C::type* __restrict__ A,
                                                const typename C::type* __restrict__ W,
                                                const typename C::type* __restrict__ bias, int N, int Kd,
                                                const int32_t* __restrict__ perm, typename C::type* __restrict__ out,
                                                lds<char>* smem) {
  using T = typename C::type;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, true>(A + tc.m0 * Kd, Kd, tc.m_rows, W + ((int64_t)tc.group * N + tc.n0) * Kd, Kd,
                           tc.n_cols, Kd, smem, acc);
  using F = Frag<C>;
  const F f;
  const T* be = bias ? bias + (int64_t)tc.group * N : nullptr;
  float bv[F::NCOL];
#pragma unroll
  for (int q = 0; q < F::NCOL; ++q) {
    const int col = f.colq(q);
    bv[q] = (be && col < tc.n_cols) ? to_f32(be[tc.n0 + col]) : 0.f;
  }
  auto elem = [&](int, int j, int r, float v) {
    v += bv[F::qidx(j, r)];
    return LAYER == 1 ? fmaxf(v, 0.f) : v;
  };
  if (LAYER == 1)
    store_out<C, T>(tc, acc, smem, out, N, elem, RowId{tc.m0}, NoVec{});
  else
    store_out<C, T>(tc, acc, smem, out, N, elem, RowVia{perm, tc.m0}, NoVec{});
}

// A group's last row tile with few enough rows runs the half-height configuration when C has
// one (the workgroup size and the LDS allocation are C's).
template <class C, class Body>
__device__ __forceinline__ void by_tile_height(const TileCoord& tc, Body body) {
  using S = typename ShortTile<C>::type;
  if constexpr (!std::is_void<S>::value) {
    static_assert(S::THREADS == C::THREADS && S::LDS <= C::LDS, "short tile inside the workgroup");
    if (tc.m_rows <= S::BM) {
      body(S{});
      return;
    }
  }
  body(C{});
}

template <class C, int LAYER>
__global__ void __launch_bounds__(C::THREADS)
    k_expert_fwd(const typename C::type* __restrict__ A, const typename C::type* __restrict__ W,
                 const typename C::type* __restrict__ bias, const int32_t* __restrict__ seg,
                 const int32_t* __restrict__ tile_start, int G, int N, int Kd, const int32_t* __restrict__ perm,
                 typename C::type* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_group_m<C>(seg, tile_start, G, N, Kd);
  if (!tc.valid) return;
  by_tile_height<C>(tc, [&](auto cfg) {
    expert_fwd_tile<decltype(cfg), LAYER>(tc, A, W, bias, N, Kd, perm, out, smem);
  });
}

// ------------------------------------------------------------------ decoder forward

// acc += bias, in place: the accumulators become the tile's logits (the statistics and the
// stored logits both read them).
template <class C>
__device__ __forceinline__ void add_bias(floatx4 (&acc)[C::MI][C::NJ], const float (&bias)[Frag<C>::NCOL]) {
  using F = Frag<C>;
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] += bias[F::qidx(j, r)];
}

// Per-wave row statistics of a logits tile: m = max over the wave's valid columns of the row,
// s = sum exp(logit - m) (as exp2 of logit log2(e) - m log2(e)), into rm / rs [WAVES_N][BM].
// m is also the row's anchor for this wave's 64 columns, the value a stored logit is relative
// to; with mxo given it is kept there too, mxo[4 i + r] for accumulator row (i, r) (TRANS: one
// row per i, at mxo[4 i]).  The accumulators are only read: subtracting in place measured
// 12 -> 424 bytes of spill per lane in the persistent forward.
// FULL: every column of the tile is valid (no column guards).
template <class C, bool FULL>
__device__ __forceinline__ void dec_row_stats(const TileCoord& tc, const floatx4 (&acc)[C::MI][C::NJ],
                                              lds<float>* rm, lds<float>* rs, float* mxo = nullptr) {
  static_assert(C::WN == kAnchorCols, "one anchor per wave and row");
  using F = Frag<C>;
  const F f;
  constexpr float kLog2e = 1.4426950408889634f;
  if constexpr (F::T) {
    // one row per i; its WN columns of this wave sit in lanes lr, lr + 16, lr + 32, lr + 48
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      float mx = -FLT_MAX;
#pragma unroll
      for (int j = 0; j < C::NJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (FULL || f.col(j, r) < tc.n_cols) mx = fmaxf(mx, acc[i][j][r]);
      mx = fmaxf(mx, shfl_xor(mx, 16));
      mx = fmaxf(mx, shfl_xor(mx, 32));
      if (mxo) mxo[4 * i] = mx;
      const float mb = mx * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < C::NJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (FULL || f.col(j, r) < tc.n_cols) s += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, -mb));
      s += shfl_xor(s, 16);
      s += shfl_xor(s, 32);
      if (f.lg == 0) {
        rm[f.wn * C::BM + f.row(i, 0)] = mx;
        rs[f.wn * C::BM + f.row(i, 0)] = s;
      }
    }
  } else {
    // four rows per i; a row's WN columns of this wave sit in the 16 lanes of one lane group
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float mx = -FLT_MAX;
#pragma unroll
        for (int j = 0; j < C::NJ; ++j)
          if (FULL || f.col(j, r) < tc.n_cols) mx = fmaxf(mx, acc[i][j][r]);
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) mx = fmaxf(mx, shfl_xor(mx, m));
        if (mxo) mxo[4 * i + r] = mx;
        const float mb = mx * kLog2e;
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < C::NJ; ++j)
          if (FULL || f.col(j, r) < tc.n_cols) s += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, -mb));
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) s += shfl_xor(s, m);
        if (f.lr == 0) {
          rm[f.wn * C::BM + f.row(i, r)] = mx;
          rs[f.wn * C::BM + f.row(i, r)] = s;
        }
      }
  }
}

// Softmax statistics of one logits tile (acc already holds accumulator + bias): per row,
// m = max over the tile's valid columns and s = sum exp(logit - m), merged over the WAVES_N
// waves that share the row through rm / rs (LDS, [WAVES_N][BM] floats each) and written as the
// tile's partials pm[n-tile][row], ps[n-tile][row].  Entered by the whole workgroup.
// The second half of dec_tile_stats: after the waves' row partials are in LDS, merge them per
// row and write the tile's (max, sum) pair, and (anc != NULL) the waves' row maxima as the
// anchors of the stored logits: anc[v / 256][row][(v % 256) / 64] for column v.  A wave with no
// valid column writes -FLT_MAX into a slot no stored logit refers to.
template <class C, bool BARRIER = true>
__device__ __forceinline__ void dec_stats_merge(const TileCoord& tc, lds<float>* rm, lds<float>* rs, int64_t n,
                                                float* __restrict__ pm, float* __restrict__ ps,
                                                float* __restrict__ anc) {
  static_assert(C::WN == kAnchorCols && (kAnchorTile / C::BN) * C::BN == kAnchorTile, "anchor slots per tile");
  typedef float avec __attribute__((ext_vector_type(C::WAVES_N)));
  if constexpr (BARRIER) wg_barrier_lds();
  for (int t = threadIdx.x; t < tc.m_rows; t += C::THREADS) {
    avec mw;
#pragma unroll
    for (int w = 0; w < C::WAVES_N; ++w) mw[w] = rm[w * C::BM + t];
    float M = mw[0];
#pragma unroll
    for (int w = 1; w < C::WAVES_N; ++w) M = fmaxf(M, mw[w]);
    float S = 0.f;
#pragma unroll
    for (int w = 0; w < C::WAVES_N; ++w) S += rs[w * C::BM + t] * __expf(mw[w] - M);
    const int64_t at = (int64_t)(tc.n0 / C::BN) * n + tc.m0 + t;
    pm[at] = M;
    ps[at] = S;
    if (anc)
      *reinterpret_cast<avec*>(anc + ((int64_t)(tc.n0 / kAnchorTile) * n + tc.m0 + t) * kAnchorSlots +
                               (tc.n0 % kAnchorTile) / kAnchorCols) = mw;
  }
}

template <class C>
__device__ __forceinline__ void dec_tile_stats(const TileCoord& tc, const floatx4 (&acc)[C::MI][C::NJ],
                                               lds<float>* rm, lds<float>* rs, int64_t n, float* __restrict__ pm,
                                               float* __restrict__ ps, float* __restrict__ anc, float* mxo) {
  if (tc.n_cols == C::BN)
    dec_row_stats<C, true>(tc, acc, rm, rs, mxo);
  else
    dec_row_stats<C, false>(tc, acc, rm, rs, mxo);
  dec_stats_merge<C>(tc, rm, rs, n, pm, ps, anc);
}

// The stored logit of accumulator element (i, j, r): its offset from the wave's row maximum
// (mx as kept by dec_row_stats; held by value, so that it stays in registers).
template <class C>
struct Anchored {
  float mx[4 * C::MI];
  __device__ __forceinline__ float operator()(int i, int, int r, float v) const {
    return v - mx[C::TRANS ? 4 * i : 4 * i + r];
  }
};

template <class C>
__device__ __forceinline__ void dec_tile_bias(const TileCoord& tc, const typename C::type* __restrict__ bD,
                                              float (&bias)[Frag<C>::NCOL]) {
  using F = Frag<C>;
  const F f;
#pragma unroll
  for (int q = 0; q < F::NCOL; ++q) {
    const int col = f.colq(q);
    bias[q] = (bD && col < tc.n_cols) ? to_f32(bD[tc.n0 + col]) : 0.f;
  }
}

// Per row and V-tile: the softmax partials (dec_tile_stats); the logits themselves are stored
// to L when L is given (saved for the backward), as offsets from their anchors (anc).  One tile
// per workgroup (register-staged engine).
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_dec_fwd(const typename C::type* __restrict__ H, const typename C::type* __restrict__ D,
              const typename C::type* __restrict__ bD, int64_t n, int V, int o, float* __restrict__ pm,
              float* __restrict__ ps, typename C::type* __restrict__ L, float* __restrict__ anc) {
  using T = typename C::type;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_plain<C>(n, V, o);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, true>(H + tc.m0 * o, o, tc.m_rows, D + (int64_t)tc.n0 * o, o, tc.n_cols, o, smem, acc);
  using F = Frag<C>;
  float bias[F::NCOL];
  dec_tile_bias<C>(tc, bD, bias);
  add_bias<C>(acc, bias);
  lds<float>* rm = reinterpret_cast<lds<float>*>(smem);  // reuses the operand buffers
  Anchored<C> an;
  dec_tile_stats<C>(tc, acc, rm, rm + C::WAVES_N * C::BM, n, pm, ps, L ? anc : nullptr, an.mx);
  if (L) {
    if constexpr (!F::T) __syncthreads();  // the LDS-staged store reuses rm / rs
    store_out<C, T>(tc, acc, smem, L, V, an, RowId{tc.m0}, NoVec{});
  }
}

// One decoder per expert (row-grouped): the slot rows of expert e against D_e [V][o] and
// bD_e; the softmax partials (dec_tile_stats, rows in slot order) and, when L is given, the
// logits (offsets from their anchors) and the anchors in slot order.  One tile per workgroup.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_dec_fwd_grouped(const typename C::type* __restrict__ Hs, const typename C::type* __restrict__ D,
                      const typename C::type* __restrict__ bD, const int32_t* __restrict__ seg,
                      const int32_t* __restrict__ tile_start, int G, int64_t n, int V, int o, float* __restrict__ pm,
                      float* __restrict__ ps, typename C::type* __restrict__ L, float* __restrict__ anc) {
  using T = typename C::type;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_group_m<C>(seg, tile_start, G, V, o);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, true>(Hs + tc.m0 * o, o, tc.m_rows, D + ((int64_t)tc.group * V + tc.n0) * o, o, tc.n_cols, o,
                           smem, acc);
  using F = Frag<C>;
  float bias[F::NCOL];
  dec_tile_bias<C>(tc, bD ? bD + (int64_t)tc.group * V : nullptr, bias);
  add_bias<C>(acc, bias);
  lds<float>* rm = reinterpret_cast<lds<float>*>(smem);  // reuses the operand buffers
  Anchored<C> an;
  dec_tile_stats<C>(tc, acc, rm, rm + C::WAVES_N * C::BM, n, pm, ps, L ? anc : nullptr, an.mx);
  if (L) {
    if constexpr (!F::T) __syncthreads();  // the LDS-staged store reuses rm / rs
    store_out<C, T>(tc, acc, smem, L, V, an, RowId{tc.m0}, NoVec{});
  }
}

// The same computation as a persistent kernel on the direct-to-LDS engine: gridDim.x workgroups
// walk the tiles blockIdx.x, blockIdx.x + gridDim.x, ...  After a tile's K loop the workgroup
// forms the tile's softmax statistics, issues the first stages of its next tile and only then
// stores the logits, so the store drain overlaps the next tile's first stages: for a full tile
// every wave issues exactly direct_stores() stores there, and the waits for the primed stages
// let those stay in flight (ragged tiles wait for everything).  The logits are stored with
// ordinary stores: a wave's store covers 64 bytes of a row, and the L2 merges the two halves of
// each 128-byte line before writing it back (non-temporal stores measured 1.5x the write
// traffic).  The row partials (rm / rs) sit past the operand ring in two buffers, alternating
// by tile (dynamic LDS = C::LDS + 2 kDecStatLds): a tile's partials are merged across waves in
// the next tile's epilogue, after that tile's K loop, whose barriers order the partials'
// writes before the merge's reads and the merge's reads before the buffer is written again.
constexpr int kDecStatLds = 2 * 4 * 256 * (int)sizeof(float);
template <class C>
__device__ __forceinline__ void dec_bias_packed(const TileCoord& tc, const bf16* __restrict__ bD,
                                                uint2 (&bp)[C::NJ]) {
  const Frag<C> f;
#pragma unroll
  for (int j = 0; j < C::NJ; ++j) {
    const int col = f.col(j, 0);  // four consecutive columns; n_cols is a multiple of 8
    bp[j] = (bD && col < tc.n_cols) ? *reinterpret_cast<const uint2*>(bD + tc.n0 + col) : uint2{0u, 0u};
  }
}
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_dec_fwd_stream(const bf16* __restrict__ H, const bf16* __restrict__ D, const bf16* __restrict__ bD, int64_t n,
                     int V, int o, float* __restrict__ pm, float* __restrict__ ps, bf16* __restrict__ L,
                     float* __restrict__ anc) {
  static_assert(C::DMA && C::TRANS, "persistent decoder forward runs the direct-to-LDS engine");
  static_assert(2 * C::WAVES_N * C::BM * (int)sizeof(float) <= kDecStatLds, "statistics scratch");
  constexpr int STORES = direct_stores<C, bf16>();  // per wave, for a full tile
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  lds<float>* rm0 = reinterpret_cast<lds<float>*>(smem + C::LDS);
  constexpr int SB = 2 * C::WAVES_N * C::BM;  // one statistics buffer (floats)
  using F = Frag<C>;
  const F f0;
  const int64_t tiles = cdiv(n, C::BM) * cdiv(V, C::BN);
  int64_t t = blockIdx.x;
  if (t >= tiles) return;
  TileCoord tc = tile_plain_at<C>(n, V, o, t);
  DmaTile<C, true, true> pipe;
  pipe.prime(H + tc.m0 * o, o, tc.m_rows, D + (int64_t)tc.n0 * o, o, tc.n_cols, o, smem);
  uint2 bp[C::NJ];
  dec_bias_packed<C>(tc, bD, bp);
  bool stores_pending = false;
  int buf = 0;
  TileCoord pc = tc;  // the previous tile, whose partials merge in this tile's epilogue
  bool have_prev = false;
  for (;;) {
    floatx4 acc[C::MI][C::NJ];
    pipe.template run<false, STORES>(smem, acc, nullptr, stores_pending);
    lds<float>* rm = rm0 + buf * SB;
    lds<float>* rs = rm + C::WAVES_N * C::BM;
    float bias[F::NCOL];
#pragma unroll
    for (int j = 0; j < C::NJ; ++j) {
      bias[4 * j + 0] = __uint_as_float(bp[j].x << 16);
      bias[4 * j + 1] = __uint_as_float(bp[j].x & 0xffff0000u);
      bias[4 * j + 2] = __uint_as_float(bp[j].y << 16);
      bias[4 * j + 3] = __uint_as_float(bp[j].y & 0xffff0000u);
    }
    // the next tile's first stages go out before the statistics, so their loads land while
    // the epilogue runs (run() ends with every wave past its last read of the ring; the
    // statistics' partials stores are then younger than the primed loads, which can only make
    // the next tile's waits stricter)
    const int64_t tn = t + gridDim.x;
    const bool more = tn < tiles;
    TileCoord nc = tc;
    if (more) {
      nc = tile_plain_at<C>(n, V, o, tn);
      dec_bias_packed<C>(nc, bD, bp);
      pipe.prime(H + nc.m0 * o, o, nc.m_rows, D + (int64_t)nc.n0 * o, o, nc.n_cols, o, smem);
    }
    add_bias<C>(acc, bias);
    // the waves' row partials, then the logits stores, then the previous tile's merge:
    // measured faster than merging before the stores.  The merge's stores are younger than
    // the logits stores, which only makes the next tile's waits stricter.
    if (tc.n_cols == C::BN)
      dec_row_stats<C, true>(tc, acc, rm, rs);
    else
      dec_row_stats<C, false>(tc, acc, rm, rs);
    // nothing may move between the primed loads and the stores: the next waits count them
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    if (L) {
      // the anchor of each row: this wave's row maximum, read back from the partials it has
      // just written (a wave's LDS accesses complete in order; the registers are full here)
      const lds<float>* rmw = rm + f0.wn * C::BM;
      store_direct<C, bf16>(tc, acc, L, V, [&](int i, int, int, float v) { return v - rmw[f0.row(i, 0)]; },
                            RowId{tc.m0}, NoVec{});
    }
    __builtin_amdgcn_sched_barrier(0);
    // the previous tile's partials were written before this tile's K loop, whose barriers
    // order them; its buffer is rewritten only after the next K loop
    if (have_prev) {
      lds<float>* pm_l = rm0 + (buf ^ 1) * SB;
      dec_stats_merge<C, false>(pc, pm_l, pm_l + C::WAVES_N * C::BM, n, pm, ps, anc);
    }
    if (!more) {
      dec_stats_merge<C>(tc, rm, rs, n, pm, ps, anc);
      break;
    }
    stores_pending = L != nullptr && tc.m_rows == C::BM && tc.n_cols == C::BN;
    pc = tc;
    have_prev = true;
    buf ^= 1;
    t = tn;
    tc = nc;
  }
}

// lse = merge of the tile partials; loss = lse - mean positive logit.  A block takes 64 rows.
// The merge reads the partials [tile][row] coalesced: lane l of wave w takes row r0 + l and the
// tiles t = w, w + 4, ... with an online (max, sum) merge, and the four waves' pairs are merged
// in wave order.  The positive logits are (row, tag) tasks, numbered row by row in tag order:
// 8 lanes per task each take every 8th 16-byte vector of the H row and the D row (row widths
// are multiples of 8, so o / (16 / sizeof(T)) vectors cover a row exactly), the 8 partial sums
// are combined by lane shuffles, and each row adds its tasks' dots in task order.
// With per-expert decoders the rows (partials and H) are in slot order: row r is sample
// perm[r], decoded by D_e, bD_e of the expert e whose segment of `seg` holds r; lse and loss
// are written in sample order.  Shared decoder: perm = seg = NULL.
constexpr int kLossRows = 64;
constexpr int kLossTasks = 512;  // tasks staged in LDS at a time

template <typename T>
__global__ void __launch_bounds__(256) k_dec_loss(const float* __restrict__ pm, const float* __restrict__ ps,
                                                  int nt, const T* __restrict__ H, const T* __restrict__ D,
                                                  const T* __restrict__ bD, int64_t n, int o, int V,
                                                  const int32_t* __restrict__ perm, const int32_t* __restrict__ seg,
                                                  int G, const int32_t* __restrict__ row_ptr,
                                                  const int32_t* __restrict__ tag, float* __restrict__ lse,
                                                  float* __restrict__ loss) {
  constexpr int EPV = 16 / sizeof(T);
  __shared__ float s_m[4][kLossRows], s_s[4][kLossRows], s_pos[kLossRows];
  __shared__ int32_t s_first[kLossRows + 1];  // first task of each row (exclusive prefix)
  __shared__ int32_t s_p0[kLossRows], s_exp[kLossRows];
  __shared__ int32_t s_trow[kLossTasks], s_ttag[kLossTasks];
  __shared__ float s_dot[kLossTasks];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int64_t r0 = (int64_t)blockIdx.x * kLossRows;
  const int rows = (int)(n - r0 < kLossRows ? n - r0 : kLossRows);
  {
    float M = -FLT_MAX, S = 0.f;
    if (l < rows)
      for (int t = w; t < nt; t += 4) {
        const float m = pm[(int64_t)t * n + r0 + l], sv = ps[(int64_t)t * n + r0 + l];
        if (m > M) {
          S = S * __expf(M - m) + sv;
          M = m;
        } else {
          S += sv * __expf(m - M);
        }
      }
    s_m[w][l] = M;
    s_s[w][l] = S;
  }
  if (threadIdx.x < kLossRows) {
    const int t = threadIdx.x;
    int32_t cnt = 0;
    if (t < rows) {
      const int64_t row = r0 + t;
      const int64_t smp = perm ? perm[row] : row;
      const int32_t p0 = row_ptr[smp];
      cnt = row_ptr[smp + 1] - p0;
      s_p0[t] = p0;
      s_exp[t] = seg ? find_segment(seg, G, row) : 0;
    }
    s_first[t + 1] = cnt;  // turned into the prefix below
    s_pos[t] = 0.f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    s_first[0] = 0;
    for (int t = 0; t < kLossRows; ++t) s_first[t + 1] += s_first[t];
  }
  __syncthreads();
  const int total = s_first[kLossRows];
  const int g = l >> 3, gl = l & 7;
  const int vpr = o / EPV;
  for (int c0 = 0; c0 < total; c0 += kLossTasks) {
    const int cn = total - c0 < kLossTasks ? total - c0 : kLossTasks;
    if (threadIdx.x < rows) {  // stage this row's tasks of the chunk
      const int t = threadIdx.x;
      const int a = s_first[t] > c0 ? s_first[t] : c0;
      const int b = s_first[t + 1] < c0 + cn ? s_first[t + 1] : c0 + cn;
      for (int j = a; j < b; ++j) {
        s_trow[j - c0] = t;
        s_ttag[j - c0] = tag[s_p0[t] + (j - s_first[t])];
      }
    }
    __syncthreads();
    // 32 tasks per step over the block; the trip count is the same for every lane of a wave
    for (int j0 = w * 8; j0 < cn; j0 += 32) {
      const int j = j0 + g;
      float sdot = 0.f;
      // a tag outside [0, V) is never dereferenced: its logit counts as 0
      if (j < cn && (unsigned)s_ttag[j] < (unsigned)V) {
        const int t = s_trow[j];
        const int32_t tg = s_ttag[j];
        const T* h = H + (r0 + t) * o;
        const T* dv = D + ((int64_t)s_exp[t] * V + tg) * o;
        int v = gl;
        for (; v + 24 < vpr; v += 32) {  // four vector pairs in flight
          i32x4 hr[4], dr[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            hr[u] = *reinterpret_cast<const i32x4*>(h + (v + 8 * u) * EPV);
            dr[u] = *reinterpret_cast<const i32x4*>(dv + (v + 8 * u) * EPV);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const T* he = reinterpret_cast<const T*>(&hr[u]);
            const T* de = reinterpret_cast<const T*>(&dr[u]);
#pragma unroll
            for (int z = 0; z < EPV; ++z) sdot += to_f32(he[z]) * to_f32(de[z]);
          }
        }
        for (; v < vpr; v += 8) {
          const i32x4 hr = *reinterpret_cast<const i32x4*>(h + v * EPV);
          const i32x4 dr = *reinterpret_cast<const i32x4*>(dv + v * EPV);
          const T* he = reinterpret_cast<const T*>(&hr);
          const T* de = reinterpret_cast<const T*>(&dr);
#pragma unroll
          for (int z = 0; z < EPV; ++z) sdot += to_f32(he[z]) * to_f32(de[z]);
        }
      }
      sdot += shfl_xor(sdot, 4);
      sdot += shfl_xor(sdot, 2);
      sdot += shfl_xor(sdot, 1);
      if (j < cn && gl == 0) {
        const int t = s_trow[j];
        const bool ok = (unsigned)s_ttag[j] < (unsigned)V;
        s_dot[j] = sdot + ((bD && ok) ? to_f32(bD[(int64_t)s_exp[t] * V + s_ttag[j]]) : 0.f);
      }
    }
    __syncthreads();
    if (threadIdx.x < rows) {  // this row's tasks of the chunk, in task order
      const int t = threadIdx.x;
      const int a = s_first[t] > c0 ? s_first[t] : c0;
      const int b = s_first[t + 1] < c0 + cn ? s_first[t + 1] : c0 + cn;
      float acc = s_pos[t];
      for (int j = a; j < b; ++j) acc += s_dot[j - c0];
      s_pos[t] = acc;
    }
    __syncthreads();
  }
  if (threadIdx.x < rows) {
    const int t = threadIdx.x;
    float M = s_m[0][t], S = s_s[0][t];
#pragma unroll
    for (int q = 1; q < 4; ++q) {
      const float m = s_m[q][t], sv = s_s[q][t];
      if (m > M) {
        S = S * __expf(M - m) + sv;
        M = m;
      } else {
        S += sv * __expf(m - M);
      }
    }
    const float Lv = M + __logf(S);
    const int64_t smp = perm ? perm[r0 + t] : r0 + t;
    lse[smp] = Lv;
    loss[smp] = Lv - s_pos[t] / (float)(s_first[t + 1] - s_first[t]);
  }
}

// ------------------------------------------------------------------ decoder backward

// Recompute path: g = (exp(logit - lse) - y) / n with the logits recomputed by the GEMM;
// g stored to G, per-tile column sums of g to part_db[mtile][V].
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_dec_grad(const typename C::type* __restrict__ H, const typename C::type* __restrict__ D,
               const typename C::type* __restrict__ bD, int64_t n, int V, int o, const float* __restrict__ lse,
               const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ tag, float inv_n,
               typename C::type* __restrict__ G, float* __restrict__ part_db) {
  using T = typename C::type;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_plain<C>(n, V, o);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, true>(H + tc.m0 * o, o, tc.m_rows, D + (int64_t)tc.n0 * o, o, tc.n_cols, o, smem, acc);
  using F = Frag<C>;
  const F f;
  float bias[F::NCOL];
#pragma unroll
  for (int q = 0; q < F::NCOL; ++q) {
    const int col = f.colq(q);
    bias[q] = (bD && col < tc.n_cols) ? to_f32(bD[tc.n0 + col]) : 0.f;
  }
  // Per-row data of the tile, staged once in LDS (the operand buffers are free now).
  constexpr int MAXT = 16;
  lds<float>* s_lse = reinterpret_cast<lds<float>*>(smem);                // [BM]
  lds<int32_t>* s_p0 = reinterpret_cast<lds<int32_t>*>(s_lse + C::BM);    // [BM]
  lds<int32_t>* s_cnt = s_p0 + C::BM;                                     // [BM]
  lds<int32_t>* s_tag = s_cnt + C::BM;                                    // [BM][MAXT]
  lds<float>* cs = reinterpret_cast<lds<float>*>(s_tag + C::BM * MAXT);   // [WAVES_M][BN]
  for (int t = threadIdx.x; t < tc.m_rows; t += C::THREADS) {
    const int64_t gr = tc.m0 + t;
    const int32_t p0 = row_ptr[gr], cnt = row_ptr[gr + 1] - p0;
    s_lse[t] = lse[gr];
    s_p0[t] = p0;
    s_cnt[t] = cnt;
    for (int q = 0; q < cnt && q < MAXT; ++q) s_tag[t * MAXT + q] = tag[p0 + q];
  }
  __syncthreads();
  const int wcol0 = tc.n0 + f.wn * C::WN;  // first column of this wave
  // g for accumulator element (i, j, r) of row `row`; rows past the tile give 0
  auto grad_row = [&](int i, int row, auto owns, auto pick) {
    const float Lr = s_lse[row];
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (pick(r)) acc[i][j][r] = __expf(acc[i][j][r] + bias[F::qidx(j, r)] - Lr);
    const int32_t cnt = s_cnt[row];
    const float y = 1.f / (float)cnt;
    for (int32_t q = 0; q < cnt; ++q) {
      const int lc = (q < MAXT ? s_tag[row * MAXT + q] : tag[s_p0[row] + q]) - wcol0;
      if (lc >= 0 && lc < C::WN && owns(lc)) {
#pragma unroll
        for (int j = 0; j < C::NJ; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (pick(r) && f.col(j, r) - f.wn * C::WN == lc) acc[i][j][r] -= y;
      }
    }
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (pick(r)) acc[i][j][r] = (f.col(j, r) < tc.n_cols) ? acc[i][j][r] * inv_n : 0.f;
  };
  if constexpr (F::T) {
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int row = f.row(i, 0);
      if (row >= tc.m_rows) {
#pragma unroll
        for (int j = 0; j < C::NJ; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        continue;
      }
      grad_row(i, row, [&](int lc) { return ((lc & 15) >> 2) == f.lg; }, [](int) { return true; });
    }
    // column sums over this tile's rows: the 16 lanes of a column's lane group, then the row waves
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < C::MI; ++i) s += acc[i][j][r];
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) s += shfl_xor(s, m);
        if (f.lr == 0) cs[f.wm * C::BN + f.col(j, r)] = s;
      }
  } else {
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = f.row(i, r);
        if (row >= tc.m_rows) {
#pragma unroll
          for (int j = 0; j < C::NJ; ++j) acc[i][j][r] = 0.f;
          continue;
        }
        grad_row(i, row, [&](int lc) { return (lc & 15) == f.lr; }, [r](int rr) { return rr == r; });
      }
    // column sums over this tile's rows: the lane groups, then the row waves
#pragma unroll
    for (int j = 0; j < C::NJ; ++j) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) s += acc[i][j][r];
      s += shfl_xor(s, 16);
      s += shfl_xor(s, 32);
      if (f.lg == 0) cs[f.wm * C::BN + f.col(j, 0)] = s;
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < tc.n_cols; t += C::THREADS) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < C::WAVES_M; ++w) s += cs[w * C::BN + t];
    part_db[(tc.m0 / C::BM) * (int64_t)V + tc.n0 + t] = s;
  }
  if constexpr (!F::T) __syncthreads();  // the LDS-staged store reuses the row data
  store_out<C, T>(tc, acc, smem, G, V, Ident{}, RowId{tc.m0}, NoVec{});
}

// Saved-logits path: g = (exp(anchor + L - lse) - y) / n elementwise over [n x V] (L holds the
// logits as offsets from their anchors, anc, one per row and 64 columns); each thread owns one
// 16-byte column vector over kGradRows rows, whose anchors are one per row (a vector never
// straddles a 64-column block), and writes its column sums to part_db[rowblock][V].
// A block covers a slab of 256 x EPV columns; per row it keeps (in LDS) only the tags that fall
// inside its slab, so the per-element work is an fma and an exp, and a tag costs one compare
// per row in the few rows that have one here.  A row with more than MAXT tags in the slab
// (flag -1) reads its tags from global memory instead.  g is stored non-temporally: it is only
// read back by the next kernels, long after it has left the caches (measured 3.07 -> 2.91 ms).
// Per-expert decoders: the rows (L, g) are in slot order, row r being sample perm[r], and a
// block takes a piece of at most kGradRows rows of one expert (pieces numbered by
// piece_start, as in the segmented sums), so its column sums belong to one decoder's dbD.
// Shared decoder: perm = piece_start = NULL and block b takes rows [b, b + 1) * kGradRows.
constexpr int kGradRows = 256;

template <typename T>
__global__ void __launch_bounds__(256) k_dec_grad_elem(const T* __restrict__ L, const float* __restrict__ anc,
                                                       const float* __restrict__ lse,
                                                       const int32_t* __restrict__ row_ptr,
                                                       const int32_t* __restrict__ tag, int64_t n, int V,
                                                       float inv_n, const int32_t* __restrict__ perm,
                                                       const int32_t* __restrict__ seg,
                                                       const int32_t* __restrict__ piece_start, int NG,
                                                       T* __restrict__ G, float* __restrict__ part_db, int slab) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int MAXT = 16;
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ float s_lse2[kGradRows], s_yn[kGradRows];
  __shared__ int32_t s_cnt[kGradRows], s_smp[kGradRows];
  __shared__ int16_t s_tag[kGradRows * MAXT];  // column within the slab
  int64_t r0, rend;
  if (piece_start) {
    if ((int64_t)blockIdx.x >= piece_start[NG]) return;
    const int e = find_segment(piece_start, NG, blockIdx.x);
    r0 = seg[e] + (int64_t)(blockIdx.x - piece_start[e]) * kGradRows;
    rend = seg[e + 1];
  } else {
    r0 = (int64_t)blockIdx.x * kGradRows;
    rend = n;
  }
  const int rows = (int)((rend - r0) < kGradRows ? (rend - r0) : kGradRows);
  const int slab0 = blockIdx.y * 256 * EPV;
  for (int t = threadIdx.x; t < rows; t += 256) {
    const int64_t smp = perm ? perm[r0 + t] : r0 + t;
    const int32_t p0 = row_ptr[smp], cnt = row_ptr[smp + 1] - p0;
    s_smp[t] = (int32_t)smp;
    s_lse2[t] = lse[smp] * kLog2e;
    s_yn[t] = inv_n / (float)cnt;
    int k = 0;
    for (int q = 0; q < cnt; ++q) {
      const int d = tag[p0 + q] - slab0;
      if ((unsigned)d < (unsigned)(256 * EPV)) {
        if (k < MAXT) s_tag[t * MAXT + k] = (int16_t)d;
        ++k;
      }
    }
    s_cnt[t] = k <= MAXT ? k : -1;
  }
  __syncthreads();
  const int c0 = slab0 + threadIdx.x * EPV;
  if (c0 >= V) return;
  const int cl = threadIdx.x * EPV;  // this thread's first column within the slab
  float cs[EPV];
#pragma unroll
  for (int e = 0; e < EPV; ++e) cs[e] = 0.f;
  // this thread's anchors: anc[c0 / 256][row][(c0 % 256) / 64], kAnchorSlots floats per row
  const float* arow = anc + anchor_index(n, r0, c0);
  // rows in groups of U: all U loads in flight before the arithmetic of the group
  constexpr int U = 4;
  for (int t0 = 0; t0 < rows; t0 += U) {
    i32x4 raw[U];
    float an[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (t0 + u < rows) {
        raw[u] = *reinterpret_cast<const i32x4*>(L + (r0 + t0 + u) * V + c0);
        an[u] = arow[(int64_t)(t0 + u) * kAnchorSlots];
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u;
      if (t >= rows) break;
      const T* lv = reinterpret_cast<const T*>(&raw[u]);
      // exp(anchor + offset - lse) = exp2(offset log2(e) + (anchor log2(e) - lse log2(e)))
      const float l2 = fmaf(an[u], kLog2e, -s_lse2[t]);
      float g[EPV];
#pragma unroll
      for (int e = 0; e < EPV; ++e) g[e] = __builtin_amdgcn_exp2f(fmaf(to_f32(lv[e]), kLog2e, l2)) * inv_n;
      const int32_t k = s_cnt[t];
      if (k != 0) {
        const float yn = s_yn[t];
        if (k > 0) {
          for (int32_t q = 0; q < k; ++q) {
            const int d = s_tag[t * MAXT + q] - cl;
            if ((unsigned)d < (unsigned)EPV) {
#pragma unroll
              for (int e = 0; e < EPV; ++e)
                if (d == e) g[e] -= yn;
            }
          }
        } else {
          const int32_t p0 = row_ptr[s_smp[t]], cnt = row_ptr[s_smp[t] + 1] - p0;
          for (int32_t q = 0; q < cnt; ++q) {
            const int d = tag[p0 + q] - c0;
            if ((unsigned)d < (unsigned)EPV) {
#pragma unroll
              for (int e = 0; e < EPV; ++e)
                if (d == e) g[e] -= yn;
            }
          }
        }
      }
      i32x4 outv;
      T* ov = reinterpret_cast<T*>(&outv);
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        cs[e] += g[e];
        ov[e] = from_f32<T>(g[e]);
      }
      // slab-major G ([column slab][n][256 EPV]): a block's stores fill one contiguous run
      T* gdst = slab ? G + ((int64_t)blockIdx.y * n + (r0 + t)) * (256 * EPV) + cl : G + (r0 + t) * V + c0;
      __builtin_nontemporal_store(outv, reinterpret_cast<i32x4*>(gdst));
    }
  }
  float* dst = part_db + (int64_t)blockIdx.x * V + c0;
#pragma unroll
  for (int e = 0; e < EPV; ++e) dst[e] = cs[e];
}

// dbD_e[v] = sum of the piece partials of expert e (pieces piece_start[e] .. piece_start[e+1]),
// in piece order.  Grid: (ceil(V / 256), NG).
__global__ void __launch_bounds__(256) k_piece_colsum(const float* __restrict__ part,
                                                      const int32_t* __restrict__ piece_start, int V,
                                                      float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int e = blockIdx.y;
  if (c >= V) return;
  float s = 0.f;
  for (int q = piece_start[e]; q < piece_start[e + 1]; ++q) s += part[(int64_t)q * V + c];
  out[(int64_t)e * V + c] = s;
}

// out[v] = sum over the rows of part[row][v] (the decoder bias gradient from per-block column
// partials).  A block takes 64 columns; its four waves sum a quarter of the rows each (in row order, four
// rows in flight) and the quarters are added in order, so the result does not depend on timing.
__global__ void __launch_bounds__(256) k_colsum_final(const float* __restrict__ part, int rows, int V,
                                                      float* __restrict__ out) {
  __shared__ float s_q[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  const int per = (rows + 3) / 4;
  const int q0 = w * per, q1 = q0 + per < rows ? q0 + per : rows;
  float s = 0.f;
  if (c < V) {
    int q = q0;
    for (; q + 4 <= q1; q += 4) {
      const float a = part[(int64_t)q * V + c], b = part[(int64_t)(q + 1) * V + c];
      const float d = part[(int64_t)(q + 2) * V + c], e = part[(int64_t)(q + 3) * V + c];
      s = (((s + a) + b) + d) + e;
    }
    for (; q < q1; ++q) s += part[(int64_t)q * V + c];
  }
  s_q[w][lane] = s;
  __syncthreads();
  if (w == 0 && c < V) out[c] = ((s_q[0][lane] + s_q[1][lane]) + s_q[2][lane]) + s_q[3][lane];
}

// dH = G D, written to expert order: dYs[inv[i]] = (G D)[i].  GW > 0: G is slab-major, [V / GW
// slabs][n][GW] (direct-to-LDS engine only).
template <class C, int GW = 0>
__global__ void __launch_bounds__(C::THREADS)
    k_dec_dH(const typename C::type* __restrict__ G, const typename C::type* __restrict__ D, int64_t n, int V, int o,
             const int32_t* __restrict__ inv, typename C::type* __restrict__ dYs) {
  using T = typename C::type;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_plain<C>(n, o, V);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  if constexpr (GW > 0) {
    static_assert(C::DMA, "slab-major G on the direct-to-LDS engine");
    DmaTile<C, true, false, GW> pipe;
    pipe.slab_a(n * GW);
    pipe.prime(G + tc.m0 * GW, GW, tc.m_rows, D + tc.n0, o, tc.n_cols, V, smem);
    pipe.run(smem, acc);
  } else {
    gemm_tile<C, true, false>(G + tc.m0 * V, V, tc.m_rows, D + tc.n0, o, tc.n_cols, V, smem, acc);
  }
  store_out<C, T>(tc, acc, smem, dYs, o, Ident{}, RowVia{inv, tc.m0}, NoVec{});
}

// out [M][N] (fp32) = A^T B, reduction over `rows` rows (A [rows][M], B [rows][N], both
// row-major): the decoder's dD = G^T H and the PCA's covariance and Gram products.  The tiles are
// run in rounds of one per resident workgroup; when the last round is only partly filled, its
// tiles are split over K instead: tiles b < t_full run whole, tile t_full + r (r < R) is computed
// as `split` K-chunks of `chunk` rows (work items t_full + r * split + c, every chunk non-empty)
// whose fp32 partials go to part[r * split + c] and are added in chunk order by k_split_reduce.
constexpr int kMaxSplitItems = 512;

template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_gemm_tn_split(const typename C::type* __restrict__ A, const typename C::type* __restrict__ B, int64_t rows,
                    int M, int N, float* __restrict__ out, int64_t t_full, int split, int64_t chunk,
                    float* __restrict__ part, int64_t a_sstride, int a_sw) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const int64_t T = cdiv(M, C::BM) * cdiv(N, C::BN);
  const int64_t b = blockIdx.x;
  // A's columns m0 .. of a tile: row-major (ld M), or slab-major (a_sw > 0: a tile lies in one
  // slab of a_sw columns, rows a_sw apart)
  auto a_at = [&](int64_t m0) { return a_sw ? A + (m0 / a_sw) * a_sstride + (m0 % a_sw) : A + m0; };
  const int64_t lda = a_sw ? a_sw : M;
  floatx4 acc[C::MI][C::NJ];
  if (b < t_full) {
    const TileCoord tc = tile_plain_at<C>(M, N, (int)rows, b);
    if (!tc.valid) return;
    gemm_tile<C, false, false>(a_at(tc.m0), lda, tc.m_rows, B + tc.n0, N, tc.n_cols, (int)rows, smem, acc);
    store_out<C, float>(tc, acc, smem, out, N, Ident{}, RowId{tc.m0}, NoVec{});
    return;
  }
  const int64_t q = b - t_full;
  const int64_t t = t_full + q / split;
  if (t >= T) return;
  const int c = (int)(q % split);
  const TileCoord tc = tile_plain_at<C>(M, N, (int)rows, t);
  const int64_t k0 = c * chunk;
  const int klen = (int)(rows - k0 < chunk ? rows - k0 : chunk);
  gemm_tile<C, false, false>(a_at(tc.m0) + k0 * lda, lda, tc.m_rows, B + tc.n0 + k0 * N, N, tc.n_cols, klen, smem,
                             acc);
  TileCoord lt = tc;
  lt.m0 = 0;
  lt.n0 = 0;
  store_out<C, float>(lt, acc, smem, part + q * (int64_t)(C::BM * C::BN), C::BN, Ident{}, RowId{0}, NoVec{});
}

template <class C>
__global__ void __launch_bounds__(256) k_split_reduce(const float* __restrict__ part, int64_t rows, int M, int N,
                                                      int64_t t_full, int split, int R, float* __restrict__ out) {
  constexpr int TE = C::BM * C::BN;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)R * TE) return;
  const int r = (int)(idx / TE), e = (int)(idx % TE);
  const int i = e / C::BN, j = e % C::BN;
  const TileCoord tc = tile_plain_at<C>(M, N, (int)rows, t_full + r);
  if (i >= tc.m_rows || j >= tc.n_cols) return;
  float s = 0.f;
  for (int c = 0; c < split; ++c) s += part[((int64_t)r * split + c) * TE + e];
  out[(tc.m0 + i) * (int64_t)N + tc.n0 + j] = s;
}

// Launches k_gemm_tn_split (and its reduction) for out = A^T B; `part` holds kMaxSplitItems
// tiles of fp32 partials.  rows > 0.  a_sw > 0: A is slab-major (see k_gemm_tn_split).
template <class C>
static int launch_tn_split(const char* label, const typename C::type* A, const typename C::type* B, int64_t rows,
                           int M, int N, float* out, float* part, hipStream_t st, int64_t a_sstride = 0,
                           int a_sw = 0) {
  // rounds of `slots` concurrent tiles (one workgroup per 160 KB of LDS per CU)
  const int64_t tiles = cdiv(M, C::BM) * cdiv(N, C::BN);
  int64_t slots = (int64_t)device_cus() * ((160 * 1024) / C::LDS);
  if (slots > kMaxSplitItems) slots = kMaxSplitItems;
  const int64_t R = tiles % slots;
  const int64_t t_full = tiles - R;
  int split = R > 0 ? (int)(slots / R) : 1;
  // chunks of a multiple of 32 rows and at least 256 (fewer chunks when rows are few); split is
  // then recounted so that no chunk is empty
  int64_t chunk = cdiv(cdiv(rows, split), 32) * 32;
  if (chunk < 256) chunk = 256;
  split = (int)cdiv(rows, chunk);
  HMOE_LAUNCH(label, k_gemm_tn_split<C>, dim3((unsigned)(t_full + R * split)), dim3(C::THREADS), C::LDS, st, A, B,
              rows, M, N, out, t_full, split, chunk, part, a_sstride, a_sw);
  if (R > 0)
    HMOE_LAUNCH("split-K reduce", k_split_reduce<C>, dim3((unsigned)cdiv(R * C::BM * C::BN, 256)), dim3(256), 0, st,
                (const float*)part, rows, M, N, t_full, split, (int)R, out);
  return HMOE_OK;
}

// ------------------------------------------------------------------ expert backward

// dW_e = A_e^T B_e over the rows of expert e (reduction-grouped; an empty expert writes zeros).
//   A: [rows][M] (ld M), B: [rows][N] (ld N), out: [G][M][N] fp32.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
    k_expert_wgrad(const typename C::type* __restrict__ A, const typename C::type* __restrict__ B,
                   const int32_t* __restrict__ seg, const int32_t* __restrict__ order, int G, int M, int N,
                   float* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_group_k<C>(seg, order, G, M, N);
  if (!tc.valid) return;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, false, false>(A + tc.k0 * M + tc.m0, M, tc.m_rows, B + tc.k0 * N + tc.n0, N, tc.n_cols, tc.k_len,
                             smem, acc);
  store_out<C, float>(tc, acc, smem, out + (int64_t)tc.group * M * N, N, Ident{}, RowId{tc.m0}, NoVec{});
}

// Zeroes the elements of a stored vector (16 bytes from store_tile, four elements from
// store_direct) where the saved activation is not positive.
template <typename T>
struct ReluMask {
  const T* __restrict__ H1s;
  int64_t m0;
  int N, n0;
  template <typename V>
  __device__ __forceinline__ V operator()(int64_t, int row, int col, V v) const {
    constexpr int E = sizeof(V) / sizeof(T);
    const V h = *reinterpret_cast<const V*>(H1s + (m0 + row) * N + n0 + col);
    const T* hv = reinterpret_cast<const T*>(&h);
    T* vv = reinterpret_cast<T*>(&v);
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (!(to_f32(hv[e]) > 0.f)) vv[e] = from_f32<T>(0.f);
    return v;
  }
};

// Row-grouped input gradients.  MASK: dZ[m] = (dYs[m] W2_e) * [H1s[m] > 0], stored in expert
// order.  !MASK: dX[perm[m]] = dZ[m] W1_e, stored in sample order (in slot order, row m, when
// perm is NULL: the per-expert decoders' dH = g D_e).
//   A: [rows][Kd] (ld Kd), W: [G][Kd][N] (the layer's [out][in] weights seen as [K][N]).
template <class C, bool MASK>
__device__ __forceinline__ void expert_dgrad_tile(const TileCoord& tc, const typename C::type* __restrict__ A,
                                                  const typename C::type* __restrict__ W, int N, int Kd,
                                                  const typename C::type* __restrict__ H1s,
                                                  const int32_t* __restrict__ perm,
                                                  typename C::type* __restrict__ out, lds<char>* smem) {
  using T = typename C::type;
  floatx4 acc[C::MI][C::NJ];
  gemm_tile<C, true, false>(A + tc.m0 * Kd, Kd, tc.m_rows, W + (int64_t)tc.group * Kd * N + tc.n0, N, tc.n_cols,
                            Kd, smem, acc);
  if (MASK)
    store_out<C, T>(tc, acc, smem, out, N, Ident{}, RowId{tc.m0}, ReluMask<T>{H1s, tc.m0, N, tc.n0});
  else if (perm)
    store_out<C, T>(tc, acc, smem, out, N, Ident{}, RowVia{perm, tc.m0}, NoVec{});
  else
    store_out<C, T>(tc, acc, smem, out, N, Ident{}, RowId{tc.m0}, NoVec{});
}

template <class C, bool MASK, bool XCD = false>
__global__ void __launch_bounds__(C::THREADS)
    k_expert_dgrad(const typename C::type* __restrict__ A, const typename C::type* __restrict__ W,
                   const int32_t* __restrict__ seg, const int32_t* __restrict__ tile_start, int G, int N, int Kd,
                   const typename C::type* __restrict__ H1s, const int32_t* __restrict__ perm,
                   typename C::type* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds<char>* smem = (lds<char>*)smem_raw;
  const TileCoord tc = tile_group_m<C, XCD>(seg, tile_start, G, N, Kd);
  if (!tc.valid) return;
  by_tile_height<C>(tc, [&](auto cfg) {
    expert_dgrad_tile<decltype(cfg), MASK>(tc, A, W, N, Kd, H1s, perm, out, smem);
  });
}

// ------------------------------------------------------------------ launchers

struct MoeShape {
  int64_t n;
  int K, d, h, o, V;
  int nd;  // decoders: 1 shared, or K (one per expert)
};

static MoeShape shape_of(const hmoe_moe_params_t* p, int64_t n) {
  return MoeShape{n, p->K, p->d_in, p->d_hid, p->d_out, p->vocab, p->decoders > 1 ? p->decoders : 1};
}

template <typename T>
static size_t fwd_ws(const MoeShape& s) {
  using C = typename Pick<T>::C;
  Workspace ws(nullptr, 0);
  const int64_t ntv = cdiv(s.V, C::BN);
  ws.take<int32_t>(s.K + 1);
  ws.take<float>((size_t)ntv * s.n);
  ws.take<float>((size_t)ntv * s.n);
  if (s.nd > 1) ws.take<T>((size_t)s.n * s.o);
  ws.take<double>(kSumBlocks);
  return ws.off;
}

template <typename T>
static size_t bwd_ws(const MoeShape& s) {
  using C = typename Pick<T>::C;
  Workspace ws(nullptr, 0);
  ws.take<int32_t>(s.K + 1);
  ws.take<int32_t>(s.K);
  constexpr int GW = 256 * (16 / (int)sizeof(T));  // G padded to whole slabs (backward_t)
  ws.take<T>(sizeof(T) == 2 && s.nd == 1 ? (size_t)s.n * cdiv(s.V, GW) * GW : (size_t)s.n * s.V);
  ws.take<T>((size_t)s.n * s.o);
  ws.take<T>((size_t)s.n * s.h);
  const int64_t prow = cdiv(s.n, C::BM) > cdiv(s.n, kGradRows) ? cdiv(s.n, C::BM) : cdiv(s.n, kGradRows);
  ws.take<float>((size_t)(prow + s.K) * s.V);
  ws.take<float>((size_t)kMaxSplitItems * C::BM * C::BN);
  if (s.nd > 1) {
    ws.take<T>((size_t)s.n * s.o);
    ws.take<int32_t>(s.K + 1);
  }
  const int w = s.h > s.o ? s.h : s.o;
  return ws.off + segsum_ws(s.n, s.K, w) + 256;
}

size_t moe_ws_bytes(const hmoe_moe_params_t* p, int64_t n) {
  const MoeShape s = shape_of(p, n);
  const size_t a = p->dt == HMOE_BF16 ? fwd_ws<bf16>(s) : fwd_ws<float>(s);
  const size_t b = p->dt == HMOE_BF16 ? bwd_ws<bf16>(s) : bwd_ws<float>(s);
  return a > b ? a : b;
}

template <typename T>
static int forward_t(const hmoe_moe_params_t* p, int64_t n, const T* Xs, const int32_t* offsets, const int32_t* perm,
                     const hmoe_labels_t* y, T* H1s, T* H, T* Lg, float* anc, float* lse, float* loss,
                     float* loss_mean, Workspace& ws, hipStream_t st) {
  using C = typename Pick<T>::C;
  const MoeShape s = shape_of(p, n);
  const int ntv = (int)cdiv(s.V, C::BN);
  int32_t* ts = ws.take<int32_t>(s.K + 1);
  float* pm = ws.take<float>((size_t)ntv * n);
  float* ps = ws.take<float>((size_t)ntv * n);
  T* Hs = s.nd > 1 ? ws.take<T>((size_t)n * s.o) : nullptr;  // H in slot order
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const T* W1 = (const T*)p->W1;
  const T* W2 = (const T*)p->W2;
  const T* D = (const T*)p->D;
  if (!Lg) anc = nullptr;
  HMOE_TRY(launch_seg_tiles(offsets, s.K, C::BM, ts, st));
  const int64_t mt_bound = cdiv(n, C::BM) + s.K;
  HMOE_LAUNCH("expert layer 1", (k_expert_fwd<C, 1>), dim3((unsigned)(mt_bound * cdiv(s.h, C::BN))),
              dim3(C::THREADS), C::LDS, st, Xs, W1, (const T*)p->b1, offsets, ts, s.K, s.h, s.d, perm, H1s);
  HMOE_LAUNCH("expert layer 2", (k_expert_fwd<C, 2>), dim3((unsigned)(mt_bound * cdiv(s.o, C::BN))),
              dim3(C::THREADS), C::LDS, st, (const T*)H1s, W2, (const T*)p->b2, offsets, ts, s.K, s.o, s.h,
              perm, H);
  if (s.nd > 1) {
    // one decoder per expert: decode in slot order
    HMOE_TRY(launch_permute(H, Hs, perm, n, s.o, p->dt, st));
    HMOE_LAUNCH("decoder forward", k_dec_fwd_grouped<C>, dim3((unsigned)(mt_bound * ntv)), dim3(C::THREADS), C::LDS,
                st, (const T*)Hs, D, (const T*)p->bD, offsets, ts, s.K, n, s.V, s.o, pm, ps, Lg, anc);
    HMOE_LAUNCH("decoder loss", k_dec_loss<T>, dim3((unsigned)cdiv(n, kLossRows)), dim3(256), 0, st, pm, ps, ntv,
                (const T*)Hs, D, (const T*)p->bD, n, s.o, s.V, perm, offsets, s.K, y->row_ptr, y->tag, lse, loss);
    return launch_sum_f32(loss, n, 1.0 / (double)n, nullptr, loss_mean, ws, st);
  }
  if constexpr (C::DMA) {
    // persistent: one workgroup per resident slot
    const int64_t tiles = cdiv(n, C::BM) * ntv;
    constexpr int lds_bytes = C::LDS + 2 * kDecStatLds;
    int64_t slots = (int64_t)device_cus() * ((160 * 1024) / lds_bytes);
    if (slots > tiles) slots = tiles;
    HMOE_LAUNCH("decoder forward", k_dec_fwd_stream<C>, dim3((unsigned)slots), dim3(C::THREADS), lds_bytes, st,
                (const bf16*)H, (const bf16*)D, (const bf16*)p->bD, n, s.V, s.o, pm, ps, (bf16*)Lg, anc);
  } else {
    HMOE_LAUNCH("decoder forward", k_dec_fwd<C>, dim3((unsigned)(cdiv(n, C::BM) * ntv)), dim3(C::THREADS), C::LDS,
                st, (const T*)H, D, (const T*)p->bD, n, s.V, s.o, pm, ps, Lg, anc);
  }
  HMOE_LAUNCH("decoder loss", k_dec_loss<T>, dim3((unsigned)cdiv(n, kLossRows)), dim3(256), 0, st, pm, ps, ntv, (const T*)H, D,
              (const T*)p->bD, n, s.o, s.V, (const int32_t*)nullptr, (const int32_t*)nullptr, 0, y->row_ptr,
              y->tag, lse, loss);
  return launch_sum_f32(loss, n, 1.0 / (double)n, nullptr, loss_mean, ws, st);
}

template <typename T>
static int backward_t(const hmoe_moe_params_t* p, int64_t n, const T* Xs, const int32_t* offsets, const int32_t* perm,
                      const int32_t* inv, const hmoe_labels_t* y, const T* H1s, const T* H, const T* Lg,
                      const float* anc, const float* lse, float* dW1, float* db1, float* dW2, float* db2, float* dD, float* dbD, T* dX,
                      Workspace& ws, hipStream_t st) {
  using C = typename Pick<T>::C;
  const MoeShape s = shape_of(p, n);
  int32_t* ts = ws.take<int32_t>(s.K + 1);
  int32_t* order = ws.take<int32_t>(s.K);
  constexpr int EPV = 16 / sizeof(T);
  // bf16 logits through the shared decoder: G slab-major, [V / GW slabs][n][GW] (see
  // k_dec_grad_elem), which the grad kernel writes contiguously; the last slab is padded.
  constexpr int GW = 256 * EPV;
  const bool slab = sizeof(T) == 2 && Lg && s.nd == 1;
  T* G = ws.take<T>(slab ? (size_t)n * cdiv(s.V, GW) * GW : (size_t)n * s.V);
  T* dYs = ws.take<T>((size_t)n * s.o);
  T* dZ = ws.take<T>((size_t)n * s.h);
  const int mt = (int)cdiv(n, C::BM);
  const int gr = (int)cdiv(n, kGradRows);
  float* pdb = ws.take<float>((size_t)((mt > gr ? mt : gr) + s.K) * s.V);
  float* split_part = ws.take<float>((size_t)kMaxSplitItems * C::BM * C::BN);
  T* Hs = nullptr;
  int32_t* gts = nullptr;
  if (s.nd > 1) {
    Hs = ws.take<T>((size_t)n * s.o);  // H in slot order
    gts = ws.take<int32_t>(s.K + 1);   // first gradient piece of each expert
  }
  if (!ws.fits()) return HMOE_EWORKSPACE;
  const T* W1 = (const T*)p->W1;
  const T* W2 = (const T*)p->W2;
  const T* D = (const T*)p->D;
  const int ntv = (int)cdiv(s.V, C::BN);
  const int64_t mt_bound = cdiv(n, C::BM) + s.K;
  HMOE_TRY(launch_seg_tiles(offsets, s.K, C::BM, ts, st));
  HMOE_TRY(launch_seg_order(offsets, s.K, order, st));
  if (s.nd > 1) {
    // One decoder per expert, everything in slot order (the API guarantees saved logits):
    // g from the stored logits in pieces that stay within one expert, dbD_e from the pieces'
    // column sums, dH = g D_e (row-grouped), dD_e = g_e^T H_e (reduction-grouped).
    HMOE_TRY(launch_seg_tiles(offsets, s.K, kGradRows, gts, st));
    HMOE_LAUNCH("decoder grad", k_dec_grad_elem<T>, dim3((unsigned)(gr + s.K), (unsigned)cdiv(s.V, 256 * EPV)),
                dim3(256), 0, st, Lg, anc, lse, y->row_ptr, y->tag, n, s.V, (float)(1.0 / (double)n), perm, offsets,
                gts, s.K, G, pdb, 0);
    if (dbD)
      HMOE_LAUNCH("decoder bias grad", k_piece_colsum, dim3((unsigned)cdiv(s.V, 256), (unsigned)s.K), dim3(256), 0,
                  st, pdb, gts, s.V, dbD);
    HMOE_TRY(launch_permute(H, Hs, perm, n, s.o, p->dt, st));
    // XCD-grouped tile order: the o / BN tiles of an m-tile share one G row block (V wide)
    HMOE_LAUNCH("decoder dH", (k_expert_dgrad<C, false, true>),
                dim3((unsigned)(cdiv(mt_bound, 64) * 64 * cdiv(s.o, C::BN))), dim3(C::THREADS), C::LDS, st,
                (const T*)G, D, offsets, ts, s.K, s.o, s.V, (const T*)nullptr, (const int32_t*)nullptr, dYs);
    HMOE_LAUNCH("decoder dD", k_expert_wgrad<C>,
                dim3((unsigned)((int64_t)s.K * cdiv(s.V, C::BM) * cdiv(s.o, C::BN))), dim3(C::THREADS), C::LDS, st,
                (const T*)G, (const T*)Hs, offsets, order, s.K, s.V, s.o, dD);
  } else {
  int prow;
  if (Lg) {
    HMOE_LAUNCH("decoder grad", k_dec_grad_elem<T>, dim3((unsigned)gr, (unsigned)cdiv(s.V, 256 * EPV)), dim3(256),
                0, st, Lg, anc, lse, y->row_ptr, y->tag, n, s.V, (float)(1.0 / (double)n), (const int32_t*)nullptr,
                (const int32_t*)nullptr, (const int32_t*)nullptr, 0, G, pdb, (int)slab);
    prow = gr;
  } else {
    HMOE_LAUNCH("decoder grad", k_dec_grad<C>, dim3((unsigned)(mt * ntv)), dim3(C::THREADS), C::LDS, st, H, D,
                (const T*)p->bD, n, s.V, s.o, lse, y->row_ptr, y->tag, (float)(1.0 / (double)n), G, pdb);
    prow = mt;
  }
  if (dbD)
    HMOE_LAUNCH("decoder bias grad", k_colsum_final, dim3((unsigned)cdiv(s.V, 64)), dim3(256), 0, st, pdb, prow,
                s.V, dbD);
  if constexpr (sizeof(T) == 2) {
    if (slab) {
      HMOE_LAUNCH("decoder dH", (k_dec_dH<C, GW>), dim3((unsigned)(mt * cdiv(s.o, C::BN))), dim3(C::THREADS),
                  C::LDS, st, (const T*)G, D, n, s.V, s.o, inv, dYs);
      HMOE_TRY(launch_tn_split<C>("decoder dD", (const T*)G, H, n, s.V, s.o, dD, split_part, st, n * GW, GW));
    }
  }
  if (!slab) {
    HMOE_LAUNCH("decoder dH", k_dec_dH<C>, dim3((unsigned)(mt * cdiv(s.o, C::BN))), dim3(C::THREADS), C::LDS, st,
                (const T*)G, D, n, s.V, s.o, inv, dYs);
    HMOE_TRY(launch_tn_split<C>("decoder dD", (const T*)G, H, n, s.V, s.o, dD, split_part, st));
  }
  }
  // experts
  const size_t mark = ws.off;
  if (db2) HMOE_TRY(launch_segsum<T, float>(dYs, s.o, nullptr, offsets, s.K, s.o, n, db2, 0, ws, st));
  ws.off = mark;
  HMOE_LAUNCH("expert dW2", k_expert_wgrad<C>, dim3((unsigned)((int64_t)s.K * cdiv(s.o, C::BM) * cdiv(s.h, C::BN))),
              dim3(C::THREADS), C::LDS, st, (const T*)dYs, H1s, offsets, order, s.K, s.o, s.h, dW2);
  HMOE_LAUNCH("expert dH1", (k_expert_dgrad<C, true>), dim3((unsigned)(mt_bound * cdiv(s.h, C::BN))),
              dim3(C::THREADS), C::LDS, st, (const T*)dYs, W2, offsets, ts, s.K, s.h, s.o, H1s, perm, dZ);
  if (db1) HMOE_TRY(launch_segsum<T, float>(dZ, s.h, nullptr, offsets, s.K, s.h, n, db1, 0, ws, st));
  ws.off = mark;
  HMOE_LAUNCH("expert dW1", k_expert_wgrad<C>, dim3((unsigned)((int64_t)s.K * cdiv(s.h, C::BM) * cdiv(s.d, C::BN))),
              dim3(C::THREADS), C::LDS, st, (const T*)dZ, Xs, offsets, order, s.K, s.h, s.d, dW1);
  if (dX)
    HMOE_LAUNCH("expert dX", (k_expert_dgrad<C, false>), dim3((unsigned)(mt_bound * cdiv(s.d, C::BN))),
                dim3(C::THREADS), C::LDS, st, (const T*)dZ, W1, offsets, ts, s.K, s.d, s.h,
                (const T*)nullptr, perm, dX);
  return HMOE_OK;
}

// ------------------------------------------------------------------ plain products (the PCA)

// seg = {0, rows}: one group for the grouped kernels below.
static __global__ void k_seg_one(int32_t* __restrict__ seg, int64_t rows) {
  if (threadIdx.x == 0) {
    seg[0] = 0;
    seg[1] = (int32_t)rows;
  }
}

// out [M][N] fp32 = A^T B over `rows` rows (A [rows][M], B [rows][N]), split over K when the
// tiles alone would leave most of the chip idle.
template <typename T>
size_t gemm_tn_ws() {
  using C = typename Pick<T>::C;
  return ((size_t)kMaxSplitItems * C::BM * C::BN) * sizeof(float) + 256;
}

template <typename T>
int launch_gemm_tn(const T* A, const T* B, int64_t rows, int M, int N, float* out, Workspace& ws, hipStream_t st,
                   const char* label) {
  using C = typename Pick<T>::C;
  float* part = ws.take<float>((size_t)kMaxSplitItems * C::BM * C::BN);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  if (rows <= 0) return launch_zero_f32(out, (int64_t)M * N, st);
  return launch_tn_split<C>(label, A, B, rows, M, N, out, part, st);
}

// out [rows][N] = A W (A [rows][Kd], W [Kd][N]), in the data dtype: the row-grouped kernel with
// a single group.
template <typename T>
int launch_gemm_nn(const T* A, const T* W, int64_t rows, int Kd, int N, T* out, Workspace& ws, hipStream_t st) {
  using C = typename Pick<T>::C;
  int32_t* seg = ws.take<int32_t>(2);
  int32_t* ts = ws.take<int32_t>(2);
  if (!ws.fits()) return HMOE_EWORKSPACE;
  HMOE_LAUNCH("one segment", k_seg_one, dim3(1), dim3(64), 0, st, seg, rows);
  HMOE_TRY(launch_seg_tiles(seg, 1, C::BM, ts, st));
  HMOE_LAUNCH("gemm nn", (k_expert_dgrad<C, false>), dim3((unsigned)((cdiv(rows, C::BM) + 1) * cdiv(N, C::BN))),
              dim3(C::THREADS), C::LDS, st, A, W, seg, ts, 1, N, Kd, (const T*)nullptr, (const int32_t*)nullptr, out);
  return HMOE_OK;
}

template size_t gemm_tn_ws<float>();
template size_t gemm_tn_ws<bf16>();
template int launch_gemm_tn<float>(const float*, const float*, int64_t, int, int, float*, Workspace&, hipStream_t,
                                   const char*);
template int launch_gemm_tn<bf16>(const bf16*, const bf16*, int64_t, int, int, float*, Workspace&, hipStream_t,
                                  const char*);
template int launch_gemm_nn<float>(const float*, const float*, int64_t, int, int, float*, Workspace&, hipStream_t);

int launch_moe_forward(const hmoe_moe_params_t* p, int64_t n, const void* Xs, const int32_t* offsets,
                       const int32_t* perm, const hmoe_labels_t* y, void* H1s, void* H, void* logits, float* anc,
                       float* lse, float* loss, float* loss_mean, Workspace& ws, hipStream_t st) {
  if (p->dt == HMOE_BF16)
    return forward_t<bf16>(p, n, (const bf16*)Xs, offsets, perm, y, (bf16*)H1s, (bf16*)H, (bf16*)logits, anc, lse,
                           loss, loss_mean, ws, st);
  return forward_t<float>(p, n, (const float*)Xs, offsets, perm, y, (float*)H1s, (float*)H, (float*)logits, anc, lse,
                          loss, loss_mean, ws, st);
}

int launch_moe_backward(const hmoe_moe_params_t* p, int64_t n, const void* Xs, const int32_t* offsets,
                        const int32_t* perm, const int32_t* inv, const hmoe_labels_t* y, const void* H1s,
                        const void* H, const void* logits, const float* anc, const float* lse, float* dW1,
                        float* db1, float* dW2, float* db2, float* dD, float* dbD, void* dX, Workspace& ws,
                        hipStream_t st) {
  if (p->dt == HMOE_BF16)
    return backward_t<bf16>(p, n, (const bf16*)Xs, offsets, perm, inv, y, (const bf16*)H1s, (const bf16*)H,
                            (const bf16*)logits, anc, lse, dW1, db1, dW2, db2, dD, dbD, (bf16*)dX, ws, st);
  return backward_t<float>(p, n, (const float*)Xs, offsets, perm, inv, y, (const float*)H1s, (const float*)H,
                           (const float*)logits, anc, lse, dW1, db1, dW2, db2, dD, dbD, (float*)dX, ws, st);
}

}  // namespace hmoe
