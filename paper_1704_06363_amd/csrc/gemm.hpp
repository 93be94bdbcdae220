// gemm.hpp -- the MFMA tile engines shared by every dense contraction of the hot path: the
// register-staged engine described first (Cfg) and the direct-to-LDS engine further down
// (CfgD), which runs the bf16 MoE contractions, the larger assignments and the fp32
// contractions with K-contiguous operands.
//
// C[m, n] = sum_k A(m, k) * B(n, k) over one BM x BN output tile per workgroup, split into
// (BM/WM) x (BN/WN) wavefronts of WM x WN.  Operands are staged through LDS in a row-major,
// K-contiguous layout whatever their layout in HBM:
//   K-contiguous operand (stored [rows][K]): 16-byte vector loads go straight to LDS;
//   K-strided operand    (stored [K][rows]): each thread loads a block of K-rows x 4 rows --
//                        8 x 4 for bf16, 4 x 4 for fp32 -- and transposes it in registers, so
//                        the LDS store is again one 16-byte vector (one chunk) per row.
// One stage covers 128 bytes of K per row (64 bf16 or 32 fp32), i.e. 8 chunks of 16 bytes.
// LDS rows are not padded; chunk c of row r lives at chunk c ^ ((r ^ (r >> 2)) & 7).  That
// XOR pattern was chosen by measuring the LDS bank-conflict counter on gfx950 for the three
// access patterns used here -- MFMA operand reads (16 consecutive rows, one chunk per 16
// lanes), direct stores (one row, 8 chunks per 8 lanes) and transposed stores (rows four
// apart) -- and is conflict-free for all of them (r ^ (r >> 3), for instance, is 2-way
// conflicted on the operand reads).
// bf16 uses v_mfma_f32_16x16x32_bf16 (8 consecutive k per lane); fp32 uses
// v_mfma_f32_16x16x4_f32 fed from the same 16-byte LDS reads (4 consecutive k per lane,
// consumed by 4 MFMAs).  Accumulation is fp32.  The K loop is double-buffered: the next
// stage's global loads are in flight while the current stage feeds the MFMAs.
//
// Accumulator ownership (verified layout of the 16x16 MFMA outputs): lane l of wave w holds,
// for sub-tile (i, j) and r = 0..3,
//   row = wm * WM + 16 i + 4 (l / 16) + r,     col = wn * WN + 16 j + (l % 16),
// with wm = w / (BN / WN), wn = w % (BN / WN).
#pragma once
#include "common.hpp"

namespace hmoe {

constexpr int kStageRowBytes = 128;  // K extent of one stage, in bytes

template <typename T, int BM_, int BN_, int WM_, int WN_>
struct Cfg {
  using type = T;
  static constexpr bool DMA = false;  // register-staged engine
  static constexpr bool TRANS = false;  // accumulator element (i, j, r) at row 16 i + 4 (l / 16) + r, col 16 j + l % 16
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int WAVES_N = BN / WN, WAVES_M = BM / WM;
  static constexpr int WAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int MI = WM / 16, NJ = WN / 16;
  static constexpr int EPV = 16 / sizeof(T);             // elements per 16-byte vector
  static constexpr int BK = kStageRowBytes / sizeof(T);  // K per stage
  static constexpr int A_BYTES = BM * kStageRowBytes, B_BYTES = BN * kStageRowBytes;
  static constexpr int LDS = 2 * (A_BYTES + B_BYTES);
};

// fp32 GEMMs and narrow problems: 128 x 128 tiles, four waves of 64 x 64.
template <typename T>
using CfgSmall = Cfg<T, 128, 128, 64, 64>;
// Few columns (the gater's assignment with K <= 64 centres): 256 x 64 tiles, four waves of
// 64 x 64 stacked along the rows, so no MFMA work is spent on absent centres.
template <typename T>
using CfgNarrow = Cfg<T, 256, 64, 64, 64>;

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kStageRowBytes + ((chunk ^ ((row ^ (row >> 2)) & 7)) << 4);
}

// ------------------------------------------------------------------ operand staging

// One ROWS-row operand tile of one K stage, held in registers between the global loads and
// the LDS store.  Rows >= rows_valid and K positions >= k_valid read as zero.
template <typename T, int ROWS, int THREADS, bool KCONTIG>
struct Stager {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr bool BF = sizeof(T) == 2;
  // K-contiguous: ROWS * 8 vectors of 16 bytes.
  // K-strided bf16: ROWS / 4 * 8 pieces of 8 K-rows x 4 rows, loaded as 8-byte rows.
  // K-strided fp32: ROWS / 4 * 8 blocks of 4 K-rows x 4 rows, loaded as 16-byte rows.
  static constexpr int NPIECE = KCONTIG ? 0 : (ROWS / 4) * 8 / THREADS;
  static constexpr int NV = KCONTIG ? ROWS * 8 / THREADS : (BF ? NPIECE * 4 : NPIECE * 4);
  static_assert(KCONTIG ? (ROWS * 8) % THREADS == 0 : ((ROWS / 4) * 8) % THREADS == 0, "tile/threads");
  i32x4 v[NV];

  // K-contiguous: element (r, k) at base + r * ld + k (k_valid a multiple of EPV).
  // K-strided:    element (r, k) at base + k * ld + r (rows_valid a multiple of 4).
  __device__ __forceinline__ void load(const T* __restrict__ base, int64_t ld, int rows_valid, int k0,
                                       int k_valid) {
    const int t = threadIdx.x;
    if constexpr (KCONTIG) {
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int vi = t + THREADS * q;
        const int r = vi >> 3;
        const int k = k0 + (vi & 7) * EPV;
        if (r < rows_valid && k < k_valid)
          v[q] = *reinterpret_cast<const i32x4*>(base + (int64_t)r * ld + k);
        else
          v[q] = i32x4{0, 0, 0, 0};
      }
    } else {
      constexpr int RQ = ROWS / 4;  // groups of 4 rows
#pragma unroll
      for (int q = 0; q < NPIECE; ++q) {
        const int pc = t + THREADS * q;
        const int r = (pc % RQ) * 4;
        const int kb = pc / RQ;  // which 16-byte chunk of the stage
        if constexpr (BF) {
          // 8 K-rows x 4 bf16: two K-rows per i32x4 (low pair from even, high pair from odd)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int k = k0 + kb * 8 + 2 * i;
            uint2 e = make_uint2(0u, 0u), o = make_uint2(0u, 0u);
            if (r < rows_valid && k < k_valid) e = *reinterpret_cast<const uint2*>(base + (int64_t)k * ld + r);
            if (r < rows_valid && k + 1 < k_valid) o = *reinterpret_cast<const uint2*>(base + (int64_t)(k + 1) * ld + r);
            v[q * 4 + i] = i32x4{(int)e.x, (int)e.y, (int)o.x, (int)o.y};
          }
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int k = k0 + kb * 4 + i;
            if (r < rows_valid && k < k_valid)
              v[q * 4 + i] = *reinterpret_cast<const i32x4*>(base + (int64_t)k * ld + r);
            else
              v[q * 4 + i] = i32x4{0, 0, 0, 0};
          }
        }
      }
    }
  }

  __device__ __forceinline__ void store(lds<char>* dst) const {
    const int t = threadIdx.x;
    if constexpr (KCONTIG) {
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int vi = t + THREADS * q;
        *reinterpret_cast<lds<i32x4>*>(dst + swz(vi >> 3, vi & 7)) = v[q];
      }
    } else {
      constexpr int RQ = ROWS / 4;
#pragma unroll
      for (int q = 0; q < NPIECE; ++q) {
        const int pc = t + THREADS * q;
        const int r0 = (pc % RQ) * 4;
        const int kb = pc / RQ;
        if constexpr (BF) {
          // v[q*4+i] = (K-row 2i: rows r0..r0+3 as 2 words, K-row 2i+1: 2 words).
          // Output row j = 8 consecutive K values: word p = (K-row 2p, K-row 2p+1) of row j.
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int word = j >> 1;
            const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
            uint32_t o[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) {
              const uint32_t a = (uint32_t)v[q * 4 + p][word];      // K-row 2p
              const uint32_t c = (uint32_t)v[q * 4 + p][2 + word];  // K-row 2p+1
              o[p] = __builtin_amdgcn_perm(c, a, sel);
            }
            *reinterpret_cast<lds<i32x4>*>(dst + swz(r0 + j, kb)) = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
          }
        } else {
          const i32x4 s0 = v[q * 4 + 0], s1 = v[q * 4 + 1], s2 = v[q * 4 + 2], s3 = v[q * 4 + 3];
          *reinterpret_cast<lds<i32x4>*>(dst + swz(r0 + 0, kb)) = i32x4{s0[0], s1[0], s2[0], s3[0]};
          *reinterpret_cast<lds<i32x4>*>(dst + swz(r0 + 1, kb)) = i32x4{s0[1], s1[1], s2[1], s3[1]};
          *reinterpret_cast<lds<i32x4>*>(dst + swz(r0 + 2, kb)) = i32x4{s0[2], s1[2], s2[2], s3[2]};
          *reinterpret_cast<lds<i32x4>*>(dst + swz(r0 + 3, kb)) = i32x4{s0[3], s1[3], s2[3], s3[3]};
        }
      }
    }
  }

  // Squared norms of the K-contiguous rows this thread staged: xs[q] gets row
  // (threadIdx.x + THREADS * q) >> 3; the 8 lanes sharing a row together hold its full norm.
  __device__ __forceinline__ void add_sq(float* xs) const {
    static_assert(KCONTIG, "row norms need a K-contiguous operand");
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const T* e = reinterpret_cast<const T*>(&v[q]);
#pragma unroll
      for (int z = 0; z < EPV; ++z) {
        const float f = to_f32(e[z]);
        xs[q] += f * f;
      }
    }
  }
};

// ------------------------------------------------------------------ MFMA stage

template <class C>
__device__ __forceinline__ void mfma_stage(const lds<char>* ldsA, const lds<char>* ldsB,
                                           floatx4 (&acc)[C::MI][C::NJ]) {
  const int l = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w / C::WAVES_N, wn = w % C::WAVES_N;
  const int lr = l & 15, lg = l >> 4;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int chunk = 4 * s + lg;
    i32x4 a[C::MI], b[C::NJ];
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
      a[i] = *reinterpret_cast<const lds<i32x4>*>(ldsA + swz(wm * C::WM + 16 * i + lr, chunk));
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
      b[j] = *reinterpret_cast<const lds<i32x4>*>(ldsB + swz(wn * C::WN + 16 * j + lr, chunk));
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
#pragma unroll
      for (int j = 0; j < C::NJ; ++j) {
        if constexpr (sizeof(typename C::type) == 2) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
        } else {
          const floatx4 af = __builtin_bit_cast(floatx4, a[i]);
          const floatx4 bf = __builtin_bit_cast(floatx4, b[j]);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[e], bf[e], acc[i][j], 0, 0, 0);
        }
      }
    }
  }
}

// Full K loop for one tile.  A rows [0, a_rows), B rows [0, b_rows), K positions [0, k_len).
// With ROWNORM (K-contiguous A only) xs[] collects squared row norms of A (see add_sq).
template <class C, bool A_KC, bool B_KC, bool ROWNORM = false>
__device__ __forceinline__ void gemm_tile_reg(const typename C::type* __restrict__ A, int64_t lda, int a_rows,
                                          const typename C::type* __restrict__ B, int64_t ldb, int b_rows,
                                          int k_len, lds<char>* smem, floatx4 (&acc)[C::MI][C::NJ],
                                          float* xs = nullptr) {
  using T = typename C::type;
  using SA = Stager<T, C::BM, C::THREADS, A_KC>;
  static_assert(!C::DMA, "register-staged engine");
  using SB = Stager<T, C::BN, C::THREADS, B_KC>;
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NJ; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  if constexpr (ROWNORM) {
#pragma unroll
    for (int q = 0; q < SA::NV; ++q) xs[q] = 0.f;
  }
  const int nk = (int)cdiv(k_len, C::BK);
  if (nk == 0) return;
  SA sa;
  SB sb;
  lds<char>* const bufA0 = smem;
  lds<char>* const bufB0 = smem + 2 * C::A_BYTES;
  sa.load(A, lda, a_rows, 0, k_len);
  sb.load(B, ldb, b_rows, 0, k_len);
  if constexpr (ROWNORM) sa.add_sq(xs);
  sa.store(bufA0);
  sb.store(bufB0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      sa.load(A, lda, a_rows, (kt + 1) * C::BK, k_len);
      sb.load(B, ldb, b_rows, (kt + 1) * C::BK, k_len);
    }
    mfma_stage<C>(bufA0 + cur * C::A_BYTES, bufB0 + cur * C::B_BYTES, acc);
    if (more) {
      if constexpr (ROWNORM) sa.add_sq(xs);
      sa.store(bufA0 + (cur ^ 1) * C::A_BYTES);
      sb.store(bufB0 + (cur ^ 1) * C::B_BYTES);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ direct-to-LDS engine
//
// The same BM x BN tile and wave split (bf16; fp32 for K-contiguous operands, see CfgD), but
// operands travel from HBM to LDS without passing through registers: global_load_lds_dwordx4 writes lane l's 16 bytes to LDS at (wave-uniform
// base) + 16 l, so the LDS layout -- including its bank swizzle -- is chosen by the global
// address each lane loads.  A stage covers 32 K (64 bytes per row); NS stages form a ring and
// the loads for stage kt + NS - 1 are issued while stage kt feeds the MFMAs, each wave waiting
// (vmcnt) only for its own loads of the stage it is about to read.
//   K-contiguous operand: LDS [rows][32 K] (64-byte rows, chunk c of row r at c ^ ((r >> 1) & 3));
//                         MFMA operands come from one ds_read_b128 per 16 x 32 fragment.
//   K-strided operand:    LDS [32 K][rows] as in HBM (rows contiguous, 16-byte chunk c of K-row
//                         k at c ^ 2 ((k & 3) | ((k >> 1) & 4))); MFMA operands come from two
//                         ds_read_b64_tr_b16 per fragment.  Within each 16-lane group that read
//                         returns to lane i, slot s, element i % 4 of the 8 bytes addressed by lane
//                         4 s + i / 4 (verified on gfx950), so lane j addressing K-row
//                         8 (l / 16) + 4 h + j / 4, rows 4 (j % 4) .. + 3 gives every lane the 4
//                         consecutive K of its own row that the MFMA layout expects.
// Both swizzles make the MFMA operand reads conflict-free (checked with the LDS bank-conflict
// counter).  Rows past the valid range load a clamped (valid) address -- they only feed
// output rows / columns that are never stored -- and a last partial K stage is staged through
// registers with zero fill.  Needs every row width (ld) and valid row count in the row
// direction of a K-strided operand to be a multiple of 8 elements.

// fp32 operands (F32) take the same path for contractions with both operands K-contiguous: the
// engine stages 16-bit units (a float is two, every ld and K doubled), so a 64-byte row still
// holds one stage, and each 16-byte fragment -- four consecutive K of one row -- feeds four
// v_mfma_f32_16x16x4_f32, the lane group g supplying K = 4 g + q to the q-th of them.
template <typename T, int BM_, int BN_, int WM_, int WN_, int NS_>
struct CfgD {
  using type = T;
  static constexpr bool F32 = sizeof(T) == 4;
  static constexpr bool DMA = true;
  static constexpr bool TRANS = true;  // accumulator element (i, j, r) at row 16 i + l % 16, col 16 j + 4 (l / 16) + r
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int WAVES_N = BN / WN, WAVES_M = BM / WM;
  static constexpr int WAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int MI = WM / 16, NJ = WN / 16;
  static constexpr int BK = 32, NS = NS_;  // BK in 16-bit units (64-byte rows)
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS = NS * STAGE;
  static_assert(sizeof(T) == 2 || sizeof(T) == 4, "bf16 or fp32 operands");
};

// 256 x 256 tiles, eight waves of 128 x 64, a 4-stage ring (128 KB): 3 and 5 stages measured
// slower for the decoder and expert GEMMs.
typedef CfgD<bf16, 256, 256, 128, 64, 4> CfgDma;
// The last row tile of a group with at most 128 rows (the short buckets of skewed routing) runs
// at half height: 128 x 256, eight waves of 64 x 64, a 5-stage ring (120 KB, inside the
// 256 x 256 tile's allocation), with half the MFMA work of the padded 256-row tile.  Such a
// tile streams a whole weight panel for few rows: with one row per bucket, 1024 tiles read
// their 1.07 GB of panels at ~4 TB/s whether the ring runs 4, 5 or 6 stages.
typedef CfgD<bf16, 128, 256, 64, 64, 5> CfgDmaShort;
template <class C>
struct ShortTile {
  using type = void;
};
template <>
struct ShortTile<CfgDma> {
  using type = CfgDmaShort;
};
typedef CfgD<float, 256, 256, 128, 64, 4> CfgDmaF32;        // fp32, K-contiguous operands
// fp32 with at most 64 columns (the gater's assignment, K <= 64): 128 x 64 tiles of four waves
// and a 3-stage ring (36 KB), four workgroups per CU -- measured against 256 x 64 (4 stages:
// 11% slower; 3 stages: 15%), 128 x 64 with 2 or 4 stages (10%, 8%) and 64 x 64 (17%)
typedef CfgD<float, 128, 64, 32, 64, 3> CfgDmaF32Narrow;
typedef CfgD<bf16, 128, 64, 32, 64, 3> CfgDmaNarrow;

// 16-byte chunk swizzle of the 64-byte K-contiguous rows (used by the DMA slot mapping and the
// operand reads alike).  Measured with the LDS bank-conflict counter on gfx950 for the MFMA
// operand read (16 rows x 4 chunks per ds_read_b128): (r >> 1) & 3 is conflict-free, while no
// swizzle, r & 3, (r >> 2) & 3, (r ^ (r >> 2)) & 3 and (r >> 3) & 3 are all 2-way conflicted.
__device__ __forceinline__ int kc_swz(int row) { return (row >> 1) & 3; }
__device__ __forceinline__ int kc_off(int row, int chunk) { return row * 64 + ((chunk ^ kc_swz(row)) << 4); }
template <int R>
__device__ __forceinline__ int ks_off(int k, int byte) {
  const int sw = ((k & 3) | ((k >> 1) & 4)) << 1;
  return k * (R * 2) + ((((byte >> 4) ^ sw)) << 4) + (byte & 15);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }
__device__ __forceinline__ void wg_barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// One operand of R rows: per-thread slot offsets and the per-stage DMA / tail staging.
template <int R, int THREADS, bool KC>
struct DmaOperand {
  static constexpr int SLOTS = KC ? R * 4 : 32 * (R / 8);  // 16-byte slots per stage
  static constexpr int NQ = SLOTS / THREADS;
  static_assert(SLOTS % THREADS == 0, "slots/threads");
  int64_t off[NQ];   // element offset of the slot's source for k0 = 0
  bool live[NQ];     // KC: chunk K-position tracking is per stage; KS: column valid
  int kk[NQ];        // KC: K offset of the chunk (0..31); KS: K-row within the stage

  // KC: element (r, k) at base + r * ld + k.  KS: element (r, k) at base + k * ld + r.
  __device__ __forceinline__ void init(int64_t ld, int rows_valid) {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int slot = (q * (THREADS / 64) + w) * 64 + l;
      if constexpr (KC) {
        const int r = slot >> 2, p = slot & 3;
        const int c = p ^ kc_swz(r);
        const int gr = r < rows_valid ? r : rows_valid - 1;
        off[q] = (int64_t)gr * ld + c * 8;
        kk[q] = c * 8;
        live[q] = r < rows_valid;
      } else {
        constexpr int CPR = R / 8;  // chunks per K-row
        const int k = slot / CPR, p = slot % CPR;
        const int sw = ((k & 3) | ((k >> 1) & 4)) << 1;
        const int col = (p ^ sw) * 8;
        live[q] = col < rows_valid;
        off[q] = (int64_t)k * ld + (live[q] ? col : 0);
        kk[q] = k;
      }
    }
  }

  __device__ __forceinline__ void issue(const bf16* __restrict__ base, int64_t ld, int k0, lds<char>* buf) const {
    const int w = threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int64_t o = off[q] + (KC ? (int64_t)k0 : (int64_t)k0 * ld);
      lds<char>* dst = buf + (q * (THREADS / 64) + w) * 1024;
      __builtin_amdgcn_global_load_lds((const void*)(base + o), (lds<void>*)dst, 16, 0, 0);
    }
  }

  // Last partial stage [k0, k_len): through registers, zero outside the valid range.
  __device__ __forceinline__ void tail(const bf16* __restrict__ base, int64_t ld, int k0, int k_len,
                                       lds<char>* buf) const {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int slot = (q * (THREADS / 64) + w) * 64 + l;
      i32x4 v = i32x4{0, 0, 0, 0};
      const bool ok = KC ? (k0 + kk[q] < k_len) : (live[q] && k0 + kk[q] < k_len);
      if (ok) v = *reinterpret_cast<const i32x4*>(base + off[q] + (KC ? (int64_t)k0 : (int64_t)k0 * ld));
      *reinterpret_cast<lds<i32x4>*>(buf + slot * 16) = v;
    }
  }
};

template <bool KC, int R>
__device__ __forceinline__ bf16x8 dma_frag(const lds<char>* buf, int r0, int lr, int lg) {
  if constexpr (KC) {
    return *reinterpret_cast<const lds<bf16x8>*>(buf + kc_off(r0 + lr, lg));
  } else {
    typedef short s4 __attribute__((ext_vector_type(4)));
    const int byte = (r0 + 4 * (lr & 3)) * 2;
    const int k = 8 * lg + (lr >> 2);
    const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds<s4>*)(buf + ks_off<R>(k, byte)));
    const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds<s4>*)(buf + ks_off<R>(k + 4, byte)));
    typedef short s8 __attribute__((ext_vector_type(8)));
    const s8 v = s8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
}

// A stage's MFMA operands for this wave: fragments of its WM rows of A and WN rows of B.
template <class C, bool A_KC, bool B_KC>
__device__ __forceinline__ void dma_read_frags(const lds<char>* bA, const lds<char>* bB, bf16x8 (&a)[C::MI],
                                               bf16x8 (&b)[C::NJ]) {
  const int l = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w / C::WAVES_N, wn = w % C::WAVES_N;
  const int lr = l & 15, lg = l >> 4;
#pragma unroll
  for (int i = 0; i < C::MI; ++i) a[i] = dma_frag<A_KC, C::BM>(bA, wm * C::WM + 16 * i, lr, lg);
#pragma unroll
  for (int j = 0; j < C::NJ; ++j) b[j] = dma_frag<B_KC, C::BN>(bB, wn * C::WN + 16 * j, lr, lg);
}

// The stage's MFMAs.  B is the MFMA's first operand: the 16 x 16 result is the transposed
// sub-tile, so each lane ends up with four consecutive output columns of one row (see TRANS).
// ROWNORM: xs[i] += squares of this lane's 8 elements of A fragment i, for the fragments
// i = wn (mod WAVES_N) that this wave is responsible for (the work is spread over the waves
// that share the rows; each row's sum stays within one wave), as four packed bf16 dot products
// (the squares of bf16 values are exact in fp32).
template <class C, bool ROWNORM>
__device__ __forceinline__ void dma_mfmas(const bf16x8 (&a)[C::MI], const bf16x8 (&b)[C::NJ],
                                          floatx4 (&acc)[C::MI][C::NJ], float* xs) {
  if constexpr (C::F32) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int j = 0; j < C::NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(floatx4, b[j])[q],
                                                           __builtin_bit_cast(floatx4, a[i])[q], acc[i][j], 0, 0, 0);
    if constexpr (ROWNORM) {
      const int wn = (threadIdx.x >> 6) % C::WAVES_N;
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
        if ((i % C::WAVES_N) == wn) {
          const floatx4 v = __builtin_bit_cast(floatx4, a[i]);
#pragma unroll
          for (int e = 0; e < 4; ++e) xs[i] = fmaf(v[e], v[e], xs[i]);
        }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  if constexpr (ROWNORM) {
    const int wn = (threadIdx.x >> 6) % C::WAVES_N;
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
      if ((i % C::WAVES_N) == wn) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 v = {a[i][2 * e], a[i][2 * e + 1]};
          xs[i] = __builtin_amdgcn_fdot2_f32_bf16(v, v, xs[i], false);
        }
      }
  }
}

template <class C, bool A_KC, bool B_KC, bool ROWNORM = false>
__device__ __forceinline__ void dma_mfma_stage(const lds<char>* bA, const lds<char>* bB,
                                               floatx4 (&acc)[C::MI][C::NJ], float* xs = nullptr) {
  bf16x8 a[C::MI], b[C::NJ];
  dma_read_frags<C, A_KC, B_KC>(bA, bB, a, b);
  // all of the stage's fragment reads go out before its MFMAs (measured faster than letting
  // the scheduler interleave them)
  __builtin_amdgcn_sched_barrier(0);
  dma_mfmas<C, ROWNORM>(a, b, acc, xs);
}

// Waits for this wave's loads of the stage that has `pending_stages` later stages in flight
// behind it, plus X more memory operations issued after those (vmcnt counts loads and stores
// alike, in issue order).
template <class C, int LOADS, int X = 0>
__device__ __forceinline__ void wait_stage(int pending_stages) {
  static_assert(C::NS <= 5 && LOADS * (C::NS - 2) + X <= 63, "vmcnt range");
  switch (pending_stages) {
    case 0: wait_vmcnt<X>(); break;
    case 1: wait_vmcnt<LOADS + X>(); break;
    case 2: wait_vmcnt<2 * LOADS + X>(); break;
    default: wait_vmcnt<3 * LOADS + X>(); break;
  }
}

// The K loop of one tile, split in two so that a persistent kernel can start the next tile's
// loads before it runs the current tile's epilogue:
//   prime()  issues stages 0 .. NS-2 of a tile into the LDS ring (the ring must be free: after
//            run()'s closing barrier, or at kernel start);
//   run()    the main loop over the primed tile and a partial last stage; it ends with a barrier
//            after which the ring is free again.  run<.., X>(.., after_prime) is for a caller
//            that issued exactly X further memory operations (per wave) between prime() and
//            run() when after_prime is true: the waits for the primed stages let those X stay
//            in flight instead of draining them first.
// A_SW > 0: A is K-contiguous and stored slab-major -- K split into slabs of A_SW columns,
// slab s of every row at A + s a_sstride (a_sstride = rows x A_SW), lda = A_SW within a slab
// -- so each stage's loads start from the base of the slab that holds it (A_SW is a multiple
// of BK, so no stage straddles two slabs).  Set the stride with slab_a() before prime().
template <class C, bool A_KC, bool B_KC, int A_SW = 0>
struct DmaTile {
  using OA = DmaOperand<C::BM, C::THREADS, A_KC>;
  using OB = DmaOperand<C::BN, C::THREADS, B_KC>;
  static constexpr int LOADS = OA::NQ + OB::NQ;
  static constexpr bool SLAB_A = A_SW > 0;
  static_assert(!SLAB_A || (A_KC && A_SW % C::BK == 0), "slab-major A: K-contiguous, whole stages per slab");
  OA oa;
  OB ob;
  const bf16* A;
  const bf16* B;
  int64_t lda, ldb;
  int k_len;
  int64_t a_sstride = 0;

  __device__ __forceinline__ void slab_a(int64_t stride) { a_sstride = stride; }
  __device__ __forceinline__ void issue_a(int k0, lds<char>* buf) const {
    if constexpr (SLAB_A) {
      const int sl = k0 / A_SW;
      oa.issue(A + sl * a_sstride, lda, k0 - sl * A_SW, buf);
    } else {
      oa.issue(A, lda, k0, buf);
    }
  }
  __device__ __forceinline__ void tail_a(int k0, lds<char>* buf) const {
    if constexpr (SLAB_A) {
      const int sl = k0 / A_SW;
      oa.tail(A + sl * a_sstride, lda, k0 - sl * A_SW, k_len - sl * A_SW, buf);
    } else {
      oa.tail(A, lda, k0, k_len, buf);
    }
  }

  __device__ __forceinline__ static lds<char>* bufA(lds<char>* smem, int s) { return smem + s * C::STAGE; }
  __device__ __forceinline__ static lds<char>* bufB(lds<char>* smem, int s) {
    return smem + s * C::STAGE + C::A_BYTES;
  }

  __device__ __forceinline__ void prime(const bf16* __restrict__ A_, int64_t lda_, int a_rows,
                                        const bf16* __restrict__ B_, int64_t ldb_, int b_rows, int k_len_,
                                        lds<char>* smem) {
    A = A_;
    B = B_;
    lda = lda_;
    ldb = ldb_;
    k_len = k_len_;
    oa.init(lda, a_rows);
    ob.init(ldb, b_rows);
    const int nfull = k_len / C::BK;
#pragma unroll
    for (int s = 0; s < C::NS - 1; ++s)
      if (s < nfull) {
        issue_a(s * C::BK, bufA(smem, s));
        ob.issue(B, ldb, s * C::BK, bufB(smem, s));
      }
  }

  template <bool ROWNORM = false, int X = 0>
  __device__ __forceinline__ void run(lds<char>* smem, floatx4 (&acc)[C::MI][C::NJ], float* xs = nullptr,
                                      bool after_prime = false) {
    static_assert(!ROWNORM || A_KC, "row norms need a K-contiguous A");
    if constexpr (ROWNORM) {
#pragma unroll
      for (int i = 0; i < C::MI; ++i) xs[i] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NJ; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int nfull = k_len / C::BK;
    // Ping-pong schedule for contractions with at least one K-contiguous operand.  With both
    // operands K-strided (two ds_read_b64_tr_b16 per fragment) the read phase outlasts the
    // MFMA phase and the single-group schedule below measured faster (dD, weight gradients).
    constexpr bool PP = A_KC || B_KC;
    auto wait_own = [&](int k) {  // this wave's loads of stage k
      const int ahead = nfull - 1 - k;
      const int pend = ahead < C::NS - 2 ? ahead : C::NS - 2;
      if (X > 0 && after_prime && k < C::NS - 1)
        wait_stage<C, LOADS, X>(pend);  // stage k was primed: the caller's X operations are younger
      else
        wait_stage<C, LOADS>(pend);
    };
    if constexpr (PP) {
      // Two wave groups (waves 0 .. WAVES/2-1 and the rest; each SIMD holds one wave of each)
      // run the same stage sequence  [barrier] read fragments + issue loads [barrier] MFMAs
      // with group 1 one phase behind group 0, so that while one group reads, the other feeds
      // the SIMD's matrix unit.  The offset comes from one extra barrier, taken by group 1
      // before the loop and by group 0 after it (the group index is wave-uniform, so those are
      // scalar branches and both groups execute the same number of barriers).  Stage kt is
      // read first by group 0, after barrier 2 kt + 1, which for group 1 is the second barrier
      // of its stage kt - 1 (or the extra one): each wave waits for its own loads of stage kt
      // before that barrier; the count of its younger loads is the same in both places.  The
      // slot of stage kt - 1 gets new loads only after barrier 2 kt + 1, when both groups'
      // reads of it have completed (lgkmcnt(0) before every second barrier).
      static_assert(C::WAVES % 2 == 0, "two wave groups");
      const bool g1 = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) >= C::WAVES / 2;
      if (nfull > 0 && g1) {
        wait_own(0);
        wg_barrier();
      }
      for (int kt = 0; kt < nfull; ++kt) {
        if (!g1) wait_own(kt);
        wg_barrier();
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 fa[C::MI], fb[C::NJ];
        const int sc = kt % C::NS;
        dma_read_frags<C, A_KC, B_KC>(bufA(smem, sc), bufB(smem, sc), fa, fb);
        const int nx = kt + C::NS - 1;
        if (nx < nfull) {
          issue_a(nx * C::BK, bufA(smem, nx % C::NS));
          ob.issue(B, ldb, nx * C::BK, bufB(smem, nx % C::NS));
        }
        if (g1 && kt + 1 < nfull) wait_own(kt + 1);
        wg_barrier_lds();
        __builtin_amdgcn_sched_barrier(0);
        dma_mfmas<C, ROWNORM>(fa, fb, acc, xs);
      }
      if (nfull > 0 && !g1) wg_barrier();
    } else {
      for (int kt = 0; kt < nfull; ++kt) {
        wait_own(kt);
        wg_barrier();
        const int nx = kt + C::NS - 1;
        if (nx < nfull) {
          const int sb = nx % C::NS;
          issue_a(nx * C::BK, bufA(smem, sb));
          ob.issue(B, ldb, nx * C::BK, bufB(smem, sb));
        }
        const int sc = kt % C::NS;
        dma_mfma_stage<C, A_KC, B_KC, ROWNORM>(bufA(smem, sc), bufB(smem, sc), acc, xs);
      }
    }
    if (nfull * C::BK < k_len) {
      const int sb = nfull % C::NS;
      tail_a(nfull * C::BK, bufA(smem, sb));
      ob.tail(B, ldb, nfull * C::BK, k_len, bufB(smem, sb));
      wg_barrier_lds();
      dma_mfma_stage<C, A_KC, B_KC, ROWNORM>(bufA(smem, sb), bufB(smem, sb), acc, xs);
    }
    wg_barrier_lds();
  }
};

template <class C, bool A_KC, bool B_KC, bool ROWNORM = false>
__device__ __forceinline__ void gemm_tile_dma(const bf16* __restrict__ A, int64_t lda, int a_rows,
                                              const bf16* __restrict__ B, int64_t ldb, int b_rows, int k_len,
                                              lds<char>* smem, floatx4 (&acc)[C::MI][C::NJ],
                                              float* xs = nullptr) {
  DmaTile<C, A_KC, B_KC> t;
  t.prime(A, lda, a_rows, B, ldb, b_rows, k_len, smem);
  t.template run<ROWNORM>(smem, acc, xs);
}

// Whether C is a direct-to-LDS configuration with fp32 operands.
template <class C>
__device__ __host__ constexpr bool dma_f32() {
  if constexpr (C::DMA)
    return C::F32;
  else
    return false;
}

// Full K loop for one tile on whichever engine the configuration names.
template <class C, bool A_KC, bool B_KC, bool ROWNORM = false>
__device__ __forceinline__ void gemm_tile(const typename C::type* __restrict__ A, int64_t lda, int a_rows,
                                          const typename C::type* __restrict__ B, int64_t ldb, int b_rows,
                                          int k_len, lds<char>* smem, floatx4 (&acc)[C::MI][C::NJ],
                                          float* xs = nullptr) {
  if constexpr (dma_f32<C>()) {
    static_assert(A_KC && B_KC, "fp32 on the direct-to-LDS engine: K-contiguous operands only");
    gemm_tile_dma<C, A_KC, B_KC, ROWNORM>(reinterpret_cast<const bf16*>(A), 2 * lda, a_rows,
                                          reinterpret_cast<const bf16*>(B), 2 * ldb, b_rows, 2 * k_len, smem, acc, xs);
  } else if constexpr (C::DMA) {
    gemm_tile_dma<C, A_KC, B_KC, ROWNORM>(A, lda, a_rows, B, ldb, b_rows, k_len, smem, acc, xs);
  } else {
    gemm_tile_reg<C, A_KC, B_KC, ROWNORM>(A, lda, a_rows, B, ldb, b_rows, k_len, smem, acc, xs);
  }
}

// ------------------------------------------------------------------ tile scheduling

// Which output tile a workgroup owns.
struct TileCoord {
  int group;      // expert id (0 for ungrouped problems)
  int64_t m0;     // first output row (global, in the row space of A / C)
  int m_rows;     // valid rows in this tile
  int n0;         // first output column
  int n_cols;     // valid columns
  int64_t k0;     // first reduction index (grouped-K problems)
  int k_len;      // reduction length
  bool valid;
};

// Plain problem: M x N tiles, bands of `band` m-tiles walked m-fastest so that concurrently
// running workgroups share both operand tiles in the caches.
template <class C>
__device__ __forceinline__ TileCoord tile_plain_at(int64_t M, int N, int K, int64_t b) {
  TileCoord tc;
  const int64_t mt = cdiv(M, C::BM);
  const int nt = (int)cdiv(N, C::BN);
  constexpr int band = 16;
  const int64_t band_tiles = (int64_t)band * nt;
  const int64_t g = b / band_tiles;
  const int64_t in = b - g * band_tiles;
  const int64_t m_first = g * band;
  const int64_t bm = (mt - m_first < band) ? (mt - m_first) : band;
  const int64_t mi = m_first + in % bm;
  const int ni = (int)(in / bm);
  tc.group = 0;
  tc.m0 = mi * C::BM;
  tc.n0 = ni * C::BN;
  tc.valid = (mi < mt) && (ni < nt);
  tc.m_rows = (int)((M - tc.m0) < C::BM ? (M - tc.m0) : C::BM);
  tc.n_cols = (N - tc.n0) < C::BN ? (N - tc.n0) : C::BN;
  tc.k0 = 0;
  tc.k_len = K;
  return tc;
}
template <class C>
__device__ __forceinline__ TileCoord tile_plain(int64_t M, int N, int K) {
  return tile_plain_at<C>(M, N, K, blockIdx.x);
}

// Row-grouped problem (experts' forward / input-gradient GEMMs): group e owns rows
// [seg[e], seg[e+1]) of A and C.  tile_start[e] = number of BM-row tiles of groups < e
// (prefix, tile_start[G] = total).  Launched over an upper bound of m-tiles x n-tiles; the
// excess workgroups find no tile and exit.
// XCD: workgroups go to the 8 XCDs round-robin (blockIdx.x % 8), each with its own L2; this
// order gives each XCD a run of 8 consecutive m-tiles with all their n-tiles (of the
// 64 nt workgroups b = 64 nt r + q: XCD x = q % 8 takes m-tile 64 r + 8 x + (q / 8) / nt,
// n-tile (q / 8) % nt), so an XCD fetches each of its A row blocks once and the B tiles of
// few groups.  The grid must then be a multiple of 64 nt (the m-tile bound rounded up to 64).
template <class C, bool XCD = false>
__device__ __forceinline__ TileCoord tile_group_m(const int32_t* __restrict__ seg,
                                                  const int32_t* __restrict__ tile_start, int G, int N,
                                                  int K) {
  TileCoord tc;
  const int nt = (int)cdiv(N, C::BN);
  const int64_t b = blockIdx.x;
  int64_t mtile;
  int ni;
  if constexpr (XCD) {
    const int64_t r = b / (64 * nt), q = b - r * 64 * nt;
    const int slot = (int)(q / 8);
    mtile = r * 64 + (q % 8) * 8 + slot / nt;
    ni = slot % nt;
  } else {
    mtile = b / nt;
    ni = (int)(b - mtile * nt);
  }
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
  tc.m0 = seg[e] + local * C::BM;
  tc.m_rows = (int)((rows - local * C::BM) < C::BM ? (rows - local * C::BM) : C::BM);
  tc.n0 = ni * C::BN;
  tc.n_cols = (N - tc.n0) < C::BN ? (N - tc.n0) : C::BN;
  tc.k0 = 0;
  tc.k_len = K;
  tc.valid = tc.m_rows > 0;
  return tc;
}

// Reduction-grouped problem (experts' weight gradients): group e reduces over the rows
// [seg[e], seg[e+1]) of both operands; output tile (m, n) of group e.  Groups are taken in the
// order `order` gives (longest reduction first), so the deepest tiles start in the first round
// instead of forming the tail of the launch.  Within a group the tiles run in bands of 16
// m-tiles, m fastest (as tile_plain_at): the tiles that share an A panel are 16 workgroups
// apart, which the round-robin placement of workgroups puts on one XCD (one L2).
template <class C>
__device__ __forceinline__ TileCoord tile_group_k(const int32_t* __restrict__ seg,
                                                  const int32_t* __restrict__ order, int G, int M, int N) {
  TileCoord tc;
  const int mt = (int)cdiv(M, C::BM), nt = (int)cdiv(N, C::BN);
  const int64_t b = blockIdx.x;
  const int per = mt * nt;
  const int slot = (int)(b / per);
  const int in = (int)(b - (int64_t)slot * per);
  constexpr int band = 16;
  const int g = in / (band * nt);
  const int inb = in - g * band * nt;
  const int m_first = g * band;
  const int bm = (mt - m_first < band) ? (mt - m_first) : band;
  const int mi = m_first + inb % bm, ni = inb / bm;
  tc.valid = slot < G;
  const int e = tc.valid ? order[slot] : 0;
  tc.group = e;
  tc.m0 = (int64_t)mi * C::BM;
  tc.m_rows = (M - mi * C::BM) < C::BM ? (M - mi * C::BM) : C::BM;
  tc.n0 = ni * C::BN;
  tc.n_cols = (N - tc.n0) < C::BN ? (N - tc.n0) : C::BN;
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

// Where accumulator element (i, j, r) of this lane sits in the tile, for either orientation.
// A lane holds MI rows x NCOL columns (TRANS: one row per i and four consecutive columns per j;
// otherwise four rows per i and one column per j); qidx(j, r) numbers the lane's columns.
template <class C>
struct Frag {
  static constexpr bool T = C::TRANS;
  static constexpr int NCOL = T ? C::NJ * 4 : C::NJ;
  int wm, wn, lr, lg;
  __device__ __forceinline__ Frag() {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    wm = w / C::WAVES_N;
    wn = w % C::WAVES_N;
    lr = l & 15;
    lg = l >> 4;
  }
  __device__ __forceinline__ int row(int i, int r) const { return wm * C::WM + 16 * i + (T ? lr : 4 * lg + r); }
  __device__ __forceinline__ int col(int j, int r) const { return wn * C::WN + 16 * j + (T ? 4 * lg + r : lr); }
  __device__ __forceinline__ static constexpr int qidx(int j, int r) { return T ? 4 * j + r : j; }
  __device__ __forceinline__ int colq(int q) const { return T ? col(q >> 2, q & 3) : col(q, 0); }
};

// Four consecutive output values of one type, as stored by store_direct.
template <typename O>
using vec4 = O __attribute__((ext_vector_type(4)));

// Epilogue store through LDS: the tile is written to LDS row-major (padded rows, conflict-free
// for the accumulator layout) in bands of rows, then copied out so that every lane stores whole
// 16-byte row segments.  Must be entered by the whole workgroup after the main loop.
//   elem(i, j, r, v)            value to store for accumulator element (i, j, r) holding v
//   rowmap(local_row)           destination row index (local_row < m_rows)
//   vec(dst_row, local_row, col, raw)  last transform of a 16-byte vector (e.g. a mask)
// n_cols must be a multiple of 16 / sizeof(O).
struct NoVec {
  template <typename V>
  __device__ __forceinline__ V operator()(int64_t, int, int, V v) const { return v; }
};

template <class C, typename O, class Elem, class RowMap, class Vec>
__device__ __forceinline__ void store_tile(const TileCoord& tc, const floatx4 (&acc)[C::MI][C::NJ],
                                           lds<char>* smem, O* __restrict__ out, int64_t ldo, Elem elem,
                                           RowMap rowmap, Vec vec) {
  constexpr int ROWB = C::BN * (int)sizeof(O) + 16;
  constexpr int FIT = C::LDS / ROWB;
  constexpr int BAND = FIT >= 256 ? 256 : (FIT >= 128 ? 128 : (FIT >= 64 ? 64 : 32));
  constexpr int VPR = C::BN * (int)sizeof(O) / 16;
  constexpr int EPV = 16 / (int)sizeof(O);
  const Frag<C> f;
#pragma unroll
  for (int b = 0; b < (C::BM + BAND - 1) / BAND; ++b) {
    if (b * BAND >= tc.m_rows) break;
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = f.row(i, r) - b * BAND;
        if (row < 0 || row >= BAND) continue;
#pragma unroll
        for (int j = 0; j < C::NJ; ++j)
          *reinterpret_cast<lds<O>*>(smem + row * ROWB + f.col(j, r) * (int)sizeof(O)) =
              from_f32<O>(elem(i, j, r, acc[i][j][r]));
      }
    __syncthreads();
    for (int q = threadIdx.x; q < BAND * VPR; q += C::THREADS) {
      const int lrow = q / VPR, v = q - lrow * VPR;
      const int row = b * BAND + lrow, col = v * EPV;
      if (row < tc.m_rows && col < tc.n_cols) {
        const int64_t dr = rowmap(row);
        i32x4 raw = *reinterpret_cast<const lds<i32x4>*>(smem + lrow * ROWB + v * 16);
        raw = vec(dr, row, col, raw);
        *reinterpret_cast<i32x4*>(out + dr * ldo + tc.n0 + col) = raw;
      }
    }
    __syncthreads();
  }
}

// Epilogue store straight from registers (TRANS orientation): no LDS, no barrier.  Same
// functors as store_tile, with vec applied to the stored vector.
//   2-byte outputs: lanes lg and lg ^ 1 (16 apart, same row) trade halves of their column
//   blocks 2p and 2p + 1 with one v_permlane16_swap per dword, after which every lane holds
//   8 consecutive columns (at 32 p + 16 (lg & 1) + 8 (lg >> 1) of the wave's columns) and
//   stores them as one 16-byte vector: each store instruction covers 64 contiguous bytes of 16
//   rows.
//   4-byte outputs: every lane stores its four consecutive columns as one 16-byte vector.
// direct_stores<C, O>() is the number of store instructions a wave issues for a full tile.
template <class C, typename O>
__device__ __forceinline__ constexpr bool direct_pairs() {
  return sizeof(O) == 2 && C::NJ % 2 == 0;
}
template <class C, typename O>
__device__ __forceinline__ constexpr int direct_stores() {
  return direct_pairs<C, O>() ? C::MI * C::NJ / 2 : C::MI * C::NJ;
}
template <class C, typename O, class Elem, class RowMap, class Vec>
__device__ __forceinline__ void store_direct(const TileCoord& tc, const floatx4 (&acc)[C::MI][C::NJ],
                                             O* __restrict__ out, int64_t ldo, Elem elem, RowMap rowmap, Vec vec) {
  static_assert(C::TRANS, "direct stores need the transposed accumulator layout");
  const Frag<C> f;
  if constexpr (direct_pairs<C, O>()) {
    typedef unsigned int u2v __attribute__((ext_vector_type(2)));
    typedef unsigned int u4v __attribute__((ext_vector_type(4)));
    typedef O v8 __attribute__((ext_vector_type(8)));
    const int cpos = 16 * (f.lg & 1) + 8 * (f.lg >> 1);
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int row = f.row(i, 0);
      const bool row_ok = row < tc.m_rows;  // the same for the two lanes of a swap
      const int64_t dr = row_ok ? rowmap(row) : 0;
#pragma unroll
      for (int p = 0; p < C::NJ / 2; ++p) {
        vec4<O> va, vb;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          va[r] = from_f32<O>(elem(i, 2 * p, r, acc[i][2 * p][r]));
          vb[r] = from_f32<O>(elem(i, 2 * p + 1, r, acc[i][2 * p + 1][r]));
        }
        const u2v a = __builtin_bit_cast(u2v, va), b = __builtin_bit_cast(u2v, vb);
        // odd 16-lane rows of the first operand trade with even rows of the second
        const u2v s0 = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
        const u2v s1 = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
        const u4v w = u4v{s0[0], s1[0], s0[1], s1[1]};
        const int col = f.wn * C::WN + 32 * p + cpos;
        if (row_ok && col < tc.n_cols)
          *reinterpret_cast<v8*>(out + dr * ldo + tc.n0 + col) = vec(dr, row, col, __builtin_bit_cast(v8, w));
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int row = f.row(i, 0);
      if (row >= tc.m_rows) continue;
      const int64_t dr = rowmap(row);
      O* orow = out + dr * ldo + tc.n0;
#pragma unroll
      for (int j = 0; j < C::NJ; ++j) {
        const int col = f.col(j, 0);
        if (col >= tc.n_cols) continue;
        vec4<O> v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = from_f32<O>(elem(i, j, r, acc[i][j][r]));
        *reinterpret_cast<vec4<O>*>(orow + col) = vec(dr, row, col, v);
      }
    }
  }
}

// Destination row of a tile row for the plain case: m0 + r.
struct RowId {
  int64_t m0;
  __device__ __forceinline__ int64_t operator()(int r) const { return m0 + r; }
};

// Tile configuration per data type: bf16 runs the 256 x 256 direct-to-LDS engine, fp32 the
// register-staged 128 x 128 one.
template <typename T>
struct Pick {
  using C = CfgSmall<float>;
};
template <>
struct Pick<bf16> {
  using C = CfgDma;
};

// The epilogue store for the configuration's orientation.
template <class C, typename O, class Elem, class RowMap, class Vec>
__device__ __forceinline__ void store_out(const TileCoord& tc, const floatx4 (&acc)[C::MI][C::NJ], lds<char>* smem,
                                          O* __restrict__ out, int64_t ldo, Elem elem, RowMap rowmap, Vec vec) {
  if constexpr (C::TRANS)
    store_direct<C, O>(tc, acc, out, ldo, elem, rowmap, vec);
  else
    store_tile<C, O>(tc, acc, smem, out, ldo, elem, rowmap, vec);
}

}  // namespace hmoe
