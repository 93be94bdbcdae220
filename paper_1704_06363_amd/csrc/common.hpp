// common.hpp -- device-side types and small helpers shared by the HIP kernels (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "hmoe.h"

namespace hmoe {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Types in LDS (address space 3).  Pointers into shared memory are kept in this address
// space explicitly so that every access compiles to ds_read / ds_write (generic pointers
// would become flat instructions that also wait on outstanding global loads).
template <typename T>
using lds = __attribute__((address_space(3))) T;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // round to nearest even

// Lane-crossing helpers over the 64-wide wavefront.
__device__ __forceinline__ float shfl_xor(float v, int m) { return __shfl_xor(v, m, kWave); }
__device__ __forceinline__ int shfl_xor(int v, int m) { return __shfl_xor(v, m, kWave); }
__device__ __forceinline__ double shfl_xor(double v, int m) { return __shfl_xor(v, m, kWave); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, shfl_xor(v, m));
  return v;
}

// (value, index) minimum with ties to the lower index.
__device__ __forceinline__ void argmin_merge(float& v, int& i, float v2, int i2) {
  if (v2 < v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

__host__ __device__ __forceinline__ int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Stored decoder logits are offsets from a per-row anchor, one per 64 columns (the row maximum
// over those columns): logit[row][v] = anc[v / 256][row][(v % 256) / 64] + stored[row][v].
constexpr int kAnchorCols = HMOE_ANCHOR_COLS;
constexpr int kAnchorTile = HMOE_ANCHOR_TILE;
constexpr int kAnchorSlots = kAnchorTile / kAnchorCols;
__host__ __device__ __forceinline__ int64_t anchor_index(int64_t n, int64_t row, int64_t col) {
  return ((col / kAnchorTile) * n + row) * kAnchorSlots + (col % kAnchorTile) / kAnchorCols;
}
__host__ __forceinline__ int64_t anchor_count(int64_t n, int64_t vocab) {
  return cdiv(vocab, kAnchorTile) * n * kAnchorSlots;
}

template <typename T>
struct DT;
template <>
struct DT<float> {
  static constexpr hmoe_dtype_t id = HMOE_F32;
};
template <>
struct DT<bf16> {
  static constexpr hmoe_dtype_t id = HMOE_BF16;
};

}  // namespace hmoe
