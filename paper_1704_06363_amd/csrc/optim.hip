// optim.hip -- the parameter update of Section 4.2: SGD with weight decay (the experts, and
// here the decoder, without momentum; the trunk with it), fused into one pass over the fp32
// master weights that also writes the weights in the compute dtype for the next forward.
// Bound by HBM: 14 bytes per parameter without momentum (w, g read; w and a bf16 copy
// written), 22 with it.
#include "launch.hpp"
#include "primitives.hpp"

namespace hmoe {

template <typename O>
using vec4o = O __attribute__((ext_vector_type(4)));

template <bool MOM>
__device__ __forceinline__ float sgd_one(float& w, float g, float& v, float lr, float wd, float mu) {
  const float gd = g + wd * w;
  if constexpr (MOM) {
    v = mu * v + gd;
    w = w - lr * v;
  } else {
    w = w - lr * gd;
  }
  return w;
}

template <typename O, bool MOM>
__global__ void __launch_bounds__(256) k_sgd(float* __restrict__ w, const float* __restrict__ g, float* __restrict__ v,
                                             O* __restrict__ wlo, int64_t count, float lr, float wd, float mu) {
  const int64_t nv = count / 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < nv; q += stride) {
    floatx4 wv = reinterpret_cast<floatx4*>(w)[q];
    const floatx4 gv = reinterpret_cast<const floatx4*>(g)[q];
    floatx4 vv = MOM ? reinterpret_cast<floatx4*>(v)[q] : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float we = wv[e], ve = vv[e];
      sgd_one<MOM>(we, gv[e], ve, lr, wd, mu);
      wv[e] = we;
      vv[e] = ve;
    }
    reinterpret_cast<floatx4*>(w)[q] = wv;
    if constexpr (MOM) reinterpret_cast<floatx4*>(v)[q] = vv;
    if (wlo) {
      vec4o<O> lo;
#pragma unroll
      for (int e = 0; e < 4; ++e) lo[e] = from_f32<O>(wv[e]);
      reinterpret_cast<vec4o<O>*>(wlo)[q] = lo;
    }
  }
  // the last count % 4 elements
  const int64_t t = nv * 4 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0 && t < count) {
    float we = w[t], ve = MOM ? v[t] : 0.f;
    sgd_one<MOM>(we, g[t], ve, lr, wd, mu);
    w[t] = we;
    if constexpr (MOM) v[t] = ve;
    if (wlo) wlo[t] = from_f32<O>(we);
  }
}

template <typename O>
static int sgd_t(float* w, const float* g, float* v, O* wlo, int64_t count, float lr, float wd, float mu,
                 hipStream_t st) {
  // one 16-byte vector per thread (a grid capped at 16 workgroups per CU looping over the
  // tensor measured 20% slower: fewer loads in flight)
  int64_t grid = cdiv(cdiv(count, 4), 256);
  if (grid < 1) grid = 1;
  if (mu > 0.f)
    HMOE_LAUNCH("sgd step", (k_sgd<O, true>), dim3((unsigned)grid), dim3(256), 0, st, w, g, v, wlo, count, lr, wd, mu);
  else
    HMOE_LAUNCH("sgd step", (k_sgd<O, false>), dim3((unsigned)grid), dim3(256), 0, st, w, g, v, wlo, count, lr, wd,
                mu);
  return HMOE_OK;
}

int launch_sgd(float* w, const float* g, float* v, void* wlo, hmoe_dtype_t dt, int64_t count, float lr, float wd,
               float mu, hipStream_t st) {
  if (count == 0) return HMOE_OK;
  if (dt == HMOE_BF16) return sgd_t<bf16>(w, g, v, (bf16*)wlo, count, lr, wd, mu, st);
  return sgd_t<float>(w, g, v, (float*)wlo, count, lr, wd, mu, st);
}

}  // namespace hmoe
