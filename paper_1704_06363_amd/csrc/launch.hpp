// launch.hpp -- launchers implemented in the .hip translation units and called by api.cpp.
// All of them only enqueue work on `st`; sizes have been validated by the caller.
#pragma once
#include "host.hpp"

namespace hmoe {

typedef __bf16 bf16;

// dispatch.hip
size_t dispatch_ws(int64_t n, int32_t K);
int launch_dispatch(const int32_t* e, int64_t n, int32_t K, int32_t* counts, int32_t* offsets,
                    int32_t* perm, int32_t* inv, Workspace& ws, hipStream_t st);
int launch_permute(const void* in, void* out, const int32_t* index, int64_t n, int32_t w,
                   hmoe_dtype_t dt, hipStream_t st);
int launch_seg_tiles(const int32_t* seg, int G, int tile, int32_t* tile_start, hipStream_t st);
int launch_seg_order(const int32_t* seg, int G, int32_t* order, hipStream_t st);
template <typename T>
size_t gemm_tn_ws();
template <typename T>
int launch_gemm_tn(const T* A, const T* B, int64_t rows, int M, int N, float* out, Workspace& ws, hipStream_t st,
                   const char* label = "gemm tn");
template <typename T>
int launch_gemm_nn(const T* A, const T* W, int64_t rows, int Kd, int N, T* out, Workspace& ws, hipStream_t st);
size_t pca_fit_ws(int64_t n, int d, int r, hmoe_dtype_t dt);
size_t pca_project_ws(int d, int r, hmoe_dtype_t dt);
int launch_pca_fit(const void* X, hmoe_dtype_t dt, int64_t n, int d, int r, int n_iter, uint64_t seed, float* mean,
                   float* comps, float* eigvals, Workspace& ws, hipStream_t st);
int launch_pca_project(const void* X, hmoe_dtype_t dt, int64_t n, int d, const float* mean, const float* comps,
                       int r, void* Z, Workspace& ws, hipStream_t st);
int launch_sgd(float* w, const float* g, float* v, void* wlo, hmoe_dtype_t dt, int64_t count, float lr, float wd,
               float mu, hipStream_t st);
int launch_topm(const void* L, const float* anc, hmoe_dtype_t dt, int64_t n, int V, int m, int32_t* idx, float* val,
                hipStream_t st);
int launch_topm_hits(const int32_t* idx, int64_t n, int m, const hmoe_labels_t* y, const int32_t* q_sample,
                     const int32_t* q_tag, int64_t S, int64_t* hits, hipStream_t st);
size_t segsum_ws(int64_t n, int G, int w);
template <typename T, typename O>
int launch_segsum(const T* X, int64_t ld, const int32_t* rowmap, const int32_t* seg, int G, int w,
                  int64_t n, O* out, int accumulate, Workspace& ws, hipStream_t st);
int launch_zero_f32(float* x, int64_t n, hipStream_t st);
int launch_sum_f32(const float* x, int64_t n, double scale, double* out_f64, float* out_f32,
                   Workspace& ws, hipStream_t st);

// kmeans.hip
size_t assign_ws(int64_t n, int32_t K, hmoe_dtype_t dt);
size_t fit_ws_bytes(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt);
size_t update_ws_bytes(int64_t n, int32_t d, int32_t K);
int launch_assign(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const void* C, int32_t K,
                  int32_t* assign, float* min_dist, Workspace& ws, hipStream_t st);
int launch_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t n_iter,
               const double* u, int32_t reseed, float* C, int32_t* assign, float* min_dist,
               int32_t* counts, double* objective, int32_t* init_idx, Workspace& ws, hipStream_t st);
int launch_update(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t* assign,
                  const float* min_dist, double* sums, int64_t* counts, float* C, int32_t mode,
                  int32_t reseed, Workspace& ws, hipStream_t st);

// moe.hip
size_t moe_ws_bytes(const hmoe_moe_params_t* p, int64_t n);
int launch_moe_forward(const hmoe_moe_params_t* p, int64_t n, const void* Xs, const int32_t* offsets,
                       const int32_t* perm, const hmoe_labels_t* y, void* H1s, void* H, void* logits,
                       float* anc, float* lse, float* loss, float* loss_mean, Workspace& ws, hipStream_t st);
int launch_moe_backward(const hmoe_moe_params_t* p, int64_t n, const void* Xs, const int32_t* offsets,
                        const int32_t* perm, const int32_t* inv, const hmoe_labels_t* y,
                        const void* H1s, const void* H, const void* logits, const float* anc, const float* lse,
                        float* dW1,
                        float* db1, float* dW2, float* db2, float* dD, float* dbD, void* dX, Workspace& ws,
                        hipStream_t st);

}  // namespace hmoe
