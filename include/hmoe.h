/*
 * hmoe.h -- C ABI of the hard mixture-of-experts hot path on MI355X (gfx950).
 *
 * Method: Gross, Ranzato & Szlam, "Hard Mixtures of Experts for Large Scale Weakly
 * Supervised Vision" (arXiv 1704.06363).  A K-means gater over feature vectors picks exactly
 * one expert per sample (Section 2, Eq. 2); each expert is trained on its own share of the
 * data; in the shared-decoder variant (Section 2, shared-decoder figure) every expert feeds
 * one decoder D whose outputs go through the multilabel softmax loss of Section 4.1, Eq. 3.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers unless stated otherwise; the caller owns all memory.
 *     The library allocates nothing and keeps no state between calls (the one exception is
 *     hmoe_moe_dispatch_noalloc's scratch array, below).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Every call is
 *     asynchronous on that stream and performs no host synchronisation.
 *   - Scratch memory comes from the caller through (ws, ws_bytes); the matching *_workspace()
 *     call returns the number of bytes needed (0 is a valid answer; ws may then be NULL).
 *   - Matrices are row-major.  Real tensors are HMOE_F32 (float) or HMOE_BF16 (bfloat16,
 *     round-to-nearest-even on store); accumulation is always fp32 or wider.
 *   - Row widths (d, d_hid, d_out, vocab for the decoder) must be multiples of 8 and device
 *     pointers 16-byte aligned, else HMOE_ESHAPE.  n may be 0 (nothing is launched).  A
 *     vocabulary of any size V is run by padding it to the next multiple of 8 with zero rows of
 *     D and bias -inf: a padded tag then has logit -inf, probability 0 and zero gradients, so
 *     lse, the loss and every gradient of the V real tags are those of the unpadded problem.
 *     Indices are int32 (n < 2^31); 1 <= K <= 4096.
 *   - Return value: HMOE_OK (0) or a negative code; argument errors are detected before any
 *     launch and described by hmoe_last_error() (thread-local).  Launch failures return
 *     HMOE_EHIP.  Faults inside kernels surface at the caller's next synchronisation.
 */
#ifndef HMOE_H_
#define HMOE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HMOE_VERSION 2

/* Layout of the anchors of stored logits (hmoe_moe_forward): one fp32 anchor per row and per
 * HMOE_ANCHOR_COLS columns, in an array [ceil(vocab / HMOE_ANCHOR_TILE)][n][HMOE_ANCHOR_TILE /
 * HMOE_ANCHOR_COLS]; column v of row i has its anchor at
 * ((v / HMOE_ANCHOR_TILE) * n + i) * (HMOE_ANCHOR_TILE / HMOE_ANCHOR_COLS)
 *   + (v % HMOE_ANCHOR_TILE) / HMOE_ANCHOR_COLS. */
#define HMOE_ANCHOR_COLS 64
#define HMOE_ANCHOR_TILE 256

enum {
  HMOE_OK = 0,
  HMOE_EINVAL = -1,     /* NULL required pointer, negative size, K out of range */
  HMOE_EDTYPE = -2,     /* unknown dtype */
  HMOE_ESHAPE = -3,     /* width not a multiple of 8, misaligned pointer */
  HMOE_EWORKSPACE = -4, /* ws_bytes smaller than the *_workspace() answer */
  HMOE_EHIP = -5,       /* a HIP launch or runtime call failed */
  HMOE_ENUMERIC = -6    /* a host-side factorisation did not converge (hmoe_pca_fit) */
};

typedef enum { HMOE_F32 = 0, HMOE_BF16 = 1 } hmoe_dtype_t;

/* Message for the last error on this thread ("" if none). */
const char* hmoe_last_error(void);
/* HMOE_VERSION of the library. */
int hmoe_version(void);

/* ------------------------------------------------------------------ gater (K-means) */

/* Nearest-centroid assignment, Section 2, Eq. 2: assign[i] = argmin_k |X_i - C_k|^2 with
 * ties going to the lowest k; min_dist[i] (optional) = that squared distance.
 *   X [n x d] and C [K x d] in dtype dt (a bf16 gater multiplies bf16 centres).
 *   The distance is computed as |c|^2 - 2 x.c + |x|^2 with fp32 accumulation (MFMA).
 *   assign: int32[n] out.  min_dist: float[n] out or NULL. */
size_t hmoe_kmeans_assign_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt);
int hmoe_kmeans_assign(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const void* C,
                       int32_t K, int32_t* assign, float* min_dist, void* ws, size_t ws_bytes,
                       void* stream);

/* Lloyd's K-means on the gater features (Section 2; K = 50 centres in Section 4.2) for a
 * fixed number of iterations: for t < n_iter: assign against C_t, J_t = sum of min
 * distances, C_{t+1} = mean of each cluster (empty clusters reseeded when reseed_empty:
 * in ascending id order each takes the farthest remaining sample whose cluster has more
 * than one member; an empty cluster that finds none keeps its centre); then a final assign
 * against C_T and J_T.
 *   init_uniforms: device double[K] in [0,1) -> k-means++ seeding (first centre row
 *     floor(u0*n), then the first row whose running sum of D^2 exceeds u_t * total);
 *     NULL -> C already holds the initial centres.
 *   C: float[K x d] in/out (fp32 master copy; a bf16 fit assigns against bf16(C)).
 *   assign: int32[n] out (final assignment).  min_dist: float[n] out or NULL.
 *   counts: int32[K] out or NULL.  objective: double[n_iter+1] out or NULL.
 *   init_idx: int32[K] out or NULL (k-means++ picks).  K <= n is required. */
size_t hmoe_kmeans_fit_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt);
int hmoe_kmeans_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K,
                    int32_t n_iter, const double* init_uniforms, int32_t reseed_empty,
                    float* C, int32_t* assign, float* min_dist, int32_t* counts,
                    double* objective, int32_t* init_idx, void* ws, size_t ws_bytes,
                    void* stream);

/* One Lloyd centre update (Section 2), also usable over data streamed in chunks.
 *   mode HMOE_UPDATE_FULL: zero sums/counts, accumulate this X, reseed (if reseed_empty)
 *     and write C.  HMOE_UPDATE_ACCUMULATE: add this chunk to sums/counts only.
 *     HMOE_UPDATE_FINALIZE: write C = sums / counts (X, assign unused; no reseeding).
 *   assign: int32[n] (in; rewritten for reseeded rows).  min_dist: float[n], required when
 *     reseeding (the "farthest" key).  sums: double[K x d] accumulator.  counts:
 *     int64[K] accumulator.  C: float[K x d] in (kept for clusters left empty) / out. */
enum { HMOE_UPDATE_FULL = 0, HMOE_UPDATE_ACCUMULATE = 1, HMOE_UPDATE_FINALIZE = 2 };
size_t hmoe_kmeans_update_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt);
int hmoe_kmeans_update(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K,
                       int32_t* assign, const float* min_dist, double* sums, int64_t* counts,
                       float* C, int32_t mode, int32_t reseed_empty, void* ws,
                       size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------ hard routing */

/* Hard partition of a batch by expert (Section 2: each expert sees its own share of the
 * data, no balancing): a stable counting sort.
 *   expert: int32[n], 0 <= e < K.  The ids live in device memory, which the library does not
 *     read back: out-of-range ids are the caller's error, and their rows are placed after
 *     every expert's (offsets[K] stops before them, counts exclude them, so the counts do not
 *     sum to n), perm and inv remaining permutations of all n rows.
 *   counts int32[K], offsets int32[K+1] (exclusive scan), perm int32[n] (slot -> sample),
 *   inv int32[n] (sample -> slot).
 *   rows [n x w] (dtype dt) and rows_sorted [n x w]: optional; when rows is non-NULL,
 *   rows_sorted[p] = rows[perm[p]].  w must be a multiple of 8. */
size_t hmoe_moe_dispatch_workspace(int64_t n, int32_t K);
int hmoe_moe_dispatch(const int32_t* expert, int64_t n, int32_t K, int32_t* counts,
                      int32_t* offsets, int32_t* perm, int32_t* inv, const void* rows,
                      void* rows_sorted, hmoe_dtype_t dt, int32_t w, void* ws,
                      size_t ws_bytes, void* stream);

/* Allocation-free variant of hmoe_moe_dispatch, for callers that cannot allocate device memory
 * or pass a workspace: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The same stable counting sort and row gather, with the same arguments minus the
 * workspace; its scratch (the per-block bucket counts, (K + 1) * ceil(n / 1024) int32) lives in
 * a device array of HMOE_DISPATCH_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends (looked up on the first call on that GPU).  The call allocates
 * nothing.  Every call on a GPU shares that GPU's array, which keeps the last call's contents;
 * nothing in it needs clearing (each call writes what it reads), but calls that overlap on one
 * GPU (on other streams or threads) race on it -- calls on one stream are ordered.  A size whose
 * scratch exceeds the array (e.g. K = 4096 with more than 2^20 rows) returns HMOE_EWORKSPACE
 * before anything is launched. */
#define HMOE_DISPATCH_SCRATCH_BYTES (16u << 20)
int hmoe_moe_dispatch_noalloc(const int32_t* expert, int64_t n, int32_t K, int32_t* counts,
                              int32_t* offsets, int32_t* perm, int32_t* inv, const void* rows,
                              void* rows_sorted, hmoe_dtype_t dt, int32_t w, void* stream);

/* Row gather out[r] = in[index[r]] for r < n (rows of w elements of dtype dt; in has n rows
 * too).  With index = inv it combines expert-ordered rows back to sample order; with perm it
 * dispatches.  An index outside [0, n) gives a row of zeros.  in and out must not overlap. */
int hmoe_permute_rows(const void* in, void* out, const int32_t* index, int64_t n, int32_t w,
                      hmoe_dtype_t dt, void* stream);

/* ------------------------------------------------------------------ experts + decoder */

/* Parameters of K expert MLPs and their decoder(s) (Section 2).
 *   W1 [K][d_hid][d_in], b1 [K][d_hid], W2 [K][d_out][d_hid], b2 [K][d_out]; all in dtype dt;
 *   biases may be NULL (no bias).
 *   decoders = 1 (or 0): one decoder shared by all experts (the shared-decoder figure),
 *     D [vocab][d_out], bD [vocab].
 *   decoders = K: every expert has its own decoder (the independent-decoder figure), and a
 *     sample is decoded by its expert's: D [K][vocab][d_out], bD [K][vocab].  The forward then
 *     stores its logits in expert (slot) order, and the backward needs them (logits != NULL)
 *     and writes dD [K][vocab][d_out], dbD [K][vocab]. */
typedef struct {
  int32_t K, d_in, d_hid, d_out, vocab;
  hmoe_dtype_t dt;
  const void *W1, *b1, *W2, *b2, *D, *bD;
  int32_t decoders;
} hmoe_moe_params_t;

/* Multilabel targets as CSR: sample i has the distinct positive tags
 * tag[row_ptr[i] .. row_ptr[i+1]) (at least one); the target puts mass 1/|P_i| on each
 * (Section 4.1, Eq. 3, with the indicator spread uniformly over the positives). */
typedef struct {
  const int32_t* row_ptr; /* int32[n+1] */
  const int32_t* tag;     /* int32[nnz], 0 <= tag < vocab.  The labels live in device memory,
                           * which the library does not read back to validate: a tag outside
                           * [0, vocab) is never dereferenced, contributes a logit of 0 to the
                           * loss and matches no column of the gradient (the result is then
                           * not Eq. 3's). */
} hmoe_labels_t;

/* Forward pass of the hard mixture with the loss of Eq. 3.
 *   X_sorted [n x d_in]: samples in expert order (from hmoe_moe_dispatch), offsets int32[K+1],
 *   perm int32[n] (slot -> sample).
 *   H1_sorted [n x d_hid] out: relu(W1_e x + b1_e) in expert order (saved for backward).
 *   H [n x d_out] out: expert outputs W2_e h1 + b2_e in SAMPLE order (the combine).
 *   logits [n x vocab] out or NULL: the logits D H_i + bD, saved so that the backward does
 *     not recompute them (n * vocab * 2 bytes in bf16; pass NULL to save the memory), stored
 *     in dtype dt as offsets from per-row anchors: logit = anchor + stored value, the sum
 *     formed in fp32.  The anchor of a row and 64-column block is the largest fp32 logit of
 *     the row in that block, so the largest logits (the ones that carry the probability mass)
 *     keep close to fp32 accuracy in a bf16 store, whatever their magnitude.  Rows in sample
 *     order with a shared decoder; in slot order (row p is sample perm[p]) with per-expert
 *     decoders, where they are required by the backward.
 *   logit_anchor float[ceil(vocab / 256) * n * 4] out (layout: HMOE_ANCHOR_*): required when
 *     logits is given, ignored otherwise.
 *   lse float[n] out: log-sum-exp of the V logits (from the fp32 logits).
 *   loss float[n] out: lse_i - mean of the logits of the positive tags.
 *   loss_mean float[1] out: mean over the batch. */
size_t hmoe_moe_workspace(const hmoe_moe_params_t* p, int64_t n);
int hmoe_moe_forward(const hmoe_moe_params_t* p, int64_t n, const void* X_sorted,
                     const int32_t* offsets, const int32_t* perm, const hmoe_labels_t* y,
                     void* H1_sorted, void* H, void* logits, float* logit_anchor, float* lse,
                     float* loss, float* loss_mean, void* ws, size_t ws_bytes, void* stream);

/* Backward pass: gradients of loss_mean (the 1/n is included) with respect to every expert
 * and decoder parameter, and optionally the input features.  The gater is fixed (Section
 * 2.2), so nothing flows to the centres.  With p = softmax(D H_i + bD), y_i the target:
 *   g = (p - y)/n; dbD = sum g; dD = g^T H; dH = g D; per expert e: db2 = sum dH,
 *   dW2 = dH^T H1, dZ = (dH W2) * [H1 > 0]; db1 = sum dZ; dW1 = dZ^T X; dX = dZ W1.
 *   Inputs are the forward's saved tensors (H1_sorted, H, lse, and logits with logit_anchor
 *   if it saved them: then p = exp(anchor + stored - lse); logits NULL recomputes them from H)
 *   and inv int32[n].
 *   dW1, db1, dW2, db2, dD, dbD: float out (overwritten; experts without samples get 0, and
 *   so do their decoders when each expert has its own; dD and dbD have D's and bD's shapes);
 *   db1, db2, dbD may be NULL.  dX [n x d_in] in dtype dt, SAMPLE order, or NULL. */
int hmoe_moe_backward(const hmoe_moe_params_t* p, int64_t n, const void* X_sorted,
                      const int32_t* offsets, const int32_t* perm, const int32_t* inv,
                      const hmoe_labels_t* y, const void* H1_sorted, const void* H,
                      const void* logits, const float* logit_anchor, const float* lse,
                      float* dW1, float* db1, float* dW2,
                      float* db2, float* dD, float* dbD, void* dX, void* ws, size_t ws_bytes,
                      void* stream);

/* ------------------------------------------------------------------ PCA before the K-means */

/* Section 4.2: the trunk's features are projected to their first 256 principal directions
 * before the K-means.
 * hmoe_pca_fit: mean float[d] out; components float[r][d] out -- the r leading eigenvectors of
 *   the sample covariance (1/(n-1)) sum_i (x_i - mean)(x_i - mean)^T as orthonormal rows in
 *   decreasing eigenvalue order, each row's largest-magnitude entry positive; eigvals float[r]
 *   out.  Subspace iteration: n_iter steps Q <- orth(C Q) from a start drawn from `seed`, then
 *   Rayleigh-Ritz; a component's accuracy depends on the gap between its eigenvalue and the
 *   (r+1)-th.  A covariance of rank below r (fewer independent directions, or n <= r) gives
 *   eigenvalues ~0 for the rest, with any orthonormal completion as their components.  X [n x d] in dtype dt; n >= 2, 8 <= r <= d, r and d multiples of 8.  The
 *   d x d x r work runs on the GPU and the r x r factorisations on the host (fp64), so the call
 *   synchronises `stream` (a preprocessing step; not for graph capture).  Device pointers
 *   throughout (eigvals too).
 * hmoe_pca_project: Z [n x r] (dtype dt) = (X - mean) components^T.
 * Both take the workspace hmoe_pca_workspace asks for. */
size_t hmoe_pca_workspace(int64_t n, int32_t d, int32_t r, hmoe_dtype_t dt);
int hmoe_pca_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t r, int32_t n_iter, uint64_t seed,
                 float* mean, float* components, float* eigvals, void* ws, size_t ws_bytes, void* stream);
int hmoe_pca_project(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const float* mean,
                     const float* components, int32_t r, void* Z, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------ parameter update */

/* One SGD step (Section 4.2: weight decay; the experts -- and the decoder trained with them --
 * without momentum, the trunk with momentum).  For each of count elements:
 *   g' = g + weight_decay * w;  momentum > 0: v = momentum * v + g', w = w - lr * v;
 *   otherwise w = w - lr * g'   (fp32 arithmetic).
 * w float[count] in/out: the fp32 master weights; g float[count]: the gradient (as written by
 * hmoe_moe_backward); v float[count] in/out, the momentum buffer, or NULL when momentum == 0;
 * w_lo [count] out in dtype dt (the updated weights rounded to nearest even, for the next
 * forward) or NULL.  Device pointers, 16-byte aligned; w_lo must not overlap w.  One fused
 * pass, bound by HBM.  Errors: HMOE_EINVAL (NULL w or g, negative count or hyperparameter,
 * momentum > 0 without v), HMOE_ESHAPE (misaligned pointer), HMOE_EDTYPE. */
int hmoe_sgd_step(float* w, const float* g, float* v, void* w_lo, hmoe_dtype_t dt, int64_t count, float lr,
                  float weight_decay, float momentum, void* stream);

/* ------------------------------------------------------------------ inference tail */

/* t_m (Section 4.4): for every row of logits [n x vocab] (dtype dt; the softmax keeps the
 * order, so these are the m most probable tags), the indices of its m largest entries in
 * decreasing order, equal values in increasing index order.  With anchor (float, the layout of
 * HMOE_ANCHOR_*, as written by hmoe_moe_forward) an entry is anchor + stored value, formed in
 * fp32, and every stored value must be <= 0 (each anchor at least every entry of its
 * HMOE_ANCHOR_COLS-column block, as hmoe_moe_forward writes them): the kernel then reads the
 * anchors and only the blocks whose anchor can reach the row's m-th entry.  With anchor NULL an
 * entry is the stored value and each row is read once.  idx int32[n][m] out; val float[n][m]
 * out or NULL (the entries at those indices).  1 <= m <= 16, m <= vocab; the entries are
 * assumed finite or -inf.  One wave per row.  Errors: HMOE_EINVAL (m out of range, NULL
 * logits or idx), HMOE_ESHAPE (vocab not a multiple of 8). */
int hmoe_topm(const void* logits, const float* anchor, hmoe_dtype_t dt, int64_t n, int32_t vocab,
              int32_t m, int32_t* idx, float* val, void* stream);

/* The counts behind p@m (Eq. 4) and q@m (Eq. 5), Section 4.4, for every m' = 1..m, from the
 * top-m lists idx int32[n][m] (hmoe_topm):
 *   hits[m' - 1]     = sum_i |t_m'(i) ∩ P_i|, so p@m' = hits[m' - 1] / (number of positives);
 *   hits[m + m' - 1] = number of the S draws (q_sample[s], q_tag[s]) whose tag is in
 *                      t_m'(q_sample[s]), so q@m' = hits[m + m' - 1] / S.
 * The draws (a tag uniformly from the dictionary, then a sample carrying it) are the caller's;
 * a draw whose sample is outside [0, n) counts as a miss.  hits int64[2m] out (device);
 * q_sample, q_tag int32[S] (device, NULL when S = 0).  1 <= m <= 16. */
int hmoe_topm_hits(const int32_t* idx, int64_t n, int32_t m, const hmoe_labels_t* y, const int32_t* q_sample,
                   const int32_t* q_tag, int64_t S, int64_t* hits, void* stream);

/* ------------------------------------------------------------------ diagnostics */

/* Launch timing for benchmarks, not part of the hot path.  While enabled, every kernel the
 * library launches is bracketed by a pair of HIP events on its stream (the pool of events
 * grows as needed and is kept for the life of the process).  hmoe_timer_enable(1) starts a
 * new recording, (0) stops it.  hmoe_timer_report() waits for the recorded events and writes
 * one line per kernel label, "label<TAB>launches<TAB>total_ms", into buf (host memory,
 * truncated to buf_bytes - 1 characters and NUL-terminated); it returns the full length of
 * the report or a negative error code.  Not thread-safe. */
int hmoe_timer_enable(int on);
int64_t hmoe_timer_report(char* buf, size_t buf_bytes);

#ifdef __cplusplus
}
#endif

#endif /* HMOE_H_ */
