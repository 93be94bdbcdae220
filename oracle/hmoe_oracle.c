/*
 * hmoe_oracle.c -- plain, slow, fp64 CPU oracle for the hard mixture-of-experts hot path
 * of Gross, Ranzato & Szlam, "Hard Mixtures of Experts for Large Scale Weakly Supervised
 * Vision" (arXiv 1704.06363).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or calls this file:
 * only the tests, the smoke check and the bench's CPU-baseline leg do.  It shares no code,
 * header, table or helper with the HIP library.
 *
 * Conventions
 *   - Every real number is a double.  Inputs are the exact values the device sees (fp32 or
 *     bf16 bytes widened to double by the caller).
 *   - Results are rounded to a storage precision only where the library's interface hands a
 *     tensor to its caller, who feeds it to a later step: centroids (fp32), the expert hidden
 *     activations H1 and outputs H, and the input gradient dX (the data dtype: "bf16 in, fp32
 *     accumulate, bf16 out" for every layer).  `store` selects that rounding: 0 = keep fp64,
 *     1 = fp32 (round to nearest even), 2 = bf16 (round to nearest even).  Everything else,
 *     the softmax and the activation gradients g, dh, dz included, stays in fp64.
 *   - Matrices are row-major.  Expert weights follow the [out][in] convention.
 *   - OpenMP is used only across independent samples / output rows; every sum runs in a
 *     fixed order (ascending sample index, ascending feature index), so results do not depend
 *     on the thread count.
 *
 * Parity pins (tests/test_oracle_*.py): brute force and closed forms for assignment, the
 * total-sum-of-squares case K=1 for the update, hand-worked reseeding, the n=K and
 * D^2-proportional pick frequency for k-means++, stability / inverse identities for the
 * dispatch, log V for a zero decoder, an independent autograd cross-check for K=1 experts,
 * and central finite differences for every gradient.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- rounding helpers */

/* Round a double to the nearest bf16 value (8 significant bits), ties to even.  The
 * default floating-point environment rounds nearbyint() to nearest-even. */
static double to_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);          /* x = m * 2^e, 0.5 <= |m| < 1 */
  double s = ldexp(m, 8);           /* 8 significant bits to the left of the point */
  return ldexp(nearbyint(s), e - 8);
}

static double store_round(double x, int store) {
  if (store == 1) return (double)(float)x;
  if (store == 2) return to_bf16(x);
  return x;
}

void hmoe_orc_round(int64_t n, double* x, int store) {
  for (int64_t i = 0; i < n; ++i) x[i] = store_round(x[i], store);
}

/* ------------------------------------------------------------- O1: nearest centroid */

/* Section 2, Eq. 2: the gater sends x to the centroid at minimum Euclidean distance.
 * The squared distance is formed from direct differences (no norm expansion); ties go to the
 * lowest centroid index.  d2 receives the second-smallest distance (+inf when K = 1) so that
 * callers can recognise near-ties. */
int hmoe_orc_assign(int64_t n, int32_t d, int32_t K, const double* X, const double* C,
                    int32_t* a, double* d1, double* d2) {
  if (n < 0 || d <= 0 || K <= 0) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const double* x = X + i * (int64_t)d;
    double best = INFINITY, second = INFINITY;
    int32_t arg = 0;
    for (int32_t k = 0; k < K; ++k) {
      const double* c = C + (int64_t)k * d;
      double s = 0.0;
      for (int32_t j = 0; j < d; ++j) {
        double t = x[j] - c[j];
        s += t * t;
      }
      if (s < best) {
        second = best;
        best = s;
        arg = k;
      } else if (s < second) {
        second = s;
      }
    }
    a[i] = arg;
    if (d1) d1[i] = best;
    if (d2) d2[i] = second;
  }
  return 0;
}

/* ----------------------------------------------------------------- O6: k-means++ */

/* Seeding for the K-means step of Section 2 (the paper does not say how the centres are
 * started; this follows Arthur & Vassilvitskii's k-means++).  u[t] in [0,1) are the uniform
 * draws, supplied by the caller.  The first centre is row floor(u0*n); each later centre is
 * the first row whose running sum of D^2 (squared distance to the nearest chosen centre)
 * exceeds u_t times the total.  If every D^2 is zero the lowest unchosen row is taken. */
int hmoe_orc_kmeanspp(int64_t n, int32_t d, int32_t K, const double* X, const double* u,
                      int32_t* idx) {
  if (n <= 0 || d <= 0 || K <= 0 || K > n) return -1;
  double* D2 = (double*)malloc(sizeof(double) * (size_t)n);
  char* chosen = (char*)calloc((size_t)n, 1);
  if (!D2 || !chosen) { free(D2); free(chosen); return -2; }
  int64_t first = (int64_t)floor(u[0] * (double)n);
  if (first > n - 1) first = n - 1;
  idx[0] = (int32_t)first;
  chosen[first] = 1;
  for (int64_t i = 0; i < n; ++i) D2[i] = INFINITY;
  for (int32_t t = 0; t < K; ++t) {
    if (t > 0) {
      double S = 0.0;
      for (int64_t i = 0; i < n; ++i) S += D2[i];
      int64_t pick = -1;
      if (S > 0.0) {
        double target = u[t] * S, P = 0.0;
        for (int64_t i = 0; i < n; ++i) {
          P += D2[i];
          if (P > target) { pick = i; break; }
        }
        /* P(n-1) == S > target always holds for u < 1; the guard below is belt and braces. */
      }
      if (pick < 0) {
        for (int64_t i = 0; i < n; ++i)
          if (!chosen[i]) { pick = i; break; }
      }
      idx[t] = (int32_t)pick;
      chosen[pick] = 1;
    }
    const double* c = X + (int64_t)idx[t] * d;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
      const double* x = X + i * (int64_t)d;
      double s = 0.0;
      for (int32_t j = 0; j < d; ++j) {
        double q = x[j] - c[j];
        s += q * q;
      }
      if (s < D2[i]) D2[i] = s;
    }
  }
  free(D2);
  free(chosen);
  return 0;
}

/* ------------------------------------------------------------- O3 + O5: Lloyd update */

typedef struct { double key; int64_t i; } cand_t;

static int cand_cmp(const void* pa, const void* pb) {
  const cand_t* A = (const cand_t*)pa;
  const cand_t* B = (const cand_t*)pb;
  if (A->key > B->key) return -1; /* larger distance first */
  if (A->key < B->key) return 1;
  return (A->i < B->i) ? -1 : (A->i > B->i); /* then lower sample index */
}

/* One Lloyd update for the K-means step of Section 2: each centre becomes the mean of the
 * rows assigned to it.  C holds the previous centres on entry and the new centres (fp64,
 * unrounded) on exit.
 *
 * Empty clusters (the paper does no balancing, Section 2, and reports every cluster in use,
 * Section 4.5): when `reseed` is set, the empty clusters, in ascending id order, each take
 * the farthest remaining row (largest d1, lower index on ties) whose current cluster has
 * more than one member; that row moves to the empty cluster, whose centre becomes the row
 * itself, and leaves its donor.  An empty cluster that finds no such row, or any empty
 * cluster when `reseed` is 0, keeps its previous centre.  `a` and `counts` are updated. */
int hmoe_orc_update(int64_t n, int32_t d, int32_t K, const double* X, int32_t* a,
                    const double* d1, int reseed, double* C, int64_t* counts) {
  if (n < 0 || d <= 0 || K <= 0) return -1;
  double* S = (double*)calloc((size_t)K * d, sizeof(double));
  if (!S) return -2;
  for (int32_t k = 0; k < K; ++k) counts[k] = 0;
  /* Sums in ascending sample order, one cluster row per thread. */
  for (int64_t i = 0; i < n; ++i) {
    if (a[i] < 0 || a[i] >= K) { free(S); return -3; }
    counts[a[i]] += 1;
  }
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t k = 0; k < K; ++k) {
    double* s = S + (int64_t)k * d;
    for (int64_t i = 0; i < n; ++i) {
      if (a[i] != k) continue;
      const double* x = X + i * (int64_t)d;
      for (int32_t j = 0; j < d; ++j) s[j] += x[j];
    }
  }
  int32_t n_empty = 0;
  for (int32_t k = 0; k < K; ++k) n_empty += (counts[k] == 0);
  if (reseed && n_empty > 0 && n > 0) {
    cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * (size_t)n);
    if (!cand) { free(S); return -2; }
    for (int64_t i = 0; i < n; ++i) { cand[i].key = d1[i]; cand[i].i = i; }
    qsort(cand, (size_t)n, sizeof(cand_t), cand_cmp);
    int64_t next = 0;
    for (int32_t k = 0; k < K; ++k) {
      if (counts[k] != 0) continue;
      while (next < n && counts[a[cand[next].i]] <= 1) ++next;
      if (next >= n) break;
      int64_t i = cand[next++].i;
      int32_t donor = a[i];
      const double* x = X + i * (int64_t)d;
      double* sd = S + (int64_t)donor * d;
      double* sk = S + (int64_t)k * d;
      for (int32_t j = 0; j < d; ++j) { sd[j] -= x[j]; sk[j] = x[j]; }
      counts[donor] -= 1;
      counts[k] = 1;
      a[i] = k;
    }
    free(cand);
  }
  for (int32_t k = 0; k < K; ++k) {
    if (counts[k] == 0) continue; /* keeps the previous centre */
    double* c = C + (int64_t)k * d;
    const double* s = S + (int64_t)k * d;
    for (int32_t j = 0; j < d; ++j) c[j] = s[j] / (double)counts[k];
  }
  free(S);
  return 0;
}

/* ------------------------------------------------------------------ O4: Lloyd fit */

/* K-means on the gater features (Section 2), run for a fixed number of Lloyd iterations:
 * for t < T: a_t = assign(C_t), J_t = sum of d1, C_{t+1} = update(a_t), stored as fp32;
 * finally a_T = assign(C_T) and J_T.  The assignment uses the centres rounded to the data
 * precision (`assign_store`: 1 fp32, 2 bf16), which is what a device that multiplies in the
 * data precision sees.  C_0 is the k-means++ seeding (u != NULL) or the given C. */
int hmoe_orc_fit(int64_t n, int32_t d, int32_t K, const double* X, int32_t n_iter,
                 const double* u, int assign_store, int reseed, double* C, int32_t* a,
                 double* J, int32_t* init_idx, int64_t* counts) {
  if (n <= 0 || d <= 0 || K <= 0 || n_iter < 0) return -1;
  int rc = 0;
  if (u) {
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    if (!idx) return -2;
    rc = hmoe_orc_kmeanspp(n, d, K, X, u, idx);
    if (rc) { free(idx); return rc; }
    for (int32_t k = 0; k < K; ++k) {
      memcpy(C + (int64_t)k * d, X + (int64_t)idx[k] * d, sizeof(double) * (size_t)d);
      if (init_idx) init_idx[k] = idx[k];
    }
    free(idx);
  }
  hmoe_orc_round((int64_t)K * d, C, 1);
  double* Cq = (double*)malloc(sizeof(double) * (size_t)K * d);
  double* d1 = (double*)malloc(sizeof(double) * (size_t)n);
  int64_t* cnt = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
  if (!Cq || !d1 || !cnt) { free(Cq); free(d1); free(cnt); return -2; }
  for (int32_t t = 0; t <= n_iter; ++t) {
    memcpy(Cq, C, sizeof(double) * (size_t)K * d);
    hmoe_orc_round((int64_t)K * d, Cq, assign_store);
    hmoe_orc_assign(n, d, K, X, Cq, a, d1, NULL);
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += d1[i];
    if (J) J[t] = s;
    if (t == n_iter) break;
    rc = hmoe_orc_update(n, d, K, X, a, d1, reseed, C, cnt);
    if (rc) break;
    hmoe_orc_round((int64_t)K * d, C, 1);
  }
  if (counts) {
    for (int32_t k = 0; k < K; ++k) counts[k] = 0;
    for (int64_t i = 0; i < n; ++i) counts[a[i]] += 1;
  }
  free(Cq);
  free(d1);
  free(cnt);
  return rc;
}

/* --------------------------------------------------------------- O7: hard dispatch */

/* Section 2: each expert trains on its own share of the data.  Rows are grouped by expert
 * with a stable order inside each group: counts, exclusive offsets, perm (slot -> sample)
 * and inv (sample -> slot). */
int hmoe_orc_dispatch(int64_t n, int32_t K, const int32_t* e, int32_t* counts,
                      int32_t* offsets, int32_t* perm, int32_t* inv) {
  if (n < 0 || K <= 0) return -1;
  for (int32_t k = 0; k < K; ++k) counts[k] = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (e[i] < 0 || e[i] >= K) return -3;
    counts[e[i]] += 1;
  }
  offsets[0] = 0;
  for (int32_t k = 0; k < K; ++k) offsets[k + 1] = offsets[k] + counts[k];
  int32_t* fill = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
  if (!fill) return -2;
  for (int32_t k = 0; k < K; ++k) fill[k] = offsets[k];
  for (int64_t i = 0; i < n; ++i) {
    int32_t p = fill[e[i]]++;
    perm[p] = (int32_t)i;
    inv[i] = p;
  }
  free(fill);
  return 0;
}

/* ------------------------------------------------- O8 + O9: experts, decoder, loss */

/* Forward pass of the hard mixture (Section 2) with the multilabel softmax loss of Section
 * 4.1, Eq. 3.  ndec = 1: one decoder shared by the experts (D [V][o], bD [V]; the
 * shared-decoder figure); ndec = K: every expert has its own (D [K][V][o], bD [K][V]; the
 * independent-decoder figure), and sample i is decoded by its expert's.  For every sample i
 * routed to expert e = a[i], with D_i, bD_i the decoder it uses:
 *   h1 = relu(W1_e x + b1_e)            (stored, rounded by `store`)
 *   y  = W2_e h1 + b2_e                 (stored as H[i], rounded by `store`)
 *   l  = D_i H[i] + bD_i                (all V logits)
 *   lse = log sum_j exp(l_j);  loss_i = lse - (1/|P_i|) sum_{j in P_i} l_j
 * The target mass is spread uniformly over the positive tags P_i (tags listed in
 * tag[row_ptr[i] .. row_ptr[i+1]), distinct); the batch loss is the mean over samples.
 * b1, b2, bD may be NULL (no bias).  probs (n x V) and logits (n x V) are optional outputs, in
 * fp64 like lse and loss. */
int hmoe_orc_moe_forward(int64_t n, int32_t d, int32_t h, int32_t o, int32_t V, int32_t K,
                         int32_t ndec, const double* X, const int32_t* a, const double* W1,
                         const double* b1, const double* W2, const double* b2, const double* D,
                         const double* bD, const int32_t* row_ptr, const int32_t* tag,
                         int store, double* H1, double* H, double* lse, double* loss,
                         double* loss_mean, double* probs, double* logits) {
  if (n < 0 || d <= 0 || h <= 0 || o <= 0 || V <= 0 || K <= 0) return -1;
  if (ndec != 1 && ndec != K) return -1;
  for (int64_t i = 0; i < n; ++i) {
    if (a[i] < 0 || a[i] >= K) return -3;
    if (row_ptr[i + 1] <= row_ptr[i]) return -4; /* every sample has a positive tag */
  }
  int bad = 0;
#pragma omp parallel
  {
    double* lg = (double*)malloc(sizeof(double) * (size_t)V);
    if (!lg) {
#pragma omp atomic write
      bad = 1;
    }
#pragma omp for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
      if (!lg) continue;
      const int32_t e = a[i];
      const double* x = X + i * (int64_t)d;
      const double* w1 = W1 + (int64_t)e * h * d;
      const double* w2 = W2 + (int64_t)e * o * h;
      double* h1 = H1 + i * (int64_t)h;
      double* y = H + i * (int64_t)o;
      for (int32_t k = 0; k < h; ++k) {
        double s = b1 ? b1[(int64_t)e * h + k] : 0.0;
        for (int32_t j = 0; j < d; ++j) s += w1[(int64_t)k * d + j] * x[j];
        h1[k] = store_round(s > 0.0 ? s : 0.0, store);
      }
      for (int32_t k = 0; k < o; ++k) {
        double s = b2 ? b2[(int64_t)e * o + k] : 0.0;
        for (int32_t j = 0; j < h; ++j) s += w2[(int64_t)k * h + j] * h1[j];
        y[k] = store_round(s, store);
      }
      /* the sample's decoder: the shared one, or its expert's own (Section 2) */
      const double* De = D + (ndec > 1 ? (int64_t)e * V * o : 0);
      const double* bDe = bD ? bD + (ndec > 1 ? (int64_t)e * V : 0) : NULL;
      double m = -INFINITY;
      for (int32_t v = 0; v < V; ++v) {
        double s = bDe ? bDe[v] : 0.0;
        const double* dv = De + (int64_t)v * o;
        for (int32_t j = 0; j < o; ++j) s += dv[j] * y[j];
        lg[v] = s;
        if (s > m) m = s;
      }
      double z = 0.0;
      for (int32_t v = 0; v < V; ++v) z += exp(lg[v] - m);
      double L = m + log(z);
      lse[i] = L;
      double pos = 0.0;
      int32_t np = row_ptr[i + 1] - row_ptr[i];
      for (int32_t q = row_ptr[i]; q < row_ptr[i + 1]; ++q) pos += lg[tag[q]];
      loss[i] = L - pos / (double)np;
      if (probs)
        for (int32_t v = 0; v < V; ++v) probs[i * (int64_t)V + v] = exp(lg[v] - L);
      if (logits)
        for (int32_t v = 0; v < V; ++v) logits[i * (int64_t)V + v] = lg[v];
    }
    free(lg);
  }
  if (bad) return -2;
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) s += loss[i];
  if (loss_mean) *loss_mean = n > 0 ? s / (double)n : 0.0;
  return 0;
}

/* --------------------------------------------------------------- O10: backward */

/* Gradient of the mean multilabel softmax loss (Section 4.1, Eq. 3) through the decoder
 * (shared, ndec = 1, or the expert's own, ndec = K; as in the forward) and the selected
 * expert (Section 2).  The gater is fixed (Section 2.2: the model is not trained end to
 * end), so nothing flows to the centroids.  Saved activations H1, H and lse are inputs (per
 * sample, in sample order).  With p = softmax(D_i H[i] + bD_i) and the uniform target y_i
 * (mass 1/|P_i| on each positive):
 *   g_i  = (p_i - y_i) * scale            (scale = 1/n for the batch mean)
 *   dbD  = sum_i g_i,  dD = sum_i g_i H[i]^T,  dh_i = D_i^T g_i
 *          (per decoder: decoder e sums over the samples of expert e when ndec = K)
 *   db2_e = sum dh,  dW2_e = sum dh h1^T,  dh1 = W2_e^T dh,  dz = dh1 * [h1 > 0]
 *   db1_e = sum dz,  dW1_e = sum dz x^T,   dx = W1_e^T dz
 * Rounding: `store` rounds dx, the one activation gradient the caller receives (in the data
 * dtype).  g, dh and dz are the paper's exact intermediate quantities and stay in fp64 unless
 * `istore` asks for them rounded (a diagnostic that models a device which stores them; dbD
 * always sums the unrounded g).  logit_round (diagnostic) rounds the recomputed logits by
 * `istore` before the softmax.  The plain gradient of Eq. 3 is istore = 0, logit_round = 0.
 * Experts that receive no sample get zero gradients.  dX may be NULL.
 * magnitude = 1 evaluates the same sums on absolute values -- |g|, then every product with
 * each factor's absolute value, nothing rounded -- which gives, per output, the scale M of the
 * standard first-order bound on the rounding error of the computation: an implementation
 * that rounds its operands with unit roundoff u stays within (number of roundings) * u * M of
 * the exact result (Higham, Accuracy and Stability of Numerical Algorithms, Section 3.1). */
static int moe_backward_impl(int64_t n, int32_t d, int32_t h, int32_t o, int32_t V, int32_t K,
                             int32_t ndec, const double* X, const int32_t* a, const double* W1,
                             const double* W2, const double* D, const double* bD,
                             const int32_t* row_ptr, const int32_t* tag, const double* H1,
                             const double* H, const double* lse, double scale, int store,
                             int istore, int logit_round, int magnitude, double* dW1, double* db1,
                             double* dW2, double* db2, double* dD, double* dbD, double* dX) {
#define MAG(x) (magnitude ? fabs(x) : (x))
  if (n < 0 || d <= 0 || h <= 0 || o <= 0 || V <= 0 || K <= 0) return -1;
  if (ndec != 1 && ndec != K) return -1;
  for (int64_t i = 0; i < n; ++i) {
    if (a[i] < 0 || a[i] >= K) return -3;
    if (row_ptr[i + 1] <= row_ptr[i]) return -4;
  }
  double* G = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * V);
  double* GS = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * V);
  double* dH = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * o);
  double* dZ = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * h);
  if (!G || !GS || !dH || !dZ) { free(G); free(GS); free(dH); free(dZ); return -2; }

  /* Per sample: g_i, dh_i, dz_i. */
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const int32_t e = a[i];
    const double* De = D + (ndec > 1 ? (int64_t)e * V * o : 0);
    const double* bDe = bD ? bD + (ndec > 1 ? (int64_t)e * V : 0) : NULL;
    const double* y = H + i * (int64_t)o;
    double* g = G + i * (int64_t)V;
    for (int32_t v = 0; v < V; ++v) {
      double s = bDe ? bDe[v] : 0.0;
      const double* dv = De + (int64_t)v * o;
      for (int32_t j = 0; j < o; ++j) s += dv[j] * y[j];
      if (logit_round) s = store_round(s, istore);
      g[v] = exp(s - lse[i]);
    }
    int32_t np = row_ptr[i + 1] - row_ptr[i];
    for (int32_t q = row_ptr[i]; q < row_ptr[i + 1]; ++q) g[tag[q]] -= 1.0 / (double)np;
    for (int32_t v = 0; v < V; ++v) g[v] = MAG(g[v] * scale);
    const int rstore = magnitude ? 0 : istore; /* the magnitude rounds nothing */
    double* gs = GS + i * (int64_t)V;
    for (int32_t v = 0; v < V; ++v) gs[v] = store_round(g[v], rstore);
    double* dh = dH + i * (int64_t)o;
    for (int32_t j = 0; j < o; ++j) dh[j] = 0.0;
    for (int32_t v = 0; v < V; ++v) {
      const double* dv = De + (int64_t)v * o;
      for (int32_t j = 0; j < o; ++j) dh[j] += gs[v] * MAG(dv[j]);
    }
    for (int32_t j = 0; j < o; ++j) dh[j] = store_round(dh[j], rstore);
    const double* w2 = W2 + (int64_t)e * o * h;
    const double* h1 = H1 + i * (int64_t)h;
    double* dz = dZ + i * (int64_t)h;
    for (int32_t k = 0; k < h; ++k) dz[k] = 0.0;
    for (int32_t j = 0; j < o; ++j)
      for (int32_t k = 0; k < h; ++k) dz[k] += dh[j] * MAG(w2[(int64_t)j * h + k]);
    for (int32_t k = 0; k < h; ++k) dz[k] = (h1[k] > 0.0) ? store_round(dz[k], rstore) : 0.0;
    if (dX) {
      const double* w1 = W1 + (int64_t)e * h * d;
      double* dx = dX + i * (int64_t)d;
      for (int32_t j = 0; j < d; ++j) dx[j] = 0.0;
      for (int32_t k = 0; k < h; ++k)
        for (int32_t j = 0; j < d; ++j) dx[j] += dz[k] * MAG(w1[(int64_t)k * d + j]);
      for (int32_t j = 0; j < d; ++j) dx[j] = store_round(dx[j], magnitude ? 0 : store);
    }
  }

  /* Decoder parameters: one (decoder, vocabulary row) per iteration, samples in ascending
   * order; decoder e sums the samples routed to expert e when every expert has its own. */
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < (int64_t)ndec * V; ++r) {
    const int32_t e = (int32_t)(r / V), v = (int32_t)(r % V);
    double* dd = dD + r * o;
    double sb = 0.0;
    for (int32_t j = 0; j < o; ++j) dd[j] = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      if (ndec > 1 && a[i] != e) continue;
      sb += G[i * (int64_t)V + v];
      const double g = GS[i * (int64_t)V + v];
      const double* y = H + i * (int64_t)o;
      for (int32_t j = 0; j < o; ++j) dd[j] += g * MAG(y[j]);
    }
    if (dbD) dbD[r] = sb;
  }

  /* Expert parameters: one (expert, output unit) row per iteration. */
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < (int64_t)K * o; ++r) {
    int32_t e = (int32_t)(r / o), j = (int32_t)(r % o);
    double* w = dW2 + ((int64_t)e * o + j) * h;
    double sb = 0.0;
    for (int32_t k = 0; k < h; ++k) w[k] = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      if (a[i] != e) continue;
      double g = dH[i * (int64_t)o + j];
      sb += g;
      const double* h1 = H1 + i * (int64_t)h;
      for (int32_t k = 0; k < h; ++k) w[k] += g * MAG(h1[k]);
    }
    if (db2) db2[(int64_t)e * o + j] = sb;
  }
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < (int64_t)K * h; ++r) {
    int32_t e = (int32_t)(r / h), k = (int32_t)(r % h);
    double* w = dW1 + ((int64_t)e * h + k) * d;
    double sb = 0.0;
    for (int32_t j = 0; j < d; ++j) w[j] = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      if (a[i] != e) continue;
      double g = dZ[i * (int64_t)h + k];
      sb += g;
      const double* x = X + i * (int64_t)d;
      for (int32_t j = 0; j < d; ++j) w[j] += g * MAG(x[j]);
    }
    if (db1) db1[(int64_t)e * h + k] = sb;
  }
  free(G);
  free(GS);
  free(dH);
  free(dZ);
  return 0;
#undef MAG
}

int hmoe_orc_moe_backward(int64_t n, int32_t d, int32_t h, int32_t o, int32_t V, int32_t K,
                          int32_t ndec, const double* X, const int32_t* a, const double* W1,
                          const double* W2, const double* D, const double* bD,
                          const int32_t* row_ptr, const int32_t* tag, const double* H1,
                          const double* H, const double* lse, double scale, int store,
                          int istore, int logit_round, int magnitude, double* dW1, double* db1,
                          double* dW2, double* db2, double* dD, double* dbD, double* dX) {
  return moe_backward_impl(n, d, h, o, V, K, ndec, X, a, W1, W2, D, bD, row_ptr, tag, H1, H, lse,
                           scale, store, istore, logit_round, magnitude, dW1, db1, dW2, db2, dD,
                           dbD, dX);
}

/* ------------------------------------------------ Section 4.4: t_m, p@m (Eq. 4), q@m (Eq. 5) */

/* t_m: the indices of the m largest entries of each row of L [n x V], in decreasing order of
 * value, equal values in increasing index order (the paper does not say how ties break).  Plain
 * selection: m scans per row, each taking the largest entry not yet taken (strict ">" keeps
 * the lowest index among equal values).  1 <= m <= V. */
int hmoe_orc_topm(int64_t n, int32_t V, int32_t m, const double* L, int32_t* idx) {
  if (n < 0 || V <= 0 || m <= 0 || m > V) return -1;
  int bad = 0;
#pragma omp parallel
  {
    char* taken = (char*)malloc((size_t)V);
    if (!taken) {
#pragma omp atomic write
      bad = 1;
    }
#pragma omp for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
      if (!taken) continue;
      const double* row = L + i * (int64_t)V;
      memset(taken, 0, (size_t)V);
      for (int32_t r = 0; r < m; ++r) {
        int32_t best = -1;
        for (int32_t v = 0; v < V; ++v)
          if (!taken[v] && (best < 0 || row[v] > row[best])) best = v;
        taken[best] = 1;
        idx[i * (int64_t)m + r] = best;
      }
    }
    free(taken);
  }
  return bad ? -2 : 0;
}

/* Counts behind Eq. 4 and Eq. 5 for every m' = 1..m, from the top-m lists idx [n x m]:
 *   p_hits[m'-1] = sum_i |t_m'(i) ∩ P_i|, so p@m' = p_hits[m'-1] / sum_i |P_i|;
 *   q_hits[m'-1] = number of the S given draws (q_sample[s], q_tag[s]) -- a tag drawn uniformly
 *   from the dictionary, then an image carrying it -- whose tag is in t_m'(q_sample[s]),
 *   so q@m' = q_hits[m'-1] / S. */
int hmoe_orc_topm_hits(int64_t n, int32_t m, const int32_t* idx, const int32_t* row_ptr,
                       const int32_t* tag, int64_t S, const int32_t* q_sample,
                       const int32_t* q_tag, int64_t* p_hits, int64_t* q_hits) {
  if (n < 0 || m <= 0 || S < 0) return -1;
  for (int32_t r = 0; r < m; ++r) p_hits[r] = q_hits[r] = 0;
  for (int64_t i = 0; i < n; ++i)
    for (int32_t r = 0; r < m; ++r) {
      const int32_t v = idx[i * (int64_t)m + r];
      int in = 0;
      for (int32_t q = row_ptr[i]; q < row_ptr[i + 1]; ++q)
        if (tag[q] == v) in = 1;
      if (in)
        for (int32_t k = r; k < m; ++k) p_hits[k] += 1; /* in t_m' for every m' > r */
    }
  for (int64_t s = 0; s < S; ++s) {
    const int64_t i = q_sample[s];
    if (i < 0 || i >= n) return -3;
    for (int32_t r = 0; r < m; ++r)
      if (idx[i * (int64_t)m + r] == q_tag[s])
        for (int32_t k = r; k < m; ++k) q_hits[k] += 1;
  }
  return 0;
}

/* ----------------------------------------------------------- Section 4.2: SGD update */

/* One SGD step on count parameters (Section 4.2: weight decay; momentum for the trunk, none
 * for the experts): g' = g + weight_decay * w; with momentum > 0, v = momentum * v + g' and
 * w = w - lr * v; otherwise w = w - lr * g'.  v may be NULL when momentum = 0. */
int hmoe_orc_sgd_step(int64_t count, double* w, const double* g, double* v, double lr,
                      double weight_decay, double momentum) {
  if (count < 0 || (momentum > 0.0 && !v)) return -1;
  for (int64_t i = 0; i < count; ++i) {
    const double gd = g[i] + weight_decay * w[i];
    if (momentum > 0.0) {
      v[i] = momentum * v[i] + gd;
      w[i] = w[i] - lr * v[i];
    } else {
      w[i] = w[i] - lr * gd;
    }
  }
  return 0;
}
