// api.hip -- the extern "C" entry points of include/hmoe.h: argument validation, workspace
// checks and dispatch to the launchers.  Host code only.
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "launch.hpp"

namespace hmoe {

static thread_local char g_err[512];

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

void clear_error() { g_err[0] = 0; }

// ------------------------------------------------------------------ launch timer
// Process-wide diagnostics state: a pool of event pairs recorded around each launch while
// enabled.  Not thread-safe; meant for a single benchmarking thread.
namespace {
struct LaunchTimer {
  bool on = false;
  std::vector<hipEvent_t> start, stop;
  std::vector<std::string> label;
  size_t used = 0;
  const char* pending = nullptr;
};
LaunchTimer g_timer;
}  // namespace

void timer_pre(const char* label, hipStream_t st) {
  if (!g_timer.on) return;
  if (g_timer.used == g_timer.start.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      hipEventDestroy(a);
      return;
    }
    g_timer.start.push_back(a);
    g_timer.stop.push_back(b);
    g_timer.label.emplace_back();
  }
  g_timer.pending = label;
  hipEventRecord(g_timer.start[g_timer.used], st);
}

void timer_post(hipStream_t st) {
  if (!g_timer.on || !g_timer.pending) return;
  hipEventRecord(g_timer.stop[g_timer.used], st);
  g_timer.label[g_timer.used] = g_timer.pending;
  g_timer.pending = nullptr;
  ++g_timer.used;
}

static int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

static int check_dtype(hmoe_dtype_t dt) {
  if (dt != HMOE_F32 && dt != HMOE_BF16) return fail(HMOE_EDTYPE, "unknown dtype %d", (int)dt);
  return HMOE_OK;
}

static int check_width(const char* name, int64_t w) {
  if (w <= 0 || w % 8 != 0) return fail(HMOE_ESHAPE, "%s = %lld must be a positive multiple of 8", name, (long long)w);
  return HMOE_OK;
}

static int check_ptr(const char* name, const void* p, bool need_align = true) {
  if (!p) return fail(HMOE_EINVAL, "%s is NULL", name);
  if (need_align && !aligned16(p)) return fail(HMOE_ESHAPE, "%s is not 16-byte aligned", name);
  return HMOE_OK;
}

static int check_k(int32_t K) {
  if (K < 1 || K > 4096) return fail(HMOE_EINVAL, "K = %d outside [1, 4096]", K);
  return HMOE_OK;
}

static int check_n(int64_t n) {
  if (n < 0 || n >= (int64_t(1) << 31)) return fail(HMOE_EINVAL, "n = %lld outside [0, 2^31)", (long long)n);
  return HMOE_OK;
}

static int check_ws(size_t need, size_t have, const void* ws) {
  if (need > 0 && (have < need || ws == nullptr))
    return fail(HMOE_EWORKSPACE, "workspace of %zu bytes given, %zu needed", have, need);
  return HMOE_OK;
}

// ------------------------------------------------------------------ allocation-free dispatch
// The scratch of hmoe_moe_dispatch_noalloc: one array per GPU the library runs on, held until
// the process ends.  In host code `scratch` names a host-side stand-in, not the array: its
// device address is looked up once per device (with that device current) and only that address
// is handed to kernels.
constexpr size_t kDispatchScratch = HMOE_DISPATCH_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kDispatchScratch];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_at[kMaxDevices];  // device address of `scratch` per device, NULL until looked up
}  // namespace

static int dispatch_scratch(void** at) {
  int dev = 0;
  HMOE_TRY(hip_check(hipGetDevice(&dev), "hipGetDevice"));
  if (dev < 0 || dev >= kMaxDevices) return fail(HMOE_EHIP, "device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_at[dev]) {
    void* p = nullptr;
    HMOE_TRY(hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
    if (!p) return fail(HMOE_EHIP, "hipGetSymbolAddress(scratch) gave NULL");
    g_scratch_at[dev] = p;
  }
  *at = g_scratch_at[dev];
  return HMOE_OK;
}

// Argument checks shared by the two dispatch entry points.
static int check_dispatch(const int32_t* expert, int64_t n, int32_t K, const int32_t* counts, const int32_t* offsets,
                          const int32_t* perm, const int32_t* inv, const void* rows, const void* rows_sorted,
                          hmoe_dtype_t dt, int32_t w) {
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_k(K));
  HMOE_TRY(check_ptr("counts", counts, false));
  HMOE_TRY(check_ptr("offsets", offsets, false));
  if (n > 0) {
    HMOE_TRY(check_ptr("expert", expert, false));
    HMOE_TRY(check_ptr("perm", perm, false));
    HMOE_TRY(check_ptr("inv", inv, false));
  }
  if (rows && n > 0) {
    HMOE_TRY(check_dtype(dt));
    HMOE_TRY(check_width("w", w));
    HMOE_TRY(check_ptr("rows", rows));
    HMOE_TRY(check_ptr("rows_sorted", rows_sorted));
  }
  return HMOE_OK;
}

static int run_dispatch(const int32_t* expert, int64_t n, int32_t K, int32_t* counts, int32_t* offsets,
                        int32_t* perm, int32_t* inv, const void* rows, void* rows_sorted, hmoe_dtype_t dt, int32_t w,
                        Workspace& wsp, hipStream_t st) {
  HMOE_TRY(launch_dispatch(expert, n, K, counts, offsets, perm, inv, wsp, st));
  if (rows && n > 0) HMOE_TRY(launch_permute(rows, rows_sorted, perm, n, w, dt, st));
  return HMOE_OK;
}

}  // namespace hmoe

using namespace hmoe;

extern "C" {

const char* hmoe_last_error(void) { return g_err; }

int hmoe_version(void) { return HMOE_VERSION; }

int hmoe_timer_enable(int on) {
  clear_error();
  g_timer.on = on != 0;
  g_timer.used = 0;
  g_timer.pending = nullptr;
  return HMOE_OK;
}

int64_t hmoe_timer_report(char* buf, size_t buf_bytes) {
  clear_error();
  // per label: launches and total milliseconds, in first-seen order
  std::vector<std::string> names;
  std::vector<double> ms;
  std::vector<long long> cnt;
  for (size_t i = 0; i < g_timer.used; ++i) {
    if (hipEventSynchronize(g_timer.stop[i]) != hipSuccess) return fail(HMOE_EHIP, "timer: event sync failed");
    float t = 0.f;
    if (hipEventElapsedTime(&t, g_timer.start[i], g_timer.stop[i]) != hipSuccess)
      return fail(HMOE_EHIP, "timer: elapsed time failed");
    size_t j = 0;
    while (j < names.size() && names[j] != g_timer.label[i]) ++j;
    if (j == names.size()) {
      names.push_back(g_timer.label[i]);
      ms.push_back(0.0);
      cnt.push_back(0);
    }
    ms[j] += t;
    cnt[j] += 1;
  }
  std::string out;
  char line[256];
  for (size_t j = 0; j < names.size(); ++j) {
    snprintf(line, sizeof(line), "%s\t%lld\t%.6f\n", names[j].c_str(), cnt[j], ms[j]);
    out += line;
  }
  if (buf && buf_bytes > 0) {
    const size_t m = out.size() < buf_bytes - 1 ? out.size() : buf_bytes - 1;
    memcpy(buf, out.data(), m);
    buf[m] = 0;
  }
  return (int64_t)out.size();
}

size_t hmoe_kmeans_assign_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt) {
  (void)d;
  (void)dt;
  if (n < 0 || K < 1) return 0;
  return assign_ws(n, K, dt);
}

int hmoe_kmeans_assign(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const void* C, int32_t K,
                       int32_t* assign, float* min_dist, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_k(K));
  HMOE_TRY(check_width("d", d));
  HMOE_TRY(check_ptr("C", C));
  if (n > 0) {
    HMOE_TRY(check_ptr("X", X));
    HMOE_TRY(check_ptr("assign", assign, false));
  }
  HMOE_TRY(check_ws(assign_ws(n, K, dt), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_assign(X, dt, n, d, C, K, assign, min_dist, w, (hipStream_t)stream);
}

size_t hmoe_kmeans_fit_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt) {
  if (n < 0 || K < 1 || d < 1) return 0;
  return fit_ws_bytes(n, d, K, dt);
}

int hmoe_kmeans_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t n_iter,
                    const double* init_uniforms, int32_t reseed_empty, float* C, int32_t* assign, float* min_dist,
                    int32_t* counts, double* objective, int32_t* init_idx, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_k(K));
  HMOE_TRY(check_width("d", d));
  if (n < K) return fail(HMOE_EINVAL, "k-means needs n >= K (n = %lld, K = %d)", (long long)n, K);
  if (n_iter < 0) return fail(HMOE_EINVAL, "n_iter = %d is negative", n_iter);
  HMOE_TRY(check_ptr("X", X));
  HMOE_TRY(check_ptr("C", C));
  HMOE_TRY(check_ptr("assign", assign, false));
  HMOE_TRY(check_ws(fit_ws_bytes(n, d, K, dt), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_fit(X, dt, n, d, K, n_iter, init_uniforms, reseed_empty, C, assign, min_dist, counts, objective,
                    init_idx, w, (hipStream_t)stream);
}

size_t hmoe_kmeans_update_workspace(int64_t n, int32_t d, int32_t K, hmoe_dtype_t dt) {
  (void)dt;
  if (n < 0 || K < 1 || d < 1) return 0;
  return update_ws_bytes(n, d, K);
}

int hmoe_kmeans_update(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t K, int32_t* assign,
                       const float* min_dist, double* sums, int64_t* counts, float* C, int32_t mode,
                       int32_t reseed_empty, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_k(K));
  HMOE_TRY(check_width("d", d));
  if (mode != HMOE_UPDATE_FULL && mode != HMOE_UPDATE_ACCUMULATE && mode != HMOE_UPDATE_FINALIZE)
    return fail(HMOE_EINVAL, "unknown update mode %d", mode);
  HMOE_TRY(check_ptr("sums", sums, false));
  HMOE_TRY(check_ptr("counts", counts, false));
  if (mode != HMOE_UPDATE_ACCUMULATE) HMOE_TRY(check_ptr("C", C, false));
  if (mode != HMOE_UPDATE_FINALIZE && n > 0) {
    HMOE_TRY(check_ptr("X", X));
    HMOE_TRY(check_ptr("assign", assign, false));
    if (mode == HMOE_UPDATE_FULL && reseed_empty) HMOE_TRY(check_ptr("min_dist", min_dist, false));
  }
  HMOE_TRY(check_ws(update_ws_bytes(n, d, K), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_update(X, dt, n, d, K, assign, min_dist, sums, counts, C, mode, reseed_empty, w,
                       (hipStream_t)stream);
}

size_t hmoe_moe_dispatch_workspace(int64_t n, int32_t K) {
  if (n < 0 || K < 1) return 0;
  return dispatch_ws(n, K);
}

int hmoe_moe_dispatch(const int32_t* expert, int64_t n, int32_t K, int32_t* counts, int32_t* offsets, int32_t* perm,
                      int32_t* inv, const void* rows, void* rows_sorted, hmoe_dtype_t dt, int32_t w, void* ws,
                      size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_dispatch(expert, n, K, counts, offsets, perm, inv, rows, rows_sorted, dt, w));
  HMOE_TRY(check_ws(dispatch_ws(n, K), ws_bytes, ws));
  Workspace wsp(ws, ws_bytes);
  return run_dispatch(expert, n, K, counts, offsets, perm, inv, rows, rows_sorted, dt, w, wsp, (hipStream_t)stream);
}

int hmoe_moe_dispatch_noalloc(const int32_t* expert, int64_t n, int32_t K, int32_t* counts, int32_t* offsets,
                              int32_t* perm, int32_t* inv, const void* rows, void* rows_sorted, hmoe_dtype_t dt,
                              int32_t w, void* stream) {
  clear_error();
  HMOE_TRY(check_dispatch(expert, n, K, counts, offsets, perm, inv, rows, rows_sorted, dt, w));
  const size_t need = dispatch_ws(n, K);
  if (need > kDispatchScratch)
    return fail(HMOE_EWORKSPACE,
                "the dispatch of n = %lld rows into K = %d experts needs %zu bytes of scratch; the allocation-free "
                "dispatch holds %zu (use hmoe_moe_dispatch with a workspace)",
                (long long)n, K, need, kDispatchScratch);
  void* at = nullptr;
  HMOE_TRY(dispatch_scratch(&at));
  Workspace wsp(at, kDispatchScratch);
  return run_dispatch(expert, n, K, counts, offsets, perm, inv, rows, rows_sorted, dt, w, wsp, (hipStream_t)stream);
}

int hmoe_permute_rows(const void* in, void* out, const int32_t* index, int64_t n, int32_t w, hmoe_dtype_t dt,
                      void* stream) {
  clear_error();
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_width("w", w));
  if (n == 0) return HMOE_OK;
  HMOE_TRY(check_ptr("in", in));
  HMOE_TRY(check_ptr("out", out));
  HMOE_TRY(check_ptr("index", index, false));
  return launch_permute(in, out, index, n, w, dt, (hipStream_t)stream);
}

static int check_params(const hmoe_moe_params_t* p) {
  if (!p) return fail(HMOE_EINVAL, "params is NULL");
  HMOE_TRY(check_dtype(p->dt));
  HMOE_TRY(check_k(p->K));
  HMOE_TRY(check_width("d_in", p->d_in));
  HMOE_TRY(check_width("d_hid", p->d_hid));
  HMOE_TRY(check_width("d_out", p->d_out));
  HMOE_TRY(check_width("vocab", p->vocab));
  if ((int64_t)p->d_hid > 8192 || (int64_t)p->d_out > 8192)
    return fail(HMOE_ESHAPE, "d_hid and d_out are limited to 8192");
  HMOE_TRY(check_ptr("W1", p->W1));
  HMOE_TRY(check_ptr("W2", p->W2));
  HMOE_TRY(check_ptr("D", p->D));
  if (p->decoders != 0 && p->decoders != 1 && p->decoders != p->K)
    return fail(HMOE_EINVAL, "decoders must be 1 (shared) or K (one per expert)");
  return HMOE_OK;
}

size_t hmoe_moe_workspace(const hmoe_moe_params_t* p, int64_t n) {
  if (!p || n < 0) return 0;
  return moe_ws_bytes(p, n);
}

int hmoe_moe_forward(const hmoe_moe_params_t* p, int64_t n, const void* X_sorted, const int32_t* offsets,
                     const int32_t* perm, const hmoe_labels_t* y, void* H1_sorted, void* H, void* logits,
                     float* logit_anchor, float* lse, float* loss, float* loss_mean, void* ws, size_t ws_bytes,
                     void* stream) {
  clear_error();
  HMOE_TRY(check_params(p));
  HMOE_TRY(check_n(n));
  if (n == 0) return HMOE_OK;
  HMOE_TRY(check_ptr("X_sorted", X_sorted));
  HMOE_TRY(check_ptr("offsets", offsets, false));
  HMOE_TRY(check_ptr("perm", perm, false));
  if (!y) return fail(HMOE_EINVAL, "labels are NULL");
  HMOE_TRY(check_ptr("labels.row_ptr", y->row_ptr, false));
  HMOE_TRY(check_ptr("labels.tag", y->tag, false));
  HMOE_TRY(check_ptr("H1_sorted", H1_sorted));
  HMOE_TRY(check_ptr("H", H));
  if (logits) {
    HMOE_TRY(check_ptr("logits", logits));
    HMOE_TRY(check_ptr("logit_anchor (required with logits)", logit_anchor));
  }
  HMOE_TRY(check_ptr("lse", lse, false));
  HMOE_TRY(check_ptr("loss", loss, false));
  HMOE_TRY(check_ptr("loss_mean", loss_mean, false));
  HMOE_TRY(check_ws(moe_ws_bytes(p, n), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_moe_forward(p, n, X_sorted, offsets, perm, y, H1_sorted, H, logits, logit_anchor, lse, loss,
                            loss_mean, w, (hipStream_t)stream);
}

int hmoe_moe_backward(const hmoe_moe_params_t* p, int64_t n, const void* X_sorted, const int32_t* offsets,
                      const int32_t* perm, const int32_t* inv, const hmoe_labels_t* y, const void* H1_sorted,
                      const void* H, const void* logits, const float* logit_anchor, const float* lse, float* dW1,
                      float* db1, float* dW2, float* db2, float* dD, float* dbD, void* dX, void* ws, size_t ws_bytes,
                      void* stream) {
  clear_error();
  HMOE_TRY(check_params(p));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_ptr("dW1", dW1, false));
  HMOE_TRY(check_ptr("dW2", dW2, false));
  HMOE_TRY(check_ptr("dD", dD, false));
  if (n == 0) {
    // empty batch: every gradient is zero
    hipStream_t st = (hipStream_t)stream;
    const int64_t K = p->K, d = p->d_in, h = p->d_hid, o = p->d_out, V = p->vocab;
    const int64_t nd = p->decoders > 1 ? p->decoders : 1;
    HMOE_TRY(launch_zero_f32(dW1, K * h * d, st));
    HMOE_TRY(launch_zero_f32(dW2, K * o * h, st));
    HMOE_TRY(launch_zero_f32(dD, nd * V * o, st));
    if (db1) HMOE_TRY(launch_zero_f32(db1, K * h, st));
    if (db2) HMOE_TRY(launch_zero_f32(db2, K * o, st));
    if (dbD) HMOE_TRY(launch_zero_f32(dbD, nd * V, st));
    return HMOE_OK;
  }
  HMOE_TRY(check_ptr("X_sorted", X_sorted));
  HMOE_TRY(check_ptr("offsets", offsets, false));
  HMOE_TRY(check_ptr("perm", perm, false));
  HMOE_TRY(check_ptr("inv", inv, false));
  if (!y) return fail(HMOE_EINVAL, "labels are NULL");
  HMOE_TRY(check_ptr("labels.row_ptr", y->row_ptr, false));
  HMOE_TRY(check_ptr("labels.tag", y->tag, false));
  HMOE_TRY(check_ptr("H1_sorted", H1_sorted));
  HMOE_TRY(check_ptr("H", H));
  HMOE_TRY(check_ptr("lse", lse, false));
  if (logits) {
    HMOE_TRY(check_ptr("logits", logits));
    HMOE_TRY(check_ptr("logit_anchor (required with logits)", logit_anchor));
  } else if (p->decoders > 1)
    return fail(HMOE_EINVAL, "with one decoder per expert the backward needs the forward's saved logits");
  if (dX) HMOE_TRY(check_ptr("dX", dX));
  HMOE_TRY(check_ws(moe_ws_bytes(p, n), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_moe_backward(p, n, X_sorted, offsets, perm, inv, y, H1_sorted, H, logits, logit_anchor, lse, dW1,
                             db1, dW2, db2, dD, dbD, dX, w, (hipStream_t)stream);
}

static int check_pca(hmoe_dtype_t dt, int64_t n, int32_t d, int32_t r) {
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_width("d", d));
  HMOE_TRY(check_width("r", r));
  if (r > d) return fail(HMOE_EINVAL, "r = %d exceeds d = %d", r, d);
  return HMOE_OK;
}

size_t hmoe_pca_workspace(int64_t n, int32_t d, int32_t r, hmoe_dtype_t dt) {
  if (n < 0 || d <= 0 || r <= 0) return 0;
  const size_t a = pca_fit_ws(n, d, r, dt), b = pca_project_ws(d, r, dt);
  return a > b ? a : b;
}

int hmoe_pca_fit(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, int32_t r, int32_t n_iter, uint64_t seed,
                 float* mean, float* components, float* eigvals, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_pca(dt, n, d, r));
  if (n < 2) return fail(HMOE_EINVAL, "n = %lld: the sample covariance needs n >= 2", (long long)n);
  if (n_iter < 0) return fail(HMOE_EINVAL, "n_iter = %d is negative", n_iter);
  HMOE_TRY(check_ptr("X", X));
  HMOE_TRY(check_ptr("mean", mean, false));
  HMOE_TRY(check_ptr("components", components));
  HMOE_TRY(check_ptr("eigvals", eigvals, false));
  HMOE_TRY(check_ws(hmoe_pca_workspace(n, d, r, dt), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_pca_fit(X, dt, n, d, r, n_iter, seed, mean, components, eigvals, w, (hipStream_t)stream);
}

int hmoe_pca_project(const void* X, hmoe_dtype_t dt, int64_t n, int32_t d, const float* mean,
                     const float* components, int32_t r, void* Z, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  HMOE_TRY(check_pca(dt, n, d, r));
  if (n == 0) return HMOE_OK;
  HMOE_TRY(check_ptr("X", X));
  HMOE_TRY(check_ptr("mean", mean, false));
  HMOE_TRY(check_ptr("components", components, false));
  HMOE_TRY(check_ptr("Z", Z));
  HMOE_TRY(check_ws(hmoe_pca_workspace(n, d, r, dt), ws_bytes, ws));
  Workspace w(ws, ws_bytes);
  return launch_pca_project(X, dt, n, d, mean, components, r, Z, w, (hipStream_t)stream);
}

int hmoe_sgd_step(float* w, const float* g, float* v, void* w_lo, hmoe_dtype_t dt, int64_t count, float lr,
                  float weight_decay, float momentum, void* stream) {
  clear_error();
  HMOE_TRY(check_dtype(dt));
  if (count < 0) return fail(HMOE_EINVAL, "count = %lld is negative", (long long)count);
  if (!(lr >= 0.f) || !(weight_decay >= 0.f) || !(momentum >= 0.f))
    return fail(HMOE_EINVAL, "lr, weight_decay and momentum must be >= 0");
  if (count == 0) return HMOE_OK;
  HMOE_TRY(check_ptr("w", w));
  HMOE_TRY(check_ptr("g", g));
  if (momentum > 0.f) HMOE_TRY(check_ptr("v (momentum buffer)", v));
  if (w_lo) HMOE_TRY(check_ptr("w_lo", w_lo));
  return launch_sgd(w, g, momentum > 0.f ? v : nullptr, w_lo, dt, count, lr, weight_decay, momentum,
                    (hipStream_t)stream);
}

int hmoe_topm(const void* logits, const float* anchor, hmoe_dtype_t dt, int64_t n, int32_t vocab, int32_t m,
              int32_t* idx, float* val, void* stream) {
  clear_error();
  HMOE_TRY(check_dtype(dt));
  HMOE_TRY(check_n(n));
  HMOE_TRY(check_width("vocab", vocab));
  if (m < 1 || m > 16 || m > vocab) return fail(HMOE_EINVAL, "m = %d outside [1, min(16, vocab)]", m);
  if (n == 0) return HMOE_OK;
  HMOE_TRY(check_ptr("logits", logits));
  HMOE_TRY(check_ptr("idx", idx, false));
  if (anchor) HMOE_TRY(check_ptr("anchor", anchor));
  return launch_topm(logits, anchor, dt, n, vocab, m, idx, val, (hipStream_t)stream);
}

int hmoe_topm_hits(const int32_t* idx, int64_t n, int32_t m, const hmoe_labels_t* y, const int32_t* q_sample,
                   const int32_t* q_tag, int64_t S, int64_t* hits, void* stream) {
  clear_error();
  HMOE_TRY(check_n(n));
  if (m < 1 || m > 16) return fail(HMOE_EINVAL, "m = %d outside [1, 16]", m);
  if (S < 0 || S >= (int64_t(1) << 31)) return fail(HMOE_EINVAL, "S = %lld outside [0, 2^31)", (long long)S);
  HMOE_TRY(check_ptr("hits", hits, false));
  if (n > 0) {
    HMOE_TRY(check_ptr("idx", idx, false));
    if (!y) return fail(HMOE_EINVAL, "labels are NULL");
    HMOE_TRY(check_ptr("labels.row_ptr", y->row_ptr, false));
    HMOE_TRY(check_ptr("labels.tag", y->tag, false));
  }
  if (S > 0) {
    HMOE_TRY(check_ptr("q_sample", q_sample, false));
    HMOE_TRY(check_ptr("q_tag", q_tag, false));
  }
  static const hmoe_labels_t none = {nullptr, nullptr};
  return launch_topm_hits(idx, n, m, y ? y : &none, q_sample, q_tag, S, hits, (hipStream_t)stream);
}

}  // extern "C"
