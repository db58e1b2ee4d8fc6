// Host side of the C ABI declared in include/imbd.h: argument validation, workspace
// layout, launch order of one SGD iteration, and the kernel-timing hooks.
//
// Launch order of an iteration (Sec. 1 of the paper; Appendix A for the products):
//   forward  for i = 1..L : Y_i = W_i X_i + b_i, X_{i+1} = relu(Y_i)   (bias/ReLU fused)
//   top      softmax cross-entropy -> loss, Delta_Y_L = (softmax - onehot)/B
//   backward for i = L..1 : [i >= 2] Delta_Y_{i-1} = (W_i^T Delta_Y_i) * [X_i > 0]
//                           db_i (and b_i -= lr db_i)
//                           Delta_W_i = Delta_Y_i X_i^T with Eq. (1) fused: W_i -= lr Delta_W_i
// The Delta_X product of a layer is enqueued before that layer's update, so it reads the
// weights of this iteration.

#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>
#include <vector>

#include "common.h"
#include "local_pair.h"

namespace imbd {

// ------------------------------------------------------------------------ errors
static thread_local char g_err[512] = "";

void set_error(const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

int check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("%s: launch failed: %s", what, hipGetErrorString(e));
    return IMBD_EHIP;
  }
  return IMBD_OK;
}

#define FAIL(code, ...)   \
  do {                    \
    set_error(__VA_ARGS__); \
    return (code);        \
  } while (0)

#define TRY(expr)                \
  do {                           \
    int rc_ = (expr);            \
    if (rc_ != IMBD_OK) return rc_; \
  } while (0)

// ------------------------------------------------------------------------ timing
namespace {
struct Timing {
  std::mutex mu;
  bool active = false;
  int cls = -1, layer = -1, max = 0, used = 0;
  std::vector<hipEvent_t> ev;  // 2 per launch
} g_timing;
}  // namespace

LaunchTimer::LaunchTimer(int cls, int layer, hipStream_t s, bool in_dispatch_)
    : stream(s), slot(-1), in_dispatch(in_dispatch_) {
  if (!g_timing.active) return;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!g_timing.active || g_timing.cls != cls || (g_timing.layer >= 0 && g_timing.layer != layer) ||
      g_timing.used >= g_timing.max)
    return;
  slot = g_timing.used++;
  if (!in_dispatch) (void)hipEventRecord(g_timing.ev[2 * slot], s);
}

LaunchTimer::~LaunchTimer() {
  if (slot >= 0 && !in_dispatch) (void)hipEventRecord(g_timing.ev[2 * slot + 1], stream);
}

hipEvent_t LaunchTimer::start() const { return slot >= 0 ? g_timing.ev[2 * slot] : nullptr; }
hipEvent_t LaunchTimer::stop() const { return slot >= 0 ? g_timing.ev[2 * slot + 1] : nullptr; }

// ------------------------------------------------------------------ validation
static bool valid_dtype(int d) { return d == IMBD_F32 || d == IMBD_BF16; }
static size_t esize(int d) { return d == IMBD_BF16 ? 2 : 4; }
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static int check_desc(const imbd_mlp_desc *d) {
  if (!d) FAIL(IMBD_EINVAL, "desc is NULL");
  if (d->n_layers < 1) FAIL(IMBD_EINVAL, "n_layers = %d, need >= 1", d->n_layers);
  if (!d->dims) FAIL(IMBD_EINVAL, "dims is NULL");
  for (int i = 0; i <= d->n_layers; ++i)
    if (d->dims[i] < 1) FAIL(IMBD_EINVAL, "dims[%d] = %d, need >= 1", i, d->dims[i]);
  if (d->batch < 1) FAIL(IMBD_EINVAL, "batch = %d, need >= 1", d->batch);
  if (!valid_dtype(d->dtype)) FAIL(IMBD_EINVAL, "unknown dtype %d", d->dtype);
  return IMBD_OK;
}

// Forward product of layer i (1-based) as a GemmProblem, without pointers.
static GemmProblem fwd_problem(const imbd_mlp_desc *d, int i) {
  GemmProblem p;
  p.dtype = d->dtype;
  p.M = d->dims[i];
  p.N = d->batch;
  p.K = d->dims[i - 1];
  p.a_kc = true;
  p.b_kc = true;
  p.lda = p.K;
  p.ldb = p.K;
  p.kclass = IMBD_K_GEMM_FWD;
  p.layer = i;
  return p;
}
static GemmProblem dx_problem(const imbd_mlp_desc *d, int i) {
  GemmProblem p;
  p.dtype = d->dtype;
  p.M = d->dims[i - 1];
  p.N = d->batch;
  p.K = d->dims[i];
  p.a_kc = false;
  p.b_kc = true;
  p.lda = d->dims[i - 1];
  p.ldb = d->dims[i];
  p.kclass = IMBD_K_GEMM_DX;
  p.layer = i;
  return p;
}
static GemmProblem dw_problem(const imbd_mlp_desc *d, int i) {
  GemmProblem p;
  p.dtype = d->dtype;
  p.M = d->dims[i - 1];
  p.N = d->dims[i];
  p.K = d->batch;
  p.a_kc = false;
  p.b_kc = false;
  p.lda = d->dims[i - 1];
  p.ldb = d->dims[i];
  p.kclass = IMBD_K_GEMM_DW;
  p.layer = i;
  return p;
}

struct MlpLayout {
  size_t act[64], dy[64];  // act[i]: X_{i+1} for layer i; dy[i]: Delta_Y_i
  size_t logits, rowloss, partial, partial_bytes, total;
};

static int mlp_layout(const imbd_mlp_desc *d, MlpLayout *lay) {
  TRY(check_desc(d));
  if (d->n_layers > 62) FAIL(IMBD_EUNSUPPORTED, "at most 62 layers are supported");
  const int L = d->n_layers;
  const size_t es = esize(d->dtype), B = (size_t)d->batch;
  size_t off = 0;
  for (int i = 1; i < L; ++i) {
    lay->act[i] = off;
    off = align256(off + B * d->dims[i] * es);
  }
  lay->logits = off;
  off = align256(off + B * d->dims[L] * 4);
  for (int i = 1; i <= L; ++i) {
    lay->dy[i] = off;
    off = align256(off + B * d->dims[i] * es);
  }
  lay->rowloss = off;
  off = align256(off + B * 4);
  size_t part = 0;
  for (int i = 1; i <= L; ++i) {
    size_t a = gemm_plan(fwd_problem(d, i)).ws_bytes;
    size_t b = i >= 2 ? gemm_plan(dx_problem(d, i)).ws_bytes : 0;
    size_t c = gemm_plan(dw_problem(d, i)).ws_bytes;
    // layer-1 Delta_X is optional but budgeted so that dx1 requests always fit
    size_t e = i == 1 ? gemm_plan(dx_problem(d, 1)).ws_bytes : 0;
    for (size_t v : {a, b, c, e})
      if (v > part) part = v;
  }
  lay->partial = off;
  lay->partial_bytes = part;
  off = align256(off + part);
  lay->total = off;
  return IMBD_OK;
}

static int check_ws(const MlpLayout &lay, const void *ws, size_t ws_bytes) {
  if (!ws) FAIL(IMBD_EWORKSPACE, "workspace is NULL (need %zu bytes)", lay.total);
  if ((uintptr_t)ws % 256) FAIL(IMBD_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < lay.total) FAIL(IMBD_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, lay.total);
  return IMBD_OK;
}

static int check_layers(const imbd_mlp_desc *d, const imbd_layer *layers, bool need_grad_out) {
  if (!layers) FAIL(IMBD_EINVAL, "layers is NULL");
  for (int i = 0; i < d->n_layers; ++i) {
    const imbd_layer &l = layers[i];
    if (!l.w || !l.w_lp || !l.b) FAIL(IMBD_EINVAL, "layer %d: w, w_lp and b must be set", i + 1);
    if (d->dtype == IMBD_F32 && l.w_lp != l.w) FAIL(IMBD_EINVAL, "layer %d: fp32 network needs w_lp == w", i + 1);
    if (need_grad_out && (!l.dw || !l.db)) FAIL(IMBD_EINVAL, "layer %d: dw and db are required without fuse_sgd", i + 1);
  }
  return IMBD_OK;
}

static char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

}  // namespace imbd

using namespace imbd;

// =============================================================================== ABI
extern "C" {

const char *imbd_status_string(int status) {
  switch (status) {
    case IMBD_OK: return "ok";
    case IMBD_EINVAL: return "invalid argument";
    case IMBD_EUNSUPPORTED: return "unsupported request";
    case IMBD_EHIP: return "HIP runtime error";
    case IMBD_EWORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

const char *mlp_status_string(int status) { return imbd_status_string(status); }

const char *imbd_last_error(void) { return g_err; }

int imbd_version(void) { return 100; }

size_t mlp_workspace_bytes(const imbd_mlp_desc *desc) {
  MlpLayout lay;
  if (mlp_layout(desc, &lay) != IMBD_OK) return 0;
  return lay.total;
}

int64_t mlp_workspace_offset(const imbd_mlp_desc *desc, int kind, int layer) {
  MlpLayout lay;
  if (mlp_layout(desc, &lay) != IMBD_OK) return -1;
  const int L = desc->n_layers;
  switch (kind) {
    case IMBD_WS_ACT: return (layer >= 1 && layer < L) ? (int64_t)lay.act[layer] : -1;
    case IMBD_WS_LOGITS: return (int64_t)lay.logits;
    case IMBD_WS_DY: return (layer >= 1 && layer <= L) ? (int64_t)lay.dy[layer] : -1;
    case IMBD_WS_ROWLOSS: return (int64_t)lay.rowloss;
    default: set_error("unknown workspace kind %d", kind); return -1;
  }
}

}  // extern "C"

namespace imbd {
// The loss mean of an iteration when it is left to a later launch of the iteration.
struct LossJob {
  const float *rows = nullptr;
  float *loss = nullptr;
  int n = 0;
  float scale = 1.0f;
  bool pending = false;
};
}  // namespace imbd

// Forward pass and loss. With job set, the fused top-layer path leaves the loss mean in
// *job for a later launch instead of launching it.
static int fwd_impl(const imbd_mlp_desc *d, const imbd_layer *layers, const void *x, const int32_t *labels,
                    void *ws, size_t ws_bytes, float *loss, hipStream_t s, LossJob *job) {
  MlpLayout lay;
  TRY(mlp_layout(d, &lay));
  TRY(check_layers(d, layers, false));
  if (!x || !labels || !loss) FAIL(IMBD_EINVAL, "x, labels and loss must be set");
  TRY(check_ws(lay, ws, ws_bytes));
  const int L = d->n_layers, B = d->batch;
  void *part = at(ws, lay.partial);
  for (int i = 1; i <= L; ++i) {
    GemmProblem p = fwd_problem(d, i);
    p.A = layers[i - 1].w_lp;
    p.B = (i == 1) ? x : at(ws, lay.act[i - 1]);
    Epilogue &e = p.epi;
    e.mode = EPI_STORE;
    e.bias = layers[i - 1].b;
    if (i < L) {
      e.relu = 1;
      e.out = at(ws, lay.act[i]);
      e.out_dtype = d->dtype;
    } else {
      e.out = at(ws, lay.logits);
      e.out_dtype = IMBD_F32;
    }
    e.ldo = d->dims[i];
    if (i == L && gemm_plan(p).cfg == PLAN_SKINNY && skinny_softmax_fits(p)) {
      // top layer: split reduce, bias and softmax cross-entropy in one pass
      if (lay.partial_bytes < gemm_plan(p).ws_bytes) FAIL(IMBD_EWORKSPACE, "partial-sum region too small");
      float *rl = reinterpret_cast<float *>(at(ws, lay.rowloss));
      TRY(run_skinny_softmax(p, part, labels, 1.0f / (float)B, rl, at(ws, lay.dy[L]), d->dims[L], d->dtype, s));
      if (!job) return run_loss_mean(B, rl, 1.0f / (float)B, loss, s);
      *job = LossJob{rl, loss, B, 1.0f / (float)B, true};
      return IMBD_OK;
    }
    if (i == L && wide_softmax_fits(p)) {
      // the same past 256 samples: the wide-batch product's partials, then one pass
      float *rl = reinterpret_cast<float *>(at(ws, lay.rowloss));
      TRY(run_wide_softmax(p, part, lay.partial_bytes, labels, 1.0f / (float)B, rl, at(ws, lay.dy[L]), d->dims[L],
                           d->dtype, s));
      if (!job) return run_loss_mean(B, rl, 1.0f / (float)B, loss, s);
      *job = LossJob{rl, loss, B, 1.0f / (float)B, true};
      return IMBD_OK;
    }
    TRY(gemm_run(p, part, lay.partial_bytes, s));
  }
  // the batch mean of the per-sample losses rides on a later launch when the caller takes
  // the job (the top layer's Delta_X product), else it follows here
  float *rl = reinterpret_cast<float *>(at(ws, lay.rowloss));
  TRY(run_softmax_xent(B, d->dims[L], reinterpret_cast<const float *>(at(ws, lay.logits)), d->dims[L], labels,
                       1.0f / (float)B, loss, rl, at(ws, lay.dy[L]), d->dims[L], d->dtype, s, L, job == nullptr));
  if (job) *job = LossJob{rl, loss, B, 1.0f / (float)B, true};
  return IMBD_OK;
}

// Backward pass. A pending loss mean in *job rides on the top layer's Delta_X launch.
static int bwd_impl(const imbd_mlp_desc *d, imbd_layer *layers, const void *x, void *ws, size_t ws_bytes,
                    int fuse_sgd, float lr, void *dx1, hipStream_t s, LossJob *job) {
  MlpLayout lay;
  TRY(mlp_layout(d, &lay));
  TRY(check_layers(d, layers, !fuse_sgd));
  if (!x) FAIL(IMBD_EINVAL, "x must be set");
  if (fuse_sgd && !std::isfinite(lr)) FAIL(IMBD_EINVAL, "lr must be finite");
  TRY(check_ws(lay, ws, ws_bytes));
  const int L = d->n_layers;
  void *part = at(ws, lay.partial);
  for (int i = L; i >= 1; --i) {
    imbd_layer &ly = layers[i - 1];
    const void *dy = at(ws, lay.dy[i]);
    const void *xi = (i == 1) ? x : at(ws, lay.act[i - 1]);
    // Delta_W_i with the bias gradient from the same pass (row sums of the Delta_Y tile)
    GemmProblem pw = dw_problem(d, i);
    pw.A = xi;
    pw.B = dy;
    pw.db_mode = fuse_sgd ? 2 : 1;
    pw.db_out = ly.db;
    pw.bias = ly.b;
    pw.bias_lr = lr;
    {
      Epilogue &e = pw.epi;
      if (fuse_sgd) {
        e.mode = EPI_SGD;
        e.out = ly.w;
        e.ldo = d->dims[i - 1];
        e.out2 = (d->dtype == IMBD_BF16) ? reinterpret_cast<uint16_t *>(ly.w_lp) : nullptr;
        e.ldo2 = d->dims[i - 1];
        e.lr = lr;
      } else {
        e.mode = EPI_STORE;
        e.out = ly.dw;
        e.ldo = d->dims[i - 1];
        e.out_dtype = IMBD_F32;
      }
    }
    // The split-K reduce of Delta_X_i (into Delta_Y_{i-1}) rides on the update launch of
    // layer i when that runs on the persistent kernel (whose MMA waves add the partials
    // once their products are done) or on the large-tile one (whose workgroups share the
    // reduce out after their tiles): Delta_Y_{i-1} is first read by the next layer's
    // launches, and neither update kernel uses the workspace.
    bool deferred = false;
    ReduceTail tail;
    if (i >= 2 || dx1) {
      GemmProblem p = dx_problem(d, i);
      p.A = ly.w_lp;
      p.B = dy;
      Epilogue &e = p.epi;
      e.mode = EPI_STORE;
      if (i >= 2) {
        e.mask = xi;
        e.ldmask = d->dims[i - 1];
        e.mask_dtype = d->dtype;
        e.out = at(ws, lay.dy[i - 1]);
      } else {
        e.out = dx1;
      }
      e.ldo = d->dims[i - 1];
      e.out_dtype = d->dtype;
      if (job && job->pending) {
        p.aux_rows = job->rows;
        p.aux_loss = job->loss;
        p.aux_n = job->n;
        p.aux_scale = job->scale;
        job->pending = false;
      }
      if (i >= 2 && fuse_sgd && (dw_sgd_route(pw) || dw_wide_route(pw)))
        TRY(gemm_run_defer(p, part, lay.partial_bytes, s, &deferred, &tail));
      else TRY(gemm_run(p, part, lay.partial_bytes, s));
    }
    if (deferred) TRY(gemm_run_dw_tail(pw, part, lay.partial_bytes, s, tail));
    else TRY(gemm_run(pw, part, lay.partial_bytes, s));
  }
  return IMBD_OK;
}

extern "C" {

int mlp_fwd(const imbd_mlp_desc *d, const imbd_layer *layers, const void *x, const int32_t *labels,
            void *ws, size_t ws_bytes, float *loss, void *stream) {
  return fwd_impl(d, layers, x, labels, ws, ws_bytes, loss, reinterpret_cast<hipStream_t>(stream), nullptr);
}

int mlp_bwd(const imbd_mlp_desc *d, imbd_layer *layers, const void *x, void *ws, size_t ws_bytes,
            int fuse_sgd, float lr, void *dx1, void *stream) {
  return bwd_impl(d, layers, x, ws, ws_bytes, fuse_sgd, lr, dx1, reinterpret_cast<hipStream_t>(stream), nullptr);
}

// One iteration; the loss mean travels with the top layer's Delta_X launch when that runs on
// the skinny-batch or wide-batch kernel (one workgroup more there, one launch fewer), else
// it gets its own launch.
int mlp_train_step(const imbd_mlp_desc *d, imbd_layer *layers, const void *x, const int32_t *labels,
                   void *ws, size_t ws_bytes, float lr, float *loss, void *stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  LossJob job;
  TRY(fwd_impl(d, layers, x, labels, ws, ws_bytes, loss, s, &job));
  const int rc = bwd_impl(d, layers, x, ws, ws_bytes, 1, lr, nullptr, s, &job);
  if (job.pending) {
    const int rc2 = run_loss_mean(job.n, job.rows, job.scale, job.loss, s);
    if (rc == IMBD_OK) return rc2;
  }
  return rc;
}

int sgd_step(float *w, void *w_lp, int lp_dtype, const float *grad, int64_t n, float lr, float grad_scale,
             void *stream) {
  if (n < 0) FAIL(IMBD_EINVAL, "n = %lld", (long long)n);
  if (n == 0) return IMBD_OK;
  if (!w || !grad) FAIL(IMBD_EINVAL, "w and grad must be set");
  if (w_lp && lp_dtype != IMBD_BF16) FAIL(IMBD_EINVAL, "w_lp needs lp_dtype IMBD_BF16");
  if (!std::isfinite(lr) || !std::isfinite(grad_scale)) FAIL(IMBD_EINVAL, "lr and grad_scale must be finite");
  return run_sgd(w, reinterpret_cast<uint16_t *>(w_lp), grad, n, lr * grad_scale,
                 reinterpret_cast<hipStream_t>(stream), 0);
}

int cast_f32_bf16(const float *src, uint16_t *dst, int64_t n, void *stream) {
  if (n < 0) FAIL(IMBD_EINVAL, "n = %lld", (long long)n);
  if (n == 0) return IMBD_OK;
  if (!src || !dst) FAIL(IMBD_EINVAL, "src and dst must be set");
  return run_cast(src, dst, n, reinterpret_cast<hipStream_t>(stream));
}

int softmax_xent(int B, int C, const float *logits, int64_t ldz, const int32_t *labels, float inv_batch,
                 float *loss, float *row_loss, void *dz, int64_t lddz, int dz_dtype, void *stream) {
  if (B < 1 || C < 1) FAIL(IMBD_EINVAL, "B = %d, C = %d, need >= 1", B, C);
  if (!logits || !labels || !loss || !row_loss) FAIL(IMBD_EINVAL, "logits, labels, loss, row_loss must be set");
  if (ldz < C) FAIL(IMBD_EINVAL, "ldz %lld < C %d", (long long)ldz, C);
  if (dz && lddz < C) FAIL(IMBD_EINVAL, "lddz %lld < C %d", (long long)lddz, C);
  if (dz && !valid_dtype(dz_dtype)) FAIL(IMBD_EINVAL, "unknown dz dtype %d", dz_dtype);
  if (!std::isfinite(inv_batch)) FAIL(IMBD_EINVAL, "inv_batch must be finite");
  return run_softmax_xent(B, C, logits, ldz, labels, inv_batch, loss, row_loss, dz, lddz, dz_dtype,
                          reinterpret_cast<hipStream_t>(stream), 0);
}

// --------------------------------------------------------------------- local blocks
static GemmProblem local_fwd_problem(int dtype, int d_out_blk, int d_in, int b_blk) {
  GemmProblem p;
  p.dtype = dtype;
  p.M = d_out_blk;
  p.N = b_blk;
  p.K = d_in;
  p.a_kc = p.b_kc = true;
  p.lda = d_in;  // contiguous blocks; the caller's leading dimensions replace these
  p.ldb = d_in;
  p.kclass = IMBD_K_GEMM_FWD;
  return p;
}
static GemmProblem local_dw_problem(int dtype, int d_out_blk, int d_in, int b_blk) {
  GemmProblem p;
  p.dtype = dtype;
  p.M = d_in;
  p.N = d_out_blk;
  p.K = b_blk;
  p.a_kc = p.b_kc = false;
  p.lda = d_in;
  p.ldb = d_out_blk;
  p.kclass = IMBD_K_GEMM_DW;
  return p;
}
static GemmProblem local_dx_problem(int dtype, int d_out_blk, int d_in, int b_blk) {
  GemmProblem p;
  p.dtype = dtype;
  p.M = d_in;
  p.N = b_blk;
  p.K = d_out_blk;
  p.a_kc = false;
  p.b_kc = true;
  p.lda = d_in;
  p.ldb = d_out_blk;
  p.kclass = IMBD_K_GEMM_DX;
  p.b_kpad8 = dtype == IMBD_BF16 && d_out_blk % 8 != 0;  // the block is then always copied
  return p;
}

// A bf16 Delta_Y block whose rows are not whole 16-byte chunks (a 250-row block of the
// 1000-wide top layer has a 500-byte pitch; any block of a width that is not a multiple
// of 8): where its rows are 4-byte aligned and the paired launch takes both backward
// products, both read it in place in 4-byte pieces; otherwise it is copied once into the
// workspace with its rows padded with zeros to a multiple of 8 elements, so that both
// products run on the large-tile kernels.
static size_t local_dy_copy_bytes(int dtype, int d_out_blk, int b_blk) {
  if (dtype != IMBD_BF16 || b_blk <= 0) return 0;
  return align256((size_t)b_blk * (size_t)((d_out_blk + 7) / 8 * 8) * 2);
}
static bool local_dy_needs_copy(int dtype, int d_out_blk, const void *dy, int64_t lddy) {
  return dtype == IMBD_BF16 && ((uintptr_t)dy % 16 != 0 || lddy % 8 != 0 || d_out_blk % 8 != 0);
}

size_t mlp_local_workspace_bytes(int which, int dtype, int d_out_blk, int d_in, int b_blk) {
  if (!valid_dtype(dtype) || d_out_blk < 1 || d_in < 1 || b_blk < 0) return 0;
  if (which == 0) return gemm_plan(local_fwd_problem(dtype, d_out_blk, d_in, b_blk)).ws_bytes;
  size_t a = gemm_plan(local_dw_problem(dtype, d_out_blk, d_in, b_blk)).ws_bytes;
  size_t b = gemm_plan(local_dx_problem(dtype, d_out_blk, d_in, b_blk)).ws_bytes;
  return local_dy_copy_bytes(dtype, d_out_blk, b_blk) + (a > b ? a : b);
}

static int check_grid(int P_r, int P_c, int d_out_blk, int d_in, int b_blk) {
  if (P_r < 1 || P_c < 1) FAIL(IMBD_EINVAL, "grid %d x %d, need P_r, P_c >= 1", P_r, P_c);
  if (d_out_blk < 1 || d_in < 1) FAIL(IMBD_EINVAL, "block %d x %d, need >= 1", d_out_blk, d_in);
  if (b_blk < 0) FAIL(IMBD_EINVAL, "b_blk = %d", b_blk);
  return IMBD_OK;
}

int mlp_local_fwd(int dtype, int relu, int P_r, int P_c, int d_out_blk, int d_in, int b_blk, const void *w_blk,
                  int64_t ldw, const float *b_blk_bias, const void *x_blk, int64_t ldx, void *y_blk, int64_t ldy,
                  int y_dtype, void *ws, size_t ws_bytes, void *stream) {
  if (!valid_dtype(dtype) || !valid_dtype(y_dtype)) FAIL(IMBD_EINVAL, "unknown dtype");
  TRY(check_grid(P_r, P_c, d_out_blk, d_in, b_blk));
  if (b_blk == 0) return IMBD_OK;
  if (!w_blk || !x_blk || !y_blk) FAIL(IMBD_EINVAL, "w_blk, x_blk and y_blk must be set");
  if (ldw < d_in || ldx < d_in || ldy < d_out_blk) FAIL(IMBD_EINVAL, "leading dimension smaller than the row");
  GemmProblem p = local_fwd_problem(dtype, d_out_blk, d_in, b_blk);
  p.A = w_blk;
  p.lda = ldw;
  p.B = x_blk;
  p.ldb = ldx;
  p.epi.mode = EPI_STORE;
  p.epi.bias = b_blk_bias;
  p.epi.relu = relu ? 1 : 0;
  p.epi.out = y_blk;
  p.epi.ldo = ldy;
  p.epi.out_dtype = y_dtype;
  return gemm_run(p, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

// The local backward pass's two products: the Delta_W (+ bias) partial and the Delta_X
// partial, on the block's operands as given.
static GemmProblem local_dw_bwd_problem(int dtype, int d_out_blk, int d_in, int b_blk, const void *x_blk, int64_t ldx,
                                        const void *dy_blk, int64_t lddy, float *dw_part, int64_t lddw,
                                        float *db_part, float scale) {
  GemmProblem pw = local_dw_problem(dtype, d_out_blk, d_in, b_blk);
  pw.A = x_blk;
  pw.lda = ldx;
  pw.B = dy_blk;
  pw.ldb = lddy;
  if (db_part) {
    pw.db_mode = 1;
    pw.db_out = db_part;
    pw.db_alpha = scale;
  }
  pw.epi.mode = EPI_STORE;
  pw.epi.alpha = scale;
  pw.epi.out = dw_part;
  pw.epi.ldo = lddw;
  pw.epi.out_dtype = IMBD_F32;
  return pw;
}

static GemmProblem local_dx_bwd_problem(int dtype, int d_out_blk, int d_in, int b_blk, const void *w_blk, int64_t ldw,
                                        const void *dy_blk, int64_t lddy, const void *x_blk, int64_t ldx,
                                        float *dx_part, int64_t lddx, int mask_relu, bool kpad8) {
  GemmProblem p = local_dx_problem(dtype, d_out_blk, d_in, b_blk);
  p.b_kpad8 = kpad8;
  p.A = w_blk;
  p.lda = ldw;
  p.B = dy_blk;
  p.ldb = lddy;
  p.epi.mode = EPI_STORE;
  if (mask_relu) {
    p.epi.mask = x_blk;
    p.epi.ldmask = ldx;
    p.epi.mask_dtype = dtype;
  }
  p.epi.out = dx_part;
  p.epi.ldo = lddx;
  p.epi.out_dtype = IMBD_F32;
  return p;
}

int mlp_local_bwd(int dtype, int P_r, int P_c, int d_out_blk, int d_in, int b_blk, const void *w_blk, int64_t ldw,
                  const void *dy_blk, int64_t lddy, const void *x_blk, int64_t ldx, float *dw_part, int64_t lddw,
                  float *db_part, float *dx_part, int64_t lddx, int mask_relu, void *ws, size_t ws_bytes,
                  void *stream) {
  if (!valid_dtype(dtype)) FAIL(IMBD_EINVAL, "unknown dtype %d", dtype);
  TRY(check_grid(P_r, P_c, d_out_blk, d_in, b_blk));
  if (!dw_part) FAIL(IMBD_EINVAL, "dw_part must be set");
  if (lddw < d_in) FAIL(IMBD_EINVAL, "lddw < d_in");
  if (b_blk > 0) {
    if (!w_blk || !dy_blk || !x_blk) FAIL(IMBD_EINVAL, "w_blk, dy_blk and x_blk must be set");
    if (ldw < d_in || lddy < d_out_blk || ldx < d_in) FAIL(IMBD_EINVAL, "leading dimension smaller than the row");
    if (dx_part && lddx < d_in) FAIL(IMBD_EINVAL, "lddx < d_in");
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const float scale = 1.0f / ((float)b_blk * (float)P_c > 0 ? (float)b_blk * (float)P_c : 1.0f);
  // the copied Delta_Y block (if any) at the start of the workspace, the products' partial
  // sums after it
  const size_t cpy = local_dy_copy_bytes(dtype, d_out_blk, b_blk);
  bool copied = false;
  const bool needs_copy = b_blk > 0 && local_dy_needs_copy(dtype, d_out_blk, dy_blk, lddy);
  if (needs_copy && dx_part) {
    // rows of Delta_Y 4-byte aligned: the paired launch may read them in place
    GemmProblem pw = local_dw_bwd_problem(dtype, d_out_blk, d_in, b_blk, x_blk, ldx, dy_blk, lddy, dw_part, lddw,
                                          db_part, scale);
    GemmProblem p = local_dx_bwd_problem(dtype, d_out_blk, d_in, b_blk, w_blk, ldw, dy_blk, lddy, x_blk, ldx,
                                         dx_part, lddx, mask_relu, false);
    p.b_dw4 = pw.b_dw4 = true;
    void *wsp = ws && cpy > 0 ? reinterpret_cast<char *>(ws) + cpy : ws;
    const int rc = run_local_dx_dw_pair(p, pw, wsp, s);
    if (rc != 1) return rc;
  }
  if (needs_copy) {
    if (!ws || (uintptr_t)ws % 256 != 0 || ws_bytes < cpy)
      FAIL(IMBD_EWORKSPACE, "the Delta_Y block needs an aligned copy: workspace of %zu bytes, 256-byte aligned, "
                            "need at least %zu", ws_bytes, cpy);
    const int64_t ld8 = (d_out_blk + 7) / 8 * 8;
    TRY(run_repack_bf16(reinterpret_cast<const uint16_t *>(dy_blk), lddy, b_blk, d_out_blk,
                        reinterpret_cast<uint16_t *>(ws), ld8, s));
    dy_blk = ws;
    lddy = ld8;
    copied = true;
  }
  if (cpy > 0) {
    ws = ws ? reinterpret_cast<char *>(ws) + cpy : nullptr;
    ws_bytes = ws_bytes > cpy ? ws_bytes - cpy : 0;
  }
  const GemmProblem pw = local_dw_bwd_problem(dtype, d_out_blk, d_in, b_blk, x_blk, ldx, dy_blk, lddy, dw_part, lddw,
                                              db_part, scale);
  if (dx_part && b_blk > 0) {
    const GemmProblem p = local_dx_bwd_problem(dtype, d_out_blk, d_in, b_blk, w_blk, ldw, dy_blk, lddy, x_blk, ldx,
                                               dx_part, lddx, mask_relu, copied);
    // the two products are independent: one launch when both run on the large-tile
    // kernels without partial sums
    const int rc = run_local_dx_dw_pair(p, pw, ws, s);
    if (rc != 1) return rc;
    TRY(gemm_run(p, ws, ws_bytes, s));
  }
  return gemm_run(pw, ws, ws_bytes, s);
}

// ------------------------------------------------------------------------- conv tile
static int check_conv(int N, int H, int W, int Ci, int Co) {
  if (N < 0 || H < 1 || W < 1 || Ci < 1 || Co < 1) FAIL(IMBD_EINVAL, "bad conv sizes");
  return IMBD_OK;
}

int conv3x3_tile_fwd(int N, int H, int W, int C_in, int C_out, const void *x_pad, const void *w, void *y,
                     int y_dtype, void *stream) {
  TRY(check_conv(N, H, W, C_in, C_out));
  if (!valid_dtype(y_dtype)) FAIL(IMBD_EINVAL, "unknown y dtype");
  if (N == 0) return IMBD_OK;
  if (!x_pad || !w || !y) FAIL(IMBD_EINVAL, "x_pad, w and y must be set");
  return run_conv_fwd(N, H, W, C_in, C_out, x_pad, w, y, y_dtype, reinterpret_cast<hipStream_t>(stream));
}

int conv3x3_tile_dgrad(int N, int H, int W, int C_in, int C_out, const void *dy_pad, const void *w, void *dx,
                       int dx_dtype, void *stream) {
  TRY(check_conv(N, H, W, C_in, C_out));
  if (!valid_dtype(dx_dtype)) FAIL(IMBD_EINVAL, "unknown dx dtype");
  if (N == 0) return IMBD_OK;
  if (!dy_pad || !w || !dx) FAIL(IMBD_EINVAL, "dy_pad, w and dx must be set");
  return run_conv_dgrad(N, H, W, C_in, C_out, dy_pad, w, dx, dx_dtype, reinterpret_cast<hipStream_t>(stream));
}

int conv3x3_tile_wgrad(int N, int H, int W, int C_in, int C_out, const void *x_pad, const void *dy_pad, float *dw,
                       void *ws, size_t ws_bytes, void *stream) {
  TRY(check_conv(N, H, W, C_in, C_out));
  if (!dw) FAIL(IMBD_EINVAL, "dw must be set");
  if (N > 0 && (!x_pad || !dy_pad)) FAIL(IMBD_EINVAL, "x_pad and dy_pad must be set");
  return run_conv_wgrad(N, H, W, C_in, C_out, x_pad, dy_pad, dw, ws, ws_bytes,
                        reinterpret_cast<hipStream_t>(stream));
}

size_t conv3x3_wgrad_workspace_bytes(int N, int H, int W, int C_in, int C_out) {
  if (N < 0 || H < 1 || W < 1 || C_in < 1 || C_out < 1) return 0;
  return conv_wgrad_ws_bytes(N, H, W, C_in, C_out);
}

int conv3x3_tile_bwd(int N, int H, int W, int C_in, int C_out, const void *x_pad, const void *w,
                     const void *dy_pad, void *dx, int dx_dtype, float *dw, void *ws, size_t ws_bytes,
                     void *stream) {
  // validate both passes before enqueueing either
  TRY(check_conv(N, H, W, C_in, C_out));
  if (dx && !valid_dtype(dx_dtype)) FAIL(IMBD_EINVAL, "unknown dx dtype");
  if (!dw) FAIL(IMBD_EINVAL, "dw must be set");
  if (N > 0 && (!x_pad || !dy_pad || (dx && !w))) FAIL(IMBD_EINVAL, "x_pad, dy_pad (and w with dx) must be set");
  if (N > 0 && ws_bytes < conv_wgrad_ws_bytes(N, H, W, C_in, C_out))
    FAIL(IMBD_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, conv_wgrad_ws_bytes(N, H, W, C_in, C_out));
  if (dx) TRY(conv3x3_tile_dgrad(N, H, W, C_in, C_out, dy_pad, w, dx, dx_dtype, stream));
  return conv3x3_tile_wgrad(N, H, W, C_in, C_out, x_pad, dy_pad, dw, ws, ws_bytes, stream);
}

// --------------------------------------------------------------------------- timing
int imbd_timing_begin(int cls, int layer, int max_launches) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (g_timing.active) FAIL(IMBD_EINVAL, "a timing recording is already open");
  if (cls < 0 || cls > IMBD_K_CONV_WGRAD || max_launches < 1 || max_launches > 100000)
    FAIL(IMBD_EINVAL, "bad timing request");
  g_timing.ev.assign(2 * (size_t)max_launches, nullptr);
  for (auto &e : g_timing.ev)
    if (hipEventCreate(&e) != hipSuccess) {
      for (auto &f : g_timing.ev)
        if (f) (void)hipEventDestroy(f);
      g_timing.ev.clear();
      FAIL(IMBD_EHIP, "hipEventCreate failed");
    }
  g_timing.cls = cls;
  g_timing.layer = layer;
  g_timing.max = max_launches;
  g_timing.used = 0;
  g_timing.active = true;
  return IMBD_OK;
}

int imbd_timing_end(int *n_launches, double *total_ms) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!g_timing.active) FAIL(IMBD_EINVAL, "no timing recording is open");
  g_timing.active = false;
  double tot = 0.0;
  int rc = IMBD_OK;
  for (int i = 0; i < g_timing.used; ++i) {
    if (hipEventSynchronize(g_timing.ev[2 * i + 1]) != hipSuccess) {
      rc = IMBD_EHIP;
      set_error("hipEventSynchronize failed");
      break;
    }
    float ms = 0.f;
    (void)hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]);
    tot += ms;
  }
  for (auto &e : g_timing.ev) (void)hipEventDestroy(e);
  g_timing.ev.clear();
  if (n_launches) *n_launches = g_timing.used;
  if (total_ms) *total_ms = tot;
  return rc;
}

}  // extern "C"
