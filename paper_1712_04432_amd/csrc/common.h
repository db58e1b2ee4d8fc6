// Internal declarations of the gfx950 library behind include/imbd.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "imbd.h"

namespace imbd {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------------- bf16 bits
// fp32 -> bf16, round to nearest, ties to even; NaN stays a (quiet) NaN. Adding
// 0x7fff plus the lowest kept bit and truncating rounds the 16 dropped bits to
// nearest-even, and a carry out of the significand correctly bumps the exponent
// (largest values overflow to infinity).
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__host__ __device__ inline float bf16_to_f32(uint16_t h) {
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// -------------------------------------------------------------------- GEMM epilogue
// Applied to each accumulated value acc(m, n) of a product; element (m, n) of every
// output lives at ptr + n*ld + m (m is the contiguous index).
enum EpiMode { EPI_STORE = 0, EPI_SGD = 1 };

struct Epilogue {
  int mode = EPI_STORE;
  float alpha = 1.0f;            // acc scale
  const float *bias = nullptr;   // STORE: + bias[m] after the scale
  int relu = 0;                  // STORE: max(., 0) after the bias
  const void *mask = nullptr;    // STORE: zero where !(mask(m, n) > 0)
  int64_t ldmask = 0;
  int mask_dtype = IMBD_BF16;
  void *out = nullptr;           // STORE: output; SGD: fp32 master weights (read-modify-write)
  int64_t ldo = 0;
  int out_dtype = IMBD_F32;
  uint16_t *out2 = nullptr;      // SGD: bf16 copy of the updated weights (may be null)
  int64_t ldo2 = 0;
  float lr = 0.0f;               // SGD: w <- w - lr * alpha * acc
};

// One product D(m, n) = sum_k A(m, k) B(k, n) for m < M, n < N, k < K.
//  A(m, k) is at A + m*lda + k when a_kc (k contiguous), else at A + k*lda + m.
//  B(k, n) is at B + n*ldb + k when b_kc, else at B + k*ldb + n.
// The three layer products map onto it as (memory is sample-major, W row-major):
//  forward  Y[b][o]  = sum_i W[o][i] X[b][i]   : m=o, n=b, k=i  (A=W k-contig, B=X k-contig)
//  dX       dX[b][i] = sum_o W[o][i] dY[b][o]  : m=i, n=b, k=o  (A=W strided,  B=dY k-contig)
//  dW       dW[o][i] = sum_b X[b][i] dY[b][o]  : m=i, n=o, k=b  (A=X strided,  B=dY strided)
struct GemmProblem {
  int dtype = IMBD_BF16;  // operand type, accumulation in fp32
  const void *A = nullptr;
  int64_t lda = 0;
  bool a_kc = true;
  const void *B = nullptr;
  int64_t ldb = 0;
  bool b_kc = true;
  int M = 0, N = 0, K = 0;
  Epilogue epi;
  // Sums of the B operand over k, db(n) = db_alpha * sum_k B(k, n), for the weight-gradient
  // product (B = Delta_Y stored [b][n], k = sample): the bias gradient comes out of the
  // same pass. db_mode 0: none, 1: store db_out[n], 2: bias[n] -= bias_lr * db(n).
  int db_mode = 0;
  float *db_out = nullptr;
  float *bias = nullptr;
  float db_alpha = 1.0f;
  float bias_lr = 0.0f;
  int kclass = IMBD_K_GEMM_FWD;  // timing tag
  int layer = 0;
  // Optional side job enqueued with the product: *aux_loss = aux_scale * sum of the aux_n
  // values at aux_rows (the batch mean of the per-sample losses, carried by a later launch
  // of the iteration instead of a launch of its own).
  const float *aux_rows = nullptr;
  float *aux_loss = nullptr;
  int aux_n = 0;
  float aux_scale = 1.0f;
  // B's rows hold zeros from K up to K rounded up to 8 (a copied block): the B <= 256
  // kernel may then take a K that is not a multiple of 8 when A is read by k-rows
  bool b_kpad8 = false;
  // B's rows only 4-byte aligned (base and pitch): the B <= 128 product kernel and the
  // 128-row large-tile weight-gradient kernel read them in 4-byte pieces (K even for the
  // former, N even for the latter); other routes do not take such a problem
  bool b_dw4 = false;
};

// Launch plan chosen for a product (a pure function of the shapes).
constexpr int PLAN_SKINNY = -1;  // GemmPlan::cfg of the skinny-batch kernel
constexpr int PLAN_WIDE = -2;    // ... of the wide-batch forward / Delta_X kernel
struct GemmPlan {
  int cfg;       // tile configuration index, or PLAN_SKINNY / PLAN_WIDE
  int bm, bn;    // tile sizes
  int splits;    // K splits (1 = no partial sums)
  int k_split;   // K elements per split (multiple of the K tile)
  size_t ws_bytes;
};

GemmPlan gemm_plan(const GemmProblem &p);
// Split-K partial sums: [split][N][ldp] floats, row pitch and split pitch kept off
// powers of two.
inline int64_t partial_ld(int M) { return ((int64_t)M + 7) / 8 * 8 + 64; }
inline int64_t partial_split_stride(int M, int N) { return (int64_t)N * partial_ld(M) + 1088; }
// Forward / Delta_X products for batches up to 256 (bf16): whether the skinny kernel
// takes the problem, its K split, the launch (kernel + its reduce) and the bytes of
// partial sums it needs in ws.
bool skinny_dims_fit(const GemmProblem &p);  // the conditions on M, N, K, dtype and epilogue mode
bool skinny_fits(const GemmProblem &p);
void skinny_plan(const GemmProblem &p, int *splits, int *k_split);
int run_skinny(const GemmProblem &p, void *ws, hipStream_t s);
// The skinny kernel's split-K reduce: its arguments, and the reduce left to a later launch.
struct SkReduceArgs {
  const float *partial;
  int64_t tpitch, sstride;
  int M, N, splits;
  Epilogue epi;
  const float *aux_rows;  // side job in one extra workgroup: *aux_loss = aux_scale * sum
  float *aux_loss;
  int aux_n;
  float aux_scale;
};
// The lean split-K reduce of the wide-batch and tiled products (partials [split][n][ldp]).
struct LeanReduceArgs {
  const float *partial;
  int64_t ldp, sstride;
  int M, N, splits;
  Epilogue epi;
};
// A split-K reduce left to a later launch: kind 1 the skinny kernel's (sk), kind 2 the lean
// one with the mask and a bf16 output (lean); items: one thread each (eight outputs of one
// sample), whole-vector accesses.
struct ReduceTail {
  int kind = 0;
  SkReduceArgs sk;
  LeanReduceArgs lean;
  int64_t items = 0;
};
// With deferred set, a reduce that one thread per item can do in its whole-vector form is
// not launched but returned in *tail (*deferred = true): the caller hands it to a later
// launch (run_dw_sgd) or to run_reduce_tail before anything reads the output or overwrites
// the partials in ws.
int run_skinny_split(const GemmProblem &p, void *ws, hipStream_t s, bool *deferred, ReduceTail *tail);
int run_reduce_tail(const ReduceTail &tail, int layer, hipStream_t s);  // the reduce's own launch
int run_skinny_reduce_tail(const ReduceTail &tail, int layer, hipStream_t s);  // ... of kind 1
size_t skinny_ws_bytes(const GemmProblem &p);
// Forward / Delta_X products for batches above 256 (bf16, B operand stored [n][k]):
// whether the large-tile kernel takes the problem (its dimensions alone, or with the
// leading dimensions and the operands' and output's alignment), its K split (slabs of 64 per split), and the launch
// (partials into partial when splits > 1; the caller adds them).
bool wide_dims_fit(const GemmProblem &p);  // the conditions on M, N, K, dtype and epilogue mode
bool wide_fits(const GemmProblem &p);
void wide_plan(const GemmProblem &p, int *splits, int *kps);
int run_wide(const GemmProblem &p, float *partial, int64_t ldp, int64_t sstride, hipStream_t s);
// The top layer's forward product with its split reduce fused into softmax cross-entropy
// (logits stored to p.epi.out, per-sample losses and the logits' gradient); the loss mean
// is left to the caller.
bool skinny_softmax_fits(const GemmProblem &p);
int run_skinny_softmax(const GemmProblem &p, void *ws, const int32_t *labels, float inv_batch, float *row_loss,
                       void *dz, int64_t lddz, int dz_dtype, hipStream_t s);
// The same pass on split partials laid out [split][row][ldp] (the wide-batch kernel's).
int run_softmax_rows_from_partials(const GemmProblem &p, const float *partial, int64_t ldp, int64_t sstride,
                                   int splits, const int32_t *labels, float inv_batch, float *row_loss, void *dz,
                                   int64_t lddz, int dz_dtype, hipStream_t s);
// ... and for a top layer on the wide-batch kernel with K split (past 256 samples).
bool wide_softmax_fits(const GemmProblem &p);
int run_wide_softmax(const GemmProblem &p, void *ws, size_t ws_bytes, const int32_t *labels, float inv_batch,
                     float *row_loss, void *dz, int64_t lddz, int dz_dtype, hipStream_t s);
int run_loss_mean(int B, const float *row_loss, float inv_batch, float *loss, hipStream_t s);
// The persistent fused weight-gradient + update kernel (bf16, K <= 2048): whether it
// takes the problem, and the launch.
bool dw_sgd_fits(const GemmProblem &p);
// tail: a skinny product's split-K reduce that the kernel's MMA waves run once their
// products are done (while the update waves finish the last tile); the launch must not
// write the reduce's partials or read its output.
int run_dw_sgd(const GemmProblem &p, hipStream_t s, const ReduceTail *tail = nullptr);
// The weight gradient on large tiles (bf16; the SGD update past 256 samples or the fp32
// store of alpha * Delta_W at any batch, in each tile's epilogue, the bias gradient on
// the column-sum kernel): whether it takes the problem, and the launch.
bool dw_wide_fits(const GemmProblem &p);
// tail (kind 2, fused update only): a wide-batch product's split-K reduce that every
// workgroup takes a share of after its tile; the launch must not write the reduce's
// partials or read its output.
int run_dw_wide(const GemmProblem &p, hipStream_t s, const ReduceTail *tail = nullptr);
// Enqueue the product; ws must hold plan.ws_bytes (partial sums) when splits > 1.
int gemm_run(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s);
// A Delta_X product whose split-K reduce a later launch may carry: as gemm_run, but on the
// skinny or wide-batch kernel (option IMBD_OPT_REDUCE_TAIL on) a deferrable reduce comes
// back in *tail (*deferred = true) instead of being launched; gemm_run_dw_tail then runs the
// weight gradient with it (on the update kernel that can carry it, or after the reduce's own
// launch). dw_sgd_route / dw_wide_route: the fused update problems that gemm_run sends to
// the persistent kernel / the large-tile kernel.
bool dw_sgd_route(const GemmProblem &p);
bool dw_wide_route(const GemmProblem &p);
int gemm_run_defer(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s, bool *deferred,
                   ReduceTail *tail);
int gemm_run_dw_tail(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s, const ReduceTail &tail);

// ----------------------------------------------------------------- other kernels
// mean: also launch the batch mean of the per-sample losses into *loss (else the caller
// enqueues it later)
int run_softmax_xent(int B, int C, const float *logits, int64_t ldz, const int32_t *labels,
                     float inv_batch, float *loss, float *row_loss, void *dz, int64_t lddz,
                     int dz_dtype, hipStream_t s, int layer, bool mean = true);
int run_bias_grad(int dtype, int M, int B, const void *dy, int64_t lddy, float alpha,
                  float *db_out, float *bias_sgd, float lr, hipStream_t s, int layer);
int run_sgd(float *w, uint16_t *w16, const float *g, int64_t n, float step, hipStream_t s,
            int layer);
int run_cast(const float *src, uint16_t *dst, int64_t n, hipStream_t s);
// dst[r][c] = src[r][c] for c < cols, 0 for cols <= c < ld_dst (bf16, any alignment of src)
int run_repack_bf16(const uint16_t *src, int64_t ld_src, int rows, int cols, uint16_t *dst, int64_t ld_dst,
                    hipStream_t s);
int run_conv_fwd(int N, int H, int W, int Ci, int Co, const void *xp, const void *w, void *y,
                 int y_dtype, hipStream_t s);
int run_conv_dgrad(int N, int H, int W, int Ci, int Co, const void *dyp, const void *w, void *dx,
                   int dx_dtype, hipStream_t s);
int run_conv_wgrad(int N, int H, int W, int Ci, int Co, const void *xp, const void *dyp,
                   float *dw, void *ws, size_t ws_bytes, hipStream_t s);
size_t conv_wgrad_ws_bytes(int N, int H, int W, int Ci, int Co);
// The forward (pass 1) and input-gradient (pass 2) passes for 256 output channels on the
// large-tile implicit-GEMM kernel: whether it takes the problem, and the launch.
bool conv_nt_fits(int pass, int N, int H, int W, int Ci, int Co, const void *act, const void *w, const void *out);
int run_conv_nt(int pass, int N, int H, int W, int Ci, int Co, const void *act, const void *w, void *out,
                int out_dtype, hipStream_t s);
// The weight-gradient pass (256 output channels, C_in a multiple of 128) on the large-tile
// kernel: fp32 split partials [split][C_out][ldp] into partial, added by the split-K reduce.
bool conv_wg_fits(int N, int H, int W, int Ci, int Co, const void *x, const void *dy, const void *dw);
void conv_wg_plan(int N, int H, int W, int Ci, int *splits, int *k_split);
int run_conv_wg(int N, int H, int W, int Ci, int Co, const void *x, const void *dy_pad, float *partial,
                int64_t ldp, int64_t sstride, hipStream_t s);

// --------------------------------------------------------------------- host helpers
// Current value of an option (enum imbd_option), set at load from the environment or by
// imbd_set_option.
int opt(int key);
void set_error(const char *fmt, ...);
int check_launch(const char *what);

// Records HIP events around one launch when timing is active for (cls, layer). With
// in_dispatch the events are not enqueued around the launch: the launch passes start()
// and stop() to hipExtLaunchKernelGGL, which stamps the kernel's own start and end.
struct LaunchTimer {
  LaunchTimer(int cls, int layer, hipStream_t s, bool in_dispatch = false);
  ~LaunchTimer();
  hipEvent_t start() const;  // nullptr when this launch is not timed
  hipEvent_t stop() const;
  hipStream_t stream;
  int slot;
  bool in_dispatch;
};

}  // namespace imbd
