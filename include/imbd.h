/*
 * imbd.h -- C ABI of the MI355X (gfx950) hot path of integrated model/batch/domain
 * parallel SGD (Gholami, Azad, Jin, Keutzer, Buluc, arXiv:1712.04432).
 *
 * One process's share of the P_r x P_c grid: for each fully connected layer the three
 * products Y = W X, Delta_W = Delta_Y X^T and Delta_X = W^T Delta_Y (Sec. 1; Appendix A),
 * the nonlinearity and its derivative, softmax cross-entropy at the top and the
 * mini-batch SGD update of Eq. (1). Also a 3x3 convolution tile of a domain-parallel
 * layer with its halo supplied (Sec. 2.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Memory. Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *   never frees or keeps it. Calls enqueue work on `stream` (a hipStream_t passed as
 *   void*, NULL = the default stream) and return without synchronising. No call
 *   allocates device memory: scratch space comes in through a `ws` argument sized by the
 *   matching *_workspace_bytes function.
 * - Layout. The paper stores one sample per column (X_i is d_{i-1} x B); here one sample
 *   is one row of a row-major array, X[b][k], which is the same bytes as the paper's
 *   column-major X_i. Weights W_i are row-major [d_i][d_{i-1}] as in the paper.
 *   "ld" arguments are leading dimensions in ELEMENTS (>= the row length), so process
 *   blocks of a larger array are passed as views without copies.
 * - Types. IMBD_BF16 operands are bfloat16 bit patterns (uint16). Accumulation is
 *   always fp32; master weights, biases, gradients and the loss are fp32.
 *   Conversions to bf16 round to nearest, ties to even.
 * - Errors. Arguments are validated on the host before anything is enqueued; a bad
 *   argument returns IMBD_EINVAL and enqueues nothing. A launch failure returns IMBD_EHIP.
 *   imbd_last_error() gives a thread-local description of the last failure. No C++
 *   exception crosses this boundary. Labels outside [0, C) are not read out of bounds;
 *   their sample's loss and its whole row of the top-layer gradient become NaN, so the
 *   batch loss and every update computed from that gradient are NaN too.
 * - Determinism. Fixed reduction orders: identical inputs give identical bits.
 * - Concurrency. Calls that share a workspace must be ordered on one stream.
 */
#ifndef IMBD_H
#define IMBD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum imbd_status {
    IMBD_OK = 0,
    IMBD_EINVAL = -1,       /* bad argument (null pointer, size, leading dimension, enum) */
    IMBD_EUNSUPPORTED = -2, /* valid request the library has no kernel for */
    IMBD_EHIP = -3,         /* the HIP runtime reported an error */
    IMBD_EWORKSPACE = -4    /* workspace missing or smaller than *_workspace_bytes says */
};

enum imbd_dtype { IMBD_F32 = 0, IMBD_BF16 = 1 };

/* Static description of a status code; never NULL. mlp_status_string is the same
 * function under the name the rest of the mlp_* calls use. */
const char *imbd_status_string(int status);
const char *mlp_status_string(int status);
/* Detail of the last failure on the calling thread ("" if none). */
const char *imbd_last_error(void);
/* Library version, major*10000 + minor*100 + patch. */
int imbd_version(void);

/* ====================================================================================
 * Whole network (one process holding the full W_i and a batch of B samples: the
 * P_r = P_c = 1 case of Sec. 2.3)
 * ==================================================================================== */

/* A network of L fully connected layers d_0 -> d_1 -> ... -> d_L: ReLU after every
 * hidden layer, softmax cross-entropy on the top layer's logits. */
typedef struct {
    int n_layers;      /* L >= 1 */
    const int *dims;   /* HOST array of L+1 widths d_0..d_L, each >= 1 */
    int batch;         /* B >= 1 */
    int dtype;         /* IMBD_F32 or IMBD_BF16: type of weights copies and activations */
} imbd_mlp_desc;

/* Parameters of layer i (all device pointers, caller-owned). */
typedef struct {
    float *w;      /* fp32 master weights [d_i][d_{i-1}], contiguous */
    void *w_lp;    /* IMBD_BF16: bf16 copy [d_i][d_{i-1}] read by the products; IMBD_F32: == w */
    float *b;      /* fp32 bias [d_i] */
    float *dw;     /* fp32 [d_i][d_{i-1}]: Delta_W output when the update is not fused, else unused */
    float *db;     /* fp32 [d_i]: bias gradient output when the update is not fused, else unused */
} imbd_layer;

/* Bytes of workspace mlp_fwd/mlp_bwd need for this network (0 if the desc is invalid).
 * It holds X_2..X_L, the logits, every Delta_Y_i, the per-sample losses and the
 * split-K partial sums. */
size_t mlp_workspace_bytes(const imbd_mlp_desc *desc);

enum imbd_ws_kind {
    IMBD_WS_ACT = 0,     /* X_{i+1} = f(Y_i) for layer i in 1..L-1, [B][d_i] in desc->dtype */
    IMBD_WS_LOGITS = 1,  /* Y_L, [B][d_L] fp32 (layer argument ignored) */
    IMBD_WS_DY = 2,      /* Delta_Y_i for layer i in 1..L, [B][d_i] in desc->dtype */
    IMBD_WS_ROWLOSS = 3  /* per-sample loss, [B] fp32 (layer argument ignored) */
};
/* Byte offset of a region inside the workspace, or -1 for an invalid request. */
int64_t mlp_workspace_offset(const imbd_mlp_desc *desc, int kind, int layer);

/* Forward pass and loss (Sec. 1: Y_i = W_i X_i + b_i, X_{i+1} = f(Y_i); softmax
 * cross-entropy at the top). x: [B][d_0] input batch in desc->dtype. labels: [B] int32
 * class indices in [0, d_L). loss: device fp32 scalar, the batch-mean loss. Also leaves
 * Delta_Y_L = (softmax - onehot)/B in the workspace for mlp_bwd: the 1/B of Eq. (1) is
 * applied here, once. */
int mlp_fwd(const imbd_mlp_desc *desc, const imbd_layer *layers, const void *x,
            const int32_t *labels, void *ws, size_t ws_bytes, float *loss, void *stream);

/* Backward pass (Sec. 1 and Appendix A.2): for i = L..1, Delta_W_i = Delta_Y_i X_i^T,
 * db_i = Delta_Y_i 1, and for i >= 2 Delta_Y_{i-1} = (W_i^T Delta_Y_i) * [X_i > 0].
 * Needs the workspace of the mlp_fwd call just before it (same desc, same x).
 * fuse_sgd != 0: apply Eq. (1) in the weight-gradient epilogue,
 *   w <- w - lr*Delta_W, w_lp <- bf16(w), b <- b - lr*db, without storing Delta_W;
 *   each layer's Delta_X product is issued before its update, so it reads the old W.
 * fuse_sgd == 0: store Delta_W into layers[i].dw and db into layers[i].db; no update.
 * dx1: optional [B][d_0] output in desc->dtype for Delta_X_1 = W_1^T Delta_Y_1 (not
 * needed for training: the backward sum of Sec. 2.2 starts at layer 2); NULL skips it. */
int mlp_bwd(const imbd_mlp_desc *desc, imbd_layer *layers, const void *x, void *ws,
            size_t ws_bytes, int fuse_sgd, float lr, void *dx1, void *stream);

/* One SGD iteration: mlp_fwd followed by mlp_bwd with the update fused. */
int mlp_train_step(const imbd_mlp_desc *desc, imbd_layer *layers, const void *x,
                   const int32_t *labels, void *ws, size_t ws_bytes, float lr, float *loss,
                   void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): mlp_train_step with its workspace
 * taken from a scratch array inside the library instead of a ws argument. The array
 * holds IMBD_STATIC_SCRATCH_BYTES on every GPU the library runs on, from the library's
 * load until the process ends; the call itself allocates nothing. The caller still
 * passes parameters, input, labels and the loss. Results are those of mlp_train_step.
 * Returns IMBD_EWORKSPACE, enqueueing nothing, when mlp_workspace_bytes(desc) exceeds
 * the scratch (the 9216-4096-4096-1000 stack at B = 256 needs 46 MiB, 25088-4096-4096-1000
 * at B = 512 needs 53 MiB). All calls on one GPU share that GPU's one array, which keeps
 * the last call's contents: calls that overlap on one GPU (other streams, other threads)
 * race, so order them on one stream. The current device must be the stream's device. */
#define IMBD_STATIC_SCRATCH_BYTES (64u << 20)
int mlp_train_step_static(const imbd_mlp_desc *desc, imbd_layer *layers, const void *x,
                          const int32_t *labels, float lr, float *loss, void *stream);

/* ====================================================================================
 * Update and conversion
 * ==================================================================================== */

/* Eq. (1) on n parameters: w <- w - lr * grad_scale * grad (fp32, one rounding), then,
 * if w_lp != NULL and lp_dtype == IMBD_BF16, w_lp <- bf16(w). grad_scale = 1 when the
 * gradient already is the mini-batch mean. n == 0 is a no-op. Used for biases and for
 * local blocks after an external reduction. */
int sgd_step(float *w, void *w_lp, int lp_dtype, const float *grad, int64_t n, float lr,
             float grad_scale, void *stream);

/* dst[i] = bf16(src[i]) (round to nearest even; NaN stays NaN), n >= 0. */
int cast_f32_bf16(const float *src, uint16_t *dst, int64_t n, void *stream);

/* ====================================================================================
 * Single operations (the top of the network and single-layer products)
 * ==================================================================================== */

/* Softmax cross-entropy over C classes for B samples (the loss of Sec. 1 and App. A.2):
 * logits [B][ldz] fp32; loss = inv_batch * sum_b (logsumexp_c z_b - z_b[label_b]);
 * dz [B][lddz] in dz_dtype = inv_batch * (softmax(z_b) - onehot(label_b)).
 * row_loss: device fp32 [B] scratch that also receives the per-sample losses.
 * dz may be NULL (loss only). */
int softmax_xent(int B, int C, const float *logits, int64_t ldz, const int32_t *labels,
                 float inv_batch, float *loss, float *row_loss, void *dz, int64_t lddz,
                 int dz_dtype, void *stream);

/* ====================================================================================
 * Local blocks of one process (r, c) of the P_r x P_c grid (Sec. 2.3, the 1.5D
 * algorithm; Appendix A). The process holds a (d_i/P_r) x d_{i-1} row block of W_i and a
 * column block of B/P_c samples of X_i and Y_i. Outputs are left UNREDUCED: Y_blk waits
 * for the all-gather over P_r, the Delta_W partial for the all-reduce over P_c and the
 * Delta_X partial for the all-reduce over P_r (those collectives are not part of this
 * library). P_r, P_c >= 1 describe the grid; d_out_blk = d_i/P_r and b_blk = B/P_c are
 * the local sizes.
 * ==================================================================================== */

/* Y_blk = W_blk X_blk + b_blk (App. A.1, model-parallel form on the local samples),
 * then ReLU if relu != 0.
 * w_blk [d_out_blk][ldw] and x_blk [b_blk][ldx] in dtype; b_blk_bias [d_out_blk] fp32 or
 * NULL; y_blk [b_blk][ldy] in y_dtype (IMBD_F32 for logits).
 * ws/ws_bytes: scratch for split-K partial sums, see mlp_local_workspace_bytes. */
int mlp_local_fwd(int dtype, int relu, int P_r, int P_c, int d_out_blk, int d_in, int b_blk,
                  const void *w_blk, int64_t ldw, const float *b_blk_bias,
                  const void *x_blk, int64_t ldx, void *y_blk, int64_t ldy, int y_dtype,
                  void *ws, size_t ws_bytes, void *stream);

/* Backward products of the block (App. A.2):
 *   dw_part[m][k] = (1/B) sum_{b in block} dy_blk[b][m] x_blk[b][k],   B = b_blk * P_c
 *   db_part[m]    = (1/B) sum_{b in block} dy_blk[b][m]
 *   dx_part[b][k] = sum_m w_blk[m][k] dy_blk[b][m]  (times [x_blk[b][k] > 0] if mask_relu)
 * dy_blk is the raw per-sample gradient dJ/dY for J = sum_b f_b; the 1/B of Eq. (1) is
 * the global batch's, so the P_c partials sum to the mini-batch mean gradient. The
 * ReLU mask uses this layer's input block, which is the same on every process of the
 * grid column, so it commutes with the all-reduce over P_r.
 * w_blk [d_out_blk][ldw], x_blk [b_blk][ldx], dy_blk [b_blk][lddy] in dtype;
 * dw_part [d_out_blk][lddw] fp32; db_part [d_out_blk] fp32 or NULL;
 * dx_part [b_blk][lddx] fp32 or NULL (skip). b_blk == 0 writes zero partials. */
int mlp_local_bwd(int dtype, int P_r, int P_c, int d_out_blk, int d_in, int b_blk,
                  const void *w_blk, int64_t ldw, const void *dy_blk, int64_t lddy,
                  const void *x_blk, int64_t ldx, float *dw_part, int64_t lddw, float *db_part,
                  float *dx_part, int64_t lddx, int mask_relu, void *ws, size_t ws_bytes,
                  void *stream);

/* Workspace bytes for mlp_local_fwd (which = 0) or mlp_local_bwd (which = 1) at these
 * sizes. */
size_t mlp_local_workspace_bytes(int which, int dtype, int d_out_blk, int d_in, int b_blk);

/* ====================================================================================
 * Domain-parallel 3x3 convolution tile (Sec. 2.2, Fig. of the domain split; sizes from
 * Eq. (2)). Stride 1, "same" padding, cross-correlation, channels-last bf16 operands:
 *   x_pad  [N][H+2][W+2][C_in]  : the tile plus its 1-pixel halo (zeros on the image border)
 *   w      [C_out][3][3][C_in]
 *   dy_pad [N][H+2][W+2][C_out] : output gradient with its 1-pixel halo from the
 *                                 neighbouring tiles (output-side halo term of Eq. (7))
 * ==================================================================================== */

/* y[n][h][w][o] = sum_{r,s,c} w[o][r][s][c] x_pad[n][h+r][w+s][c]; y [N][H][W][C_out] in
 * y_dtype. */
int conv3x3_tile_fwd(int N, int H, int W, int C_in, int C_out, const void *x_pad,
                     const void *w, void *y, int y_dtype, void *stream);

/* dx[n][h][w][c] = sum_{r,s,o} w[o][r][s][c] dy_pad[n][h+2-r][w+2-s][o];
 * dx [N][H][W][C_in] in dx_dtype. */
int conv3x3_tile_dgrad(int N, int H, int W, int C_in, int C_out, const void *dy_pad,
                       const void *w, void *dx, int dx_dtype, void *stream);

/* The tile's partial weight gradient (the all-reduce over all processes of Eq. (7)
 * completes it): dw[o][r][s][c] = sum_{n,h,w} dy[n][h][w][o] x_pad[n][h+r][w+s][c],
 * dy = interior of dy_pad; dw [C_out][3][3][C_in] fp32. */
int conv3x3_tile_wgrad(int N, int H, int W, int C_in, int C_out, const void *x_pad,
                       const void *dy_pad, float *dw, void *ws, size_t ws_bytes, void *stream);
size_t conv3x3_wgrad_workspace_bytes(int N, int H, int W, int C_in, int C_out);

/* The tile's whole backward pass (Sec. 2.2; Eq. (7) for what it exchanges): the input
 * gradient (as conv3x3_tile_dgrad, skipped when dx is NULL) and the partial weight
 * gradient (as conv3x3_tile_wgrad), on `stream` in that order. Both passes are validated
 * before either is enqueued; ws must hold conv3x3_wgrad_workspace_bytes. */
int conv3x3_tile_bwd(int N, int H, int W, int C_in, int C_out, const void *x_pad, const void *w,
                     const void *dy_pad, void *dx, int dx_dtype, float *dw, void *ws,
                     size_t ws_bytes, void *stream);

/* ====================================================================================
 * Options: kernel routing and K splits (for A/B timing and for tests that force a
 * route; the defaults are the measured choices)
 * ==================================================================================== */
enum imbd_option {
    IMBD_OPT_SKINNY_OFF = 0,    /* 1: forward / Delta_X products of B <= 256 on the tiled template */
    IMBD_OPT_SKINNY_SPLITS = 1, /* K split of the B <= 256 product kernel, 0 = planned (0..64) */
    IMBD_OPT_TOP_UNFUSED = 2,   /* 1: the top layer's softmax in a launch of its own */
    IMBD_OPT_WIDE_OFF = 3,      /* 1: forward / Delta_X products of B > 256 on the tiled template */
    IMBD_OPT_WIDE_SPLITS = 4,   /* K split of the B > 256 product kernel, 0 = planned */
    IMBD_OPT_DW_WIDE_MIN_K = 5, /* smallest batch whose fused update runs on the large-tile
                                   kernel (default 257) */
    IMBD_OPT_DW_STREAM = 6,     /* 0: past 256 samples the persistent update kernel reloads its
                                   Delta_Y block per 256 samples instead of streaming it */
    IMBD_OPT_DW_GENERIC = 7,    /* 1: the fused update on the tiled template */
    IMBD_OPT_GEMM_CFG = 8,      /* tile configuration of the tiled template, -1 = planned (-1..3) */
    IMBD_OPT_GEMM_SPLITS = 9,   /* K split of the tiled template, 0 = planned */
    IMBD_OPT_CONV_NT = 10,      /* 0: the conv tile on the tiled template; 1: on the large-tile
                                   kernels, tile height planned (default); 2 / 3: with tiles of
                                   128 / 112 output positions */
    IMBD_OPT_SKINNY_NB = 11,    /* samples per workgroup of the B <= 256 product kernel, in units
                                   of 64 (1, 2 or 4), 0 = planned */
    IMBD_OPT_DW_WIDE_DUAL = 12, /* the large-tile fused update with two workgroups per CU
                                   (128-row tiles): 1 always, 0 never, -1 = planned (-1..1) */
    IMBD_OPT_LOCAL_PAIR = 13,   /* 0: the local backward pass's Delta_X and Delta_W products in two
                                   launches instead of one (default 1) */
    IMBD_OPT_REDUCE_TAIL = 14,  /* 0: a layer's Delta_X split-K reduce in a launch of its own instead
                                   of carried by that layer's update launch (default 1) */
    IMBD_OPT_COUNT = 15
};
/* Each option starts at the value of the environment variable named by
 * imbd_option_name(key) when the library is loaded (its default if unset or out of
 * range); the environment is not read again. imbd_set_option changes it for the whole
 * process: calls made afterwards use the new value. Options that move work between
 * kernels or change a K split change the workspace the *_workspace_bytes functions
 * report, so set them before sizing a workspace, and do not change them while another
 * thread has a call in flight. Returns IMBD_EINVAL for an unknown key or a value outside
 * the option's range. */
int imbd_set_option(int key, int value);
int imbd_get_option(int key, int *value);
/* The option's environment variable ("IMBD_..."), or "" for an unknown key. */
const char *imbd_option_name(int key);

/* ====================================================================================
 * Kernel timing (diagnostics for the roofline report)
 * ==================================================================================== */
enum imbd_kernel_class {
    IMBD_K_GEMM_FWD = 0, IMBD_K_GEMM_DX = 1, IMBD_K_GEMM_DW = 2, IMBD_K_SPLITK = 3,
    IMBD_K_SOFTMAX = 4, IMBD_K_BIAS = 5, IMBD_K_SGD = 6, IMBD_K_CAST = 7,
    IMBD_K_CONV_FWD = 8, IMBD_K_CONV_DGRAD = 9, IMBD_K_CONV_WGRAD = 10
};
/* Start recording HIP events around every launch of kernel class `cls` whose layer tag
 * equals `layer` (-1: any layer), up to max_launches launches. Creates the events
 * (outside any compute call). The fused weight-gradient + update kernel takes the
 * events in its own dispatch (hipExtLaunchKernelGGL), so they hold its start and end
 * times; other launches get events enqueued before and after them. Returns IMBD_EINVAL
 * if a recording is already open. */
int imbd_timing_begin(int cls, int layer, int max_launches);
/* Stop recording, wait for the recorded events, and return the number of launches and
 * the summed kernel time in milliseconds. Destroys the events. */
int imbd_timing_end(int *n_launches, double *total_ms);

#ifdef __cplusplus
}
#endif
#endif /* IMBD_H */
