/*
 * oracle.c -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, obviously correct CPU implementation of what the data-parallel hot
 * path computes, in double precision. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it. It shares no code, header or table with
 * the device library and does not include anything from it.
 *
 * Paper: Gholami, Azad, Jin, Keutzer, Buluc, "Integrated Model, Batch and Domain
 * Parallelism in Training Neural Networks" (SPAA'18, arXiv:1712.04432).
 *
 * Orientation. The paper stores one sample per COLUMN (X_i is d_{i-1} x B). In memory
 * here one sample is one ROW of a row-major array: X[b][k] is the paper's X(k, b).
 * That is the same bytes as the paper's column-major matrix; only the indexing of the
 * comments below changes. W_i is row-major [d_i][d_{i-1}], exactly the paper's W_i.
 *
 * Every loop below is a direct transcription of a definition; OpenMP only splits the
 * independent output rows across threads and never changes a summation order.
 *
 * Parity pins for each function live in tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <omp.h>

typedef int64_t i64;

int orc_threads(void) { return omp_get_max_threads(); }
/* Threads of the parallel loops that follow (n >= 1); the results do not depend on it. */
void orc_set_threads(int n) { if (n >= 1) omp_set_num_threads(n); }

/* ---------------------------------------------------------------------------------
 * Rounding to the storage formats of the device path.
 *
 * bfloat16 has the binary32 exponent range and an 8-bit significand (7 stored bits).
 * Round-to-nearest, ties-to-even, written from the IEEE 754 definition: scale |x| so
 * that one unit in the last place of its binade is 1, round to an integer with ties
 * to even (nearbyint in the default rounding mode), scale back. Below 2^-126 the
 * spacing is fixed at 2^-133 (subnormals). Results above the largest finite bf16
 * value (0x1.fep127) overflow to infinity. NaN stays NaN.
 * --------------------------------------------------------------------------------- */
double orc_round_bf16(double x)
{
    if (x != x || x == 0.0 || isinf(x)) return x;
    double ax = fabs(x);
    int e;
    (void)frexp(ax, &e);              /* ax in [2^(e-1), 2^e) */
    int ulp_exp = e - 8;              /* 8 significant bits */
    if (ulp_exp < -133) ulp_exp = -133;
    double r = nearbyint(ldexp(ax, -ulp_exp));
    double y = ldexp(r, ulp_exp);
    if (y > 0x1.fep127) y = INFINITY;
    return copysign(y, x);
}

/* binary32 round-to-nearest-even: the C conversion double -> float in the default
 * rounding mode. */
double orc_round_f32(double x) { return (double)(float)x; }

/* mode 0: leave as is (fp64), 1: bfloat16, 2: binary32 */
void orc_round_array(double *a, i64 n, int mode)
{
    if (mode == 0) return;
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i)
        a[i] = (mode == 1) ? orc_round_bf16(a[i]) : orc_round_f32(a[i]);
}

/* ---------------------------------------------------------------------------------
 * Forward affine map of one fully connected layer (Sec. 1, forward phase: Y_i = W_i X_i;
 * Appendix A.1 for the data-parallel and model-parallel forms). A bias vector is added
 * to every column (the paper's layers carry none; the workloads here do).
 *   Y(m, b) = sum_k W(m, k) X(k, b) + bias(m)
 * memory: W [dout][ldw], X [B][ldx], Y [B][ldy]
 * --------------------------------------------------------------------------------- */
void orc_affine_fwd(int dout, int din, int B,
                    const double *W, i64 ldw, const double *X, i64 ldx,
                    const double *bias, double *Y, i64 ldy)
{
#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b)
        for (int m = 0; m < dout; ++m) {
            double s = 0.0;
            for (int k = 0; k < din; ++k) s += W[(i64)m * ldw + k] * X[(i64)b * ldx + k];
            Y[(i64)b * ldy + m] = s + (bias ? bias[m] : 0.0);
        }
}

/* Nonlinearity X_{i+1} = f(Y_i) with f = max(0, .) (Sec. 1; ReLU is the workloads' f). */
void orc_relu(double *Y, i64 n)
{
    for (i64 i = 0; i < n; ++i) Y[i] = Y[i] > 0.0 ? Y[i] : 0.0;
}

/* ---------------------------------------------------------------------------------
 * Softmax cross-entropy at the top of the network (the loss J is left unnamed in
 * Sec. 1 and Appendix A.2; the workloads use softmax cross-entropy). The mini-batch
 * mean of Eq. (1) is folded into the top gradient: with inv_batch = 1/B,
 *   loss = inv_batch * sum_b ( log sum_c exp Z(c,b) - Z(label_b, b) )
 *   dZ(c, b) = inv_batch * ( exp Z(c,b) / sum_c' exp Z(c',b) - [c == label_b] )
 * The log-sum-exp is evaluated with the column maximum subtracted first.
 * memory: Z [B][ldz], dZ [B][lddz]; per-sample losses (before the mean) in row_loss.
 * --------------------------------------------------------------------------------- */
void orc_softmax_xent(int C, int B, const double *Z, i64 ldz, const int32_t *labels,
                      double inv_batch, double *loss, double *dZ, i64 lddz, double *row_loss)
{
    double total = 0.0;
    for (int b = 0; b < B; ++b) {
        const double *z = Z + (i64)b * ldz;
        double mx = z[0];
        for (int c = 1; c < C; ++c) if (z[c] > mx) mx = z[c];
        double s = 0.0;
        for (int c = 0; c < C; ++c) s += exp(z[c] - mx);
        double lse = mx + log(s);
        double lb = lse - z[labels[b]];
        if (row_loss) row_loss[b] = lb;
        total += lb;
        if (dZ)
            for (int c = 0; c < C; ++c)
                dZ[(i64)b * lddz + c] = inv_batch * (exp(z[c] - mx) / s - (c == labels[b] ? 1.0 : 0.0));
    }
    *loss = inv_batch * total;
}

/* ---------------------------------------------------------------------------------
 * Weight and bias gradient (Sec. 1: Delta_W = Delta_Y X^T; Appendix A.2 derives it as
 * the sum over the batch of per-sample outer products). With a scale s (1 when the
 * mean is already inside Delta_Y, 1/B_global for a local partial):
 *   dW(m, k) = s * sum_b dY(m, b) X(k, b)        db(m) = s * sum_b dY(m, b)
 * The b-loop is outermost inside a row so the k-loop runs over contiguous memory; the
 * sum over b is still taken in ascending b for every (m, k).
 * memory: dY [B][lddy], X [B][ldx], dW [dout][lddw]
 * --------------------------------------------------------------------------------- */
void orc_weight_grad(int dout, int din, int B,
                     const double *dY, i64 lddy, const double *X, i64 ldx, double scale,
                     double *dW, i64 lddw, double *db)
{
#pragma omp parallel for schedule(static)
    for (int m = 0; m < dout; ++m) {
        double *row = dW + (i64)m * lddw;
        for (int k = 0; k < din; ++k) row[k] = 0.0;
        double sb = 0.0;
        for (int b = 0; b < B; ++b) {
            double g = dY[(i64)b * lddy + m];
            sb += g;
            const double *xr = X + (i64)b * ldx;
            for (int k = 0; k < din; ++k) row[k] += g * xr[k];
        }
        for (int k = 0; k < din; ++k) row[k] *= scale;
        if (db) db[m] = scale * sb;
    }
}

/* ---------------------------------------------------------------------------------
 * Activation gradient (Sec. 1 and Appendix A.2: Delta_X = W^T Delta_Y, column by column):
 *   dX(k, b) = sum_m W(m, k) dY(m, b)
 * The m-loop is outside the k-loop so both run over contiguous memory; the sum over m
 * is taken in ascending m for every (k, b).
 * memory: W [dout][ldw], dY [B][lddy], dX [B][lddx]
 * --------------------------------------------------------------------------------- */
void orc_input_grad(int dout, int din, int B,
                    const double *W, i64 ldw, const double *dY, i64 lddy,
                    double *dX, i64 lddx)
{
#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        double *out = dX + (i64)b * lddx;
        for (int k = 0; k < din; ++k) out[k] = 0.0;
        for (int m = 0; m < dout; ++m) {
            double g = dY[(i64)b * lddy + m];
            const double *wr = W + (i64)m * ldw;
            for (int k = 0; k < din; ++k) out[k] += wr[k] * g;
        }
    }
}

/* Chain rule through f = max(0, .): Delta_{Y_{i-1}} = Delta_{X_i} * f'(Y_{i-1}), with
 * f'(y) = [y > 0] (so f'(0) = 0). Y_{i-1} > 0 exactly where X_i = f(Y_{i-1}) > 0, so the
 * mask is read from the stored activation X_i. memory: dX [B][lddx], Xf [B][ldxf] */
void orc_relu_mask(int din, int B, double *dX, i64 lddx, const double *Xf, i64 ldxf)
{
    for (int b = 0; b < B; ++b)
        for (int k = 0; k < din; ++k)
            if (!(Xf[(i64)b * ldxf + k] > 0.0)) dX[(i64)b * lddx + k] = 0.0;
}

/* Mini-batch SGD, Eq. (1): w <- w - eta * g, where g is the mini-batch mean gradient. */
void orc_sgd(double *w, const double *g, i64 n, double eta)
{
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i) w[i] = w[i] - eta * g[i];
}

/* ---------------------------------------------------------------------------------
 * 3x3 stride-1 convolution on one spatial tile whose 1-pixel halo is already in place
 * (Sec. 2.2, domain parallelism: each process convolves its part of the image after
 * the boundary rows/columns have been exchanged; Sec. 2.1 for the layer and Eq. (2)
 * for its sizes). Cross-correlation, channels-last:
 *   x_pad [N][H+2][W+2][Ci], w [Co][3][3][Ci], y [N][H][W][Co]
 *   y(n,h,w,o)  = sum_{r,s,c} w(o,r,s,c) x_pad(n, h+r, w+s, c)
 * --------------------------------------------------------------------------------- */
void orc_conv3x3_fwd(int N, int H, int W, int Ci, int Co,
                     const double *xp, const double *wt, double *y)
{
    const i64 Wp = W + 2, Hp = H + 2;
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int h = 0; h < H; ++h)
            for (int w = 0; w < W; ++w)
                for (int o = 0; o < Co; ++o) {
                    double s = 0.0;
                    for (int r = 0; r < 3; ++r)
                        for (int q = 0; q < 3; ++q) {
                            const double *xv = xp + (((i64)n * Hp + h + r) * Wp + w + q) * Ci;
                            const double *wv = wt + (((i64)o * 3 + r) * 3 + q) * Ci;
                            for (int c = 0; c < Ci; ++c) s += wv[c] * xv[c];
                        }
                    y[(((i64)n * H + h) * W + w) * Co + o] = s;
                }
}

/* Input gradient of the tile. The output-gradient tile arrives with its own 1-pixel
 * halo from the neighbouring tiles (the second, output-side halo term of Eq. (7)):
 *   dy_pad [N][H+2][W+2][Co], dy_pad(n, i, j) = dy(n, i-1, j-1)
 *   dx(n,h,w,c) = sum_{r,s,o} w(o,r,s,c) dy(n, h-r+1, w-s+1, o)
 *               = sum_{r,s,o} w(o,r,s,c) dy_pad(n, h+2-r, w+2-s, o)      dx [N][H][W][Ci] */
void orc_conv3x3_dgrad(int N, int H, int W, int Ci, int Co,
                       const double *dyp, const double *wt, double *dx)
{
    const i64 Wp = W + 2, Hp = H + 2;
    /* All Ci outputs of one pixel are accumulated side by side (c innermost, so the
     * weight rows are read contiguously); each output still sums over r, then q, then o
     * in ascending order. */
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int h = 0; h < H; ++h)
            for (int w = 0; w < W; ++w) {
                double *s = dx + (((i64)n * H + h) * W + w) * Ci;
                for (int c = 0; c < Ci; ++c) s[c] = 0.0;
                for (int r = 0; r < 3; ++r)
                    for (int q = 0; q < 3; ++q) {
                        const double *g = dyp + (((i64)n * Hp + h + 2 - r) * Wp + w + 2 - q) * Co;
                        for (int o = 0; o < Co; ++o) {
                            const double *wv = wt + (((i64)o * 3 + r) * 3 + q) * Ci;
                            for (int c = 0; c < Ci; ++c) s[c] += wv[c] * g[o];
                        }
                    }
            }
}

/* Weight gradient of the tile: the tile's share of the sum over all pixels that the
 * all-reduce of Eq. (7) (third term) completes across processes.
 *   dw(o,r,s,c) = sum_{n,h,w} dy(n,h,w,o) x_pad(n, h+r, w+s, c),  dy = interior of dy_pad */
void orc_conv3x3_wgrad(int N, int H, int W, int Ci, int Co,
                       const double *xp, const double *dyp, double *dw)
{
    const i64 Wp = W + 2, Hp = H + 2;
#pragma omp parallel for schedule(static)
    for (int o = 0; o < Co; ++o) {
        double *acc = dw + (i64)o * 9 * Ci;
        for (i64 t = 0; t < 9 * (i64)Ci; ++t) acc[t] = 0.0;
        for (int n = 0; n < N; ++n)
            for (int h = 0; h < H; ++h)
                for (int w = 0; w < W; ++w) {
                    double g = dyp[(((i64)n * Hp + h + 1) * Wp + w + 1) * Co + o];
                    for (int r = 0; r < 3; ++r)
                        for (int q = 0; q < 3; ++q) {
                            const double *xv = xp + (((i64)n * Hp + h + r) * Wp + w + q) * Ci;
                            double *a = acc + (r * 3 + q) * (i64)Ci;
                            for (int c = 0; c < Ci; ++c) a[c] += g * xv[c];
                        }
                }
    }
}

/* The same three conv sums evaluated only at a list of flat output indices, for
 * spot checks of full-size tiles (same definitions as above, one output at a time). */
void orc_conv3x3_fwd_at(int N, int H, int W, int Ci, int Co, const double *xp, const double *wt,
                        const i64 *idx, i64 n_idx, double *out)
{
    const i64 Wp = W + 2, Hp = H + 2;
    (void)N;
#pragma omp parallel for schedule(static)
    for (i64 t = 0; t < n_idx; ++t) {
        i64 f = idx[t];
        int o = (int)(f % Co); f /= Co;
        int w = (int)(f % W); f /= W;
        int h = (int)(f % H); int n = (int)(f / H);
        double s = 0.0;
        for (int r = 0; r < 3; ++r)
            for (int q = 0; q < 3; ++q) {
                const double *xv = xp + (((i64)n * Hp + h + r) * Wp + w + q) * Ci;
                const double *wv = wt + (((i64)o * 3 + r) * 3 + q) * Ci;
                for (int c = 0; c < Ci; ++c) s += wv[c] * xv[c];
            }
        out[t] = s;
    }
}

void orc_conv3x3_dgrad_at(int N, int H, int W, int Ci, int Co, const double *dyp, const double *wt,
                          const i64 *idx, i64 n_idx, double *out)
{
    const i64 Wp = W + 2, Hp = H + 2;
    (void)N;
#pragma omp parallel for schedule(static)
    for (i64 t = 0; t < n_idx; ++t) {
        i64 f = idx[t];
        int c = (int)(f % Ci); f /= Ci;
        int w = (int)(f % W); f /= W;
        int h = (int)(f % H); int n = (int)(f / H);
        double s = 0.0;
        for (int r = 0; r < 3; ++r)
            for (int q = 0; q < 3; ++q) {
                const double *g = dyp + (((i64)n * Hp + h + 2 - r) * Wp + w + 2 - q) * Co;
                for (int o = 0; o < Co; ++o) s += wt[(((i64)o * 3 + r) * 3 + q) * Ci + c] * g[o];
            }
        out[t] = s;
    }
}

void orc_conv3x3_wgrad_at(int N, int H, int W, int Ci, int Co, const double *xp, const double *dyp,
                          const i64 *idx, i64 n_idx, double *out)
{
    const i64 Wp = W + 2, Hp = H + 2;
#pragma omp parallel for schedule(static)
    for (i64 t = 0; t < n_idx; ++t) {
        i64 f = idx[t];
        int c = (int)(f % Ci); f /= Ci;
        int q = (int)(f % 3); f /= 3;
        int r = (int)(f % 3); int o = (int)(f / 3);
        double s = 0.0;
        for (int n = 0; n < N; ++n)
            for (int h = 0; h < H; ++h)
                for (int w = 0; w < W; ++w)
                    s += dyp[(((i64)n * Hp + h + 1) * Wp + w + 1) * Co + o] *
                         xp[(((i64)n * Hp + h + r) * Wp + w + q) * Ci + c];
        out[t] = s;
    }
}
