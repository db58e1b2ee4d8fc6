// Bandwidth-bound kernels of the hot path: softmax cross-entropy at the top of the
// network, the bias gradient, the mini-batch SGD update of Eq. (1) and the fp32 -> bf16
// conversion of master weights. Wave64 throughout; every reduction runs in a fixed order
// so repeated calls give identical bits.

#include "common.h"
#include "loss_mean.h"

namespace imbd {

namespace {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One wave per sample row: row maximum, sum of exp(z - max), per-sample loss
// lse - z[label] and the gradient inv_batch * (softmax - onehot); a label outside [0, C)
// gives a NaN loss and a NaN gradient row (no one-hot to subtract). NPL > 0 keeps the row in
// registers (NPL values per lane, C <= 64*NPL) so the logits are read once; NPL == 0 reads
// them from memory in each pass (any C).
template <int NPL>
__global__ void __launch_bounds__(256)
    softmax_xent_rows(int B, int C, const float *__restrict__ Z, int64_t ldz,
                      const int32_t *__restrict__ labels, float inv_batch,
                      float *__restrict__ row_loss, void *__restrict__ dz, int64_t lddz, int dz_bf16) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= B) return;
  const float *z = Z + (int64_t)row * ldz;
  const int lab = labels[row];
  const bool ok = lab >= 0 && lab < C;
  float mx = -INFINITY, s = 0.f;
  float v[NPL > 0 ? NPL : 1];
  if constexpr (NPL > 0) {
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int c = lane + 64 * j;
      v[j] = c < C ? z[c] : -INFINITY;
      mx = fmaxf(mx, v[j]);
    }
    mx = wave_max(mx);
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      v[j] = expf(v[j] - mx);   // exp(-inf) = 0 for the padding
      s += v[j];
    }
  } else {
    for (int c = lane; c < C; c += 64) mx = fmaxf(mx, z[c]);
    mx = wave_max(mx);
    for (int c = lane; c < C; c += 64) s += expf(z[c] - mx);
  }
  s = wave_sum(s);
  if (lane == 0) row_loss[row] = ok ? (mx + logf(s) - z[lab]) : __builtin_nanf("");
  if (!dz) return;
  const float inv_s = 1.0f / s;
  if constexpr (NPL > 0) {
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int c = lane + 64 * j;
      if (c < C) {
        const float g = ok ? inv_batch * (v[j] * inv_s - (c == lab ? 1.0f : 0.0f)) : __builtin_nanf("");
        if (dz_bf16)
          reinterpret_cast<uint16_t *>(dz)[(int64_t)row * lddz + c] = f32_to_bf16(g);
        else
          reinterpret_cast<float *>(dz)[(int64_t)row * lddz + c] = g;
      }
    }
  } else {
    for (int c = lane; c < C; c += 64) {
      const float g = ok ? inv_batch * (expf(z[c] - mx) * inv_s - (c == lab ? 1.0f : 0.0f)) : __builtin_nanf("");
      if (dz_bf16)
        reinterpret_cast<uint16_t *>(dz)[(int64_t)row * lddz + c] = f32_to_bf16(g);
      else
        reinterpret_cast<float *>(dz)[(int64_t)row * lddz + c] = g;
    }
  }
}

// loss = inv_batch * sum_b row_loss[b], one workgroup (the fixed order of block_loss_mean).
__global__ void __launch_bounds__(256)
    loss_mean(int B, const float *__restrict__ row_loss, float inv_batch, float *__restrict__ loss) {
  __shared__ float part[256];
  block_loss_mean(B, row_loss, inv_batch, loss, part);
}

// db[m] = alpha * sum_b dy[b][m]: 64 columns per workgroup, each column's rows split in
// 4 contiguous slices summed in ascending b, the slice sums added in slice order;
// optionally bias[m] -= lr * db[m].
template <typename T>
__global__ void __launch_bounds__(256)
    bias_grad_kernel(int M, int B, const T *__restrict__ dy, int64_t lddy, float alpha,
                     float *__restrict__ db_out, float *__restrict__ bias, float lr) {
  __shared__ float part[4][64];
  const int col = threadIdx.x & 63, slice = threadIdx.x >> 6;
  const int m = blockIdx.x * 64 + col;
  const int per = (B + 3) / 4;
  const int b0 = slice * per, b1 = min(B, b0 + per);
  float s = 0.f;
  if (m < M) {
    for (int b = b0; b < b1; ++b) {
      const T v = dy[(int64_t)b * lddy + m];
      if constexpr (sizeof(T) == 2) s += bf16_to_f32(v);
      else s += v;
    }
  }
  part[slice][col] = s;
  __syncthreads();
  if (slice == 0 && m < M) {
    const float g = alpha * (((part[0][col] + part[1][col]) + part[2][col]) + part[3][col]);
    if (db_out) db_out[m] = g;
    if (bias) bias[m] = fmaf(-lr, g, bias[m]);
  }
}

// The same column sums for bf16 Delta_Y with 16-byte rows chunks (8 columns): 64 columns per
// workgroup, thread t sums chunk t%8 over the rows r = t/8 + 32i in ascending order (eight
// loads in flight per batch), then the 32 row phases are added in phase order.
__global__ void __launch_bounds__(256)
    bias_grad_wide(int M, int B, const uint16_t *__restrict__ dy, int64_t lddy, float alpha,
                   float *__restrict__ db_out, float *__restrict__ bias, float lr) {
  __shared__ float part[32][64 + 4];
  const int j = threadIdx.x & 7, q = threadIdx.x >> 3;
  const int m0 = blockIdx.x * 64 + 8 * j;
  const bool live = m0 < M;  // M % 8 == 0: a chunk is wholly in or out
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r0 = q; r0 < B; r0 += 32 * 8) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = r0 + 32 * u;
      v[u] = live && r < B ? *reinterpret_cast<const u32x4 *>(dy + (int64_t)r * lddy + m0) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[2 * e] += bf16_to_f32((uint16_t)(v[u][e] & 0xffffu));
        s[2 * e + 1] += bf16_to_f32((uint16_t)(v[u][e] >> 16));
      }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[q][8 * j + e] = s[e];
  __syncthreads();
  if (threadIdx.x < 64) {
    const int m = blockIdx.x * 64 + threadIdx.x;
    float t = 0.f;
    for (int k = 0; k < 32; ++k) t += part[k][threadIdx.x];
    if (m < M) {
      const float g = alpha * t;
      if (db_out) db_out[m] = g;
      if (bias) bias[m] = fmaf(-lr, g, bias[m]);
    }
  }
}

// w <- w - step * g (one fp32 rounding), optional bf16 copy. Four elements per thread.
__global__ void __launch_bounds__(256)
    sgd_kernel(float *__restrict__ w, uint16_t *__restrict__ w16, const float *__restrict__ g,
               int64_t n, float step) {
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    f32x4 wv = reinterpret_cast<const f32x4 *>(w)[i];
    const f32x4 gv = reinterpret_cast<const f32x4 *>(g)[i];
    f32x4 nv;
#pragma unroll
    for (int e = 0; e < 4; ++e) nv[e] = fmaf(-step, gv[e], wv[e]);
    reinterpret_cast<f32x4 *>(w)[i] = nv;
    if (w16) {
      u32x2 pk;
      pk[0] = (uint32_t)f32_to_bf16(nv[0]) | ((uint32_t)f32_to_bf16(nv[1]) << 16);
      pk[1] = (uint32_t)f32_to_bf16(nv[2]) | ((uint32_t)f32_to_bf16(nv[3]) << 16);
      reinterpret_cast<u32x2 *>(w16)[i] = pk;
    }
  }
  // tail
  const int64_t t = (n4 << 2) + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t < n && (int64_t)blockIdx.x * 256 + threadIdx.x < 4) {
    const float nw = fmaf(-step, g[t], w[t]);
    w[t] = nw;
    if (w16) w16[t] = f32_to_bf16(nw);
  }
}

// Scalar fallback for buffers that are not 16-byte aligned.
__global__ void __launch_bounds__(256)
    sgd_scalar_kernel(float *__restrict__ w, uint16_t *__restrict__ w16, const float *__restrict__ g,
                      int64_t n, float step) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float nw = fmaf(-step, g[i], w[i]);
    w[i] = nw;
    if (w16) w16[i] = f32_to_bf16(nw);
  }
}

__global__ void __launch_bounds__(256)
    cast_kernel(const float *__restrict__ src, uint16_t *__restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = f32_to_bf16(src[i]);
}

int grid_for(int64_t work, int per_block) {
  int64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > 8192) b = 8192;
  return (int)b;
}

}  // namespace

int run_softmax_xent(int B, int C, const float *logits, int64_t ldz, const int32_t *labels,
                     float inv_batch, float *loss, float *row_loss, void *dz, int64_t lddz,
                     int dz_dtype, hipStream_t s, int layer, bool mean) {
  if (B <= 0) return IMBD_OK;
  {
    LaunchTimer t(IMBD_K_SOFTMAX, layer, s);
    const int bf = dz_dtype == IMBD_BF16 ? 1 : 0;
    const dim3 grid((B + 3) / 4);
    if (C <= 64 * 4)
      hipLaunchKernelGGL(softmax_xent_rows<4>, grid, dim3(256), 0, s, B, C, logits, ldz, labels, inv_batch,
                         row_loss, dz, lddz, bf);
    else if (C <= 64 * 16)
      hipLaunchKernelGGL(softmax_xent_rows<16>, grid, dim3(256), 0, s, B, C, logits, ldz, labels, inv_batch,
                         row_loss, dz, lddz, bf);
    else
      hipLaunchKernelGGL(softmax_xent_rows<0>, grid, dim3(256), 0, s, B, C, logits, ldz, labels, inv_batch,
                         row_loss, dz, lddz, bf);
  }
  int rc = check_launch("softmax_xent_rows");
  if (rc || !mean) return rc;
  return run_loss_mean(B, row_loss, inv_batch, loss, s);
}

int run_loss_mean(int B, const float *row_loss, float inv_batch, float *loss, hipStream_t s) {
  if (B <= 0) return IMBD_OK;
  hipLaunchKernelGGL(loss_mean, dim3(1), dim3(256), 0, s, B, row_loss, inv_batch, loss);
  return check_launch("loss_mean");
}

int run_bias_grad(int dtype, int M, int B, const void *dy, int64_t lddy, float alpha,
                  float *db_out, float *bias_sgd, float lr, hipStream_t s, int layer) {
  if (M <= 0) return IMBD_OK;
  LaunchTimer t(IMBD_K_BIAS, layer, s);
  if (dtype == IMBD_BF16 && M % 8 == 0 && lddy % 8 == 0 && (uintptr_t)dy % 16 == 0)
    hipLaunchKernelGGL(bias_grad_wide, dim3((M + 63) / 64), dim3(256), 0, s, M, B,
                       reinterpret_cast<const uint16_t *>(dy), lddy, alpha, db_out, bias_sgd, lr);
  else if (dtype == IMBD_BF16)
    hipLaunchKernelGGL(bias_grad_kernel<uint16_t>, dim3((M + 63) / 64), dim3(256), 0, s, M, B,
                       reinterpret_cast<const uint16_t *>(dy), lddy, alpha, db_out, bias_sgd, lr);
  else
    hipLaunchKernelGGL(bias_grad_kernel<float>, dim3((M + 63) / 64), dim3(256), 0, s, M, B,
                       reinterpret_cast<const float *>(dy), lddy, alpha, db_out, bias_sgd, lr);
  return check_launch("bias_grad");
}

int run_sgd(float *w, uint16_t *w16, const float *g, int64_t n, float step, hipStream_t s,
            int layer) {
  if (n <= 0) return IMBD_OK;
  const bool vec = ((uintptr_t)w % 16 == 0) && ((uintptr_t)g % 16 == 0) &&
                   (w16 == nullptr || (uintptr_t)w16 % 8 == 0);
  LaunchTimer t(IMBD_K_SGD, layer, s);
  if (vec)
    hipLaunchKernelGGL(sgd_kernel, dim3(grid_for((n >> 2) > 0 ? (n >> 2) : 1, 256 * 4)), dim3(256), 0,
                       s, w, w16, g, n, step);
  else
    hipLaunchKernelGGL(sgd_scalar_kernel, dim3(grid_for(n, 256 * 4)), dim3(256), 0, s, w, w16, g, n,
                       step);
  return check_launch("sgd");
}

__global__ void __launch_bounds__(256)
    repack_bf16_kernel(const uint16_t *__restrict__ src, int64_t ld_src, int rows, int cols,
                       uint16_t *__restrict__ dst, int64_t ld_dst) {
  const int64_t total = (int64_t)rows * ld_dst;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int64_t r = t / ld_dst, c = t - r * ld_dst;
    dst[t] = c < cols ? src[r * ld_src + c] : (uint16_t)0;
  }
}

int run_repack_bf16(const uint16_t *src, int64_t ld_src, int rows, int cols, uint16_t *dst, int64_t ld_dst,
                    hipStream_t s) {
  const int64_t total = (int64_t)rows * ld_dst;
  if (total <= 0) return IMBD_OK;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(repack_bf16_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, s, src, ld_src,
                     rows, cols, dst, ld_dst);
  return check_launch("repack_bf16");
}

int run_cast(const float *src, uint16_t *dst, int64_t n, hipStream_t s) {
  if (n <= 0) return IMBD_OK;
  LaunchTimer t(IMBD_K_CAST, 0, s);
  hipLaunchKernelGGL(cast_kernel, dim3(grid_for(n, 256 * 4)), dim3(256), 0, s, src, dst, n);
  return check_launch("cast");
}

}  // namespace imbd
