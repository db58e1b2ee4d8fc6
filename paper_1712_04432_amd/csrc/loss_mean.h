// Batch mean of the per-sample losses (Sec. 1: the mini-batch loss is the mean of its
// samples' losses), shared by the standalone kernel and the launches that carry it as a
// side job.
#pragma once

#include <hip/hip_runtime.h>

namespace imbd {

// loss = inv_batch * sum_b row_loss[b] by the first 256 threads of a workgroup of at least
// 256, in a fixed order: each thread sums a strided subset in ascending order, then a fixed
// tree over the threads. part: 256 floats of LDS. Every thread of the workgroup must call
// it (the others only meet the barriers).
__device__ inline void block_loss_mean(int B, const float *__restrict__ row_loss, float inv_batch,
                                       float *__restrict__ loss, float *part) {
  const int t = (int)threadIdx.x;
  if (t < 256) {
    float s = 0.f;
    for (int b = t; b < B; b += 256) s += row_loss[b];
    part[t] = s;
  }
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) part[t] += part[t + w];
    __syncthreads();
  }
  if (t == 0) *loss = inv_batch * part[0];
}

}  // namespace imbd
