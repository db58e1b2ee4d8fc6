// The lean split-K reduce of the wide-batch and tiled products as a per-thread device
// function (csrc/gemm.hip launches it; the large-tile update kernel, csrc/dw_wide.hip, runs
// a product's reduce after its tiles): outputs m .. m+7 of column n, the splits added in split
// order, then alpha, bias, ReLU and mask as the epilogue asks, stored as OUT_BF16 says.
#pragma once

#include "common.h"

namespace imbd {

__device__ __forceinline__ uint32_t lean_pack_bf16x2(float a, float b) {
  return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}

template <bool OUT_BF16, bool MASK>
__device__ __forceinline__ void lean_reduce_item(const LeanReduceArgs &g, int n, int m) {
  const Epilogue &e = g.epi;
  const float *p0 = g.partial + (int64_t)n * g.ldp + m;
  f32x4 a0 = *reinterpret_cast<const f32x4 *>(p0);
  f32x4 a1 = *reinterpret_cast<const f32x4 *>(p0 + 4);
  for (int s0 = 1; s0 < g.splits; s0 += 4) {
    f32x4 q0[4], q1[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (s0 + u < g.splits) {
        const float *p = p0 + (int64_t)(s0 + u) * g.sstride;
        q0[u] = *reinterpret_cast<const f32x4 *>(p);
        q1[u] = *reinterpret_cast<const f32x4 *>(p + 4);
      }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (s0 + u < g.splits) {
        a0 += q0[u];
        a1 += q1[u];
      }
  }
  float x[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
  if (e.bias) {
    const f32x4 b0 = *reinterpret_cast<const f32x4 *>(e.bias + m);
    const f32x4 b1 = *reinterpret_cast<const f32x4 *>(e.bias + m + 4);
    const float bb[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = e.alpha * x[i] + bb[i];
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = e.alpha * x[i];
  }
  if (e.relu) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = x[i] > 0.f ? x[i] : 0.f;
  }
  if constexpr (MASK) {
    // mask element type follows the activation type (bf16 here, fp32 for fp32 networks)
    const int64_t off = (int64_t)n * e.ldmask + m;
    if (e.mask_dtype == IMBD_BF16) {
      const u32x4 mk = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(e.mask) + off);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint16_t h = (uint16_t)((mk[i >> 1] >> (16 * (i & 1))) & 0xffffu);
        if (!(bf16_to_f32(h) > 0.f)) x[i] = 0.f;
      }
    } else {
      const f32x4 m0 = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(e.mask) + off);
      const f32x4 m1 = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(e.mask) + off + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (!(m0[i] > 0.f)) x[i] = 0.f;
        if (!(m1[i] > 0.f)) x[i + 4] = 0.f;
      }
    }
  }
  if constexpr (OUT_BF16) {
    u32x4 pk;
#pragma unroll
    for (int i = 0; i < 4; ++i) pk[i] = lean_pack_bf16x2(x[2 * i], x[2 * i + 1]);
    *reinterpret_cast<u32x4 *>(reinterpret_cast<uint16_t *>(e.out) + (int64_t)n * e.ldo + m) = pk;
  } else {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    *reinterpret_cast<f32x4 *>(o) = f32x4{x[0], x[1], x[2], x[3]};
    *reinterpret_cast<f32x4 *>(o + 4) = f32x4{x[4], x[5], x[6], x[7]};
  }
}

}  // namespace imbd
