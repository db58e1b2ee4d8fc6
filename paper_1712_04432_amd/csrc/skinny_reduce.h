// The split-K reduce of the skinny-batch product kernel (csrc/skinny.hip) as a per-thread
// device function, so that a later launch can carry it (the fused update kernel's MMA
// waves run a layer's Delta_X reduce once their products are done, csrc/dw_sgd.hip).
#pragma once

#include "cdna4.h"

namespace imbd {

// Item tl of the reduce: adds the splits' partials and applies the store epilogue:
// out(m, n) = [mask(m, n) > 0] * relu?(alpha * sum + bias[m]). Eight consecutive m of one
// sample per group of LANES threads; VEC: every access is whole and aligned (checked on
// the host). LANES = 1: one thread adds the splits in split order (the same order and
// arithmetic as the split-K reduce of the tiled products). LANES = 4 (more than four
// splits, where one thread would wait on its loads round after round): lane j adds splits
// j, j+4, j+8, ... in that order, and the four sums are combined as (s0 + s1) + (s2 + s3)
// by lane exchanges; each exchange adds the same two values on both lanes, so every lane
// holds the same bits and the result is the same on every run.
template <bool VEC, int LANES>
__device__ __forceinline__ void sk_reduce_item(const SkReduceArgs &g, int64_t tl) {
  const int64_t t = tl / LANES;
  const int j = (int)(tl - t * LANES);
  const int tile = (int)(t / ((int64_t)g.N * 8));
  const int r = (int)(t - (int64_t)tile * g.N * 8);
  const int n = r >> 3, m = tile * 64 + 8 * (r & 7);
  if (n >= g.N || m >= g.M) return;  // the same for all LANES lanes of a group
  const Epilogue &e = g.epi;
  const float *p = g.partial + (int64_t)tile * g.tpitch + n * 64 + (m & 63);
  f32x4 a0 = *reinterpret_cast<const f32x4 *>(p + (int64_t)j * g.sstride);
  f32x4 a1 = *reinterpret_cast<const f32x4 *>(p + (int64_t)j * g.sstride + 4);
  for (int s0 = j + LANES; s0 < g.splits; s0 += 4 * LANES) {
    f32x4 q0[4], q1[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (s0 + u * LANES < g.splits) {
        const float *q = p + (int64_t)(s0 + u * LANES) * g.sstride;
        q0[u] = *reinterpret_cast<const f32x4 *>(q);
        q1[u] = *reinterpret_cast<const f32x4 *>(q + 4);
      }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (s0 + u * LANES < g.splits) {
        a0 += q0[u];
        a1 += q1[u];
      }
  }
  if constexpr (LANES > 1) {
#pragma unroll
    for (int d = 1; d < LANES; d <<= 1)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a0[i] += __shfl_xor(a0[i], d);
        a1[i] += __shfl_xor(a1[i], d);
      }
    if (j != 0) return;
  }
  const float v[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
  const int cnt = VEC ? 8 : min(8, g.M - m);
  float x[8];
  if constexpr (VEC) {
    // bias, mask and output rows are whole and aligned (checked on the host)
    float bb[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (e.bias) {
      const f32x4 b0 = *reinterpret_cast<const f32x4 *>(e.bias + m);
      const f32x4 b1 = *reinterpret_cast<const f32x4 *>(e.bias + m + 4);
      bb[0] = b0[0]; bb[1] = b0[1]; bb[2] = b0[2]; bb[3] = b0[3];
      bb[4] = b1[0]; bb[5] = b1[1]; bb[6] = b1[2]; bb[7] = b1[3];
    }
    bool keep[8] = {true, true, true, true, true, true, true, true};
    if (e.mask) {
      const int64_t off = (int64_t)n * e.ldmask + m;
      if (e.mask_dtype == IMBD_BF16) {
        const u32x4 mk = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(e.mask) + off);
#pragma unroll
        for (int i = 0; i < 8; ++i) keep[i] = bf16_to_f32((uint16_t)((mk[i >> 1] >> (16 * (i & 1))) & 0xffffu)) > 0.0f;
      } else {
        const f32x4 m0 = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(e.mask) + off);
        const f32x4 m1 = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(e.mask) + off + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          keep[i] = m0[i] > 0.0f;
          keep[i + 4] = m1[i] > 0.0f;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float y = e.alpha * v[i] + bb[i];
      if (e.relu) y = y > 0.0f ? y : 0.0f;
      x[i] = keep[i] ? y : 0.0f;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < cnt) {
        float y = e.alpha * v[i] + (e.bias ? e.bias[m + i] : 0.0f);
        if (e.relu) y = y > 0.0f ? y : 0.0f;
        if (e.mask) {
          const int64_t off = (int64_t)n * e.ldmask + m + i;
          const float mk = e.mask_dtype == IMBD_BF16 ? bf16_to_f32(reinterpret_cast<const uint16_t *>(e.mask)[off])
                                                     : reinterpret_cast<const float *>(e.mask)[off];
          if (!(mk > 0.0f)) y = 0.0f;
        }
        x[i] = y;
      }
    }
  }
  if (e.out_dtype == IMBD_BF16) {
    uint16_t *o = reinterpret_cast<uint16_t *>(e.out) + (int64_t)n * e.ldo + m;
    if constexpr (VEC) {
      u32x4 pk;
#pragma unroll
      for (int i = 0; i < 4; ++i) pk[i] = (uint32_t)f32_to_bf16(x[2 * i]) | ((uint32_t)f32_to_bf16(x[2 * i + 1]) << 16);
      *reinterpret_cast<u32x4 *>(o) = pk;
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (i < cnt) o[i] = f32_to_bf16(x[i]);
    }
  } else {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    if constexpr (VEC) {
      *reinterpret_cast<f32x4 *>(o) = f32x4{x[0], x[1], x[2], x[3]};
      *reinterpret_cast<f32x4 *>(o + 4) = f32x4{x[4], x[5], x[6], x[7]};
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (i < cnt) o[i] = x[i];
    }
  }
}

}  // namespace imbd
