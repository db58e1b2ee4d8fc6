// Forward and activation-gradient products of a fully connected layer for a batch of at
// most 256 samples, bf16 operands (Sec. 1: Y = W X and Delta_X = W^T Delta_Y; App. A for
// their block forms, which are the same products on a process's blocks).
//
// With B <= 256 these products stream the weight matrix once from HBM and do 2*B flops
// per weight element. A workgroup owns a 64-row block of W against the whole batch
// (up to 256 samples) over one K-range; K is split so that the grid fills the chip, and
// the splits' fp32 partials are added in split order by the split-K reduce, which also
// applies the bias/ReLU or mask epilogue. Both operands travel through LDS in 64-k slabs
// written by buffer loads that go straight to LDS (no registers; out-of-range lanes
// land as zeros), each load instruction covering whole 128-byte lines (8 rows x 128 B):
// MFMA-layout loads into registers touch 16 half-lines per instruction and move less
// than half as many bytes per clock from L2. Eight waves in three groups, each with its
// own memory counter so that no group waits on another's loads:
//  * waves 4-5 stream W through an eight-slot ring (up to six slabs in flight from HBM);
//  * waves 6-7 stream the activation slab (L2 hits: the workgroups of one K-range run on
//    one XCD) through a three-slot ring;
//  * waves 0-3 read MFMA fragments from LDS: 16-byte reads, or for W used transposed
//    (Delta_X) the gfx950 LDS transpose read, and accumulate the tile in registers.
// Every group meets at one barrier per slab. Rows sit in LDS with their 16-byte chunks
// XOR-swizzled so that each fragment read touches every bank once.

#include <stdlib.h>

#include "cdna4.h"
#include "dw_wide_body.h"
#include "local_pair.h"
#include "loss_mean.h"
#include "skinny_reduce.h"

namespace imbd {
namespace {

struct SkArgs {
  const uint16_t *A;  // W: [M][lda] (k contiguous) or [K][lda] (m contiguous, A_TR)
  const uint16_t *B;  // activations: [N][ldb], k contiguous
  int64_t lda, ldb;
  int M, N, K;
  int k_split, splits, tiles_m, tiles_n;  // a workgroup: 64 rows x 64*NB samples x one K-range
  float *partial;     // [split][tile][N][64]: one contiguous block per (split, row tile)
  int64_t tpitch, sstride;
  // splits == 1 and fused: the store epilogue applied here instead of writing partials
  int fused;
  float alpha;
  const float *bias;        // [M] or null
  int relu;
  const uint16_t *mask;     // bf16 [N][ldmask] or null: zero where !(mask > 0)
  int64_t ldmask;
  void *out;                // [N][ldo], bf16 (out_bf16) or fp32
  int64_t ldo;
  int out_bf16;
  int vec;                  // out, mask and bias rows 8-byte (bf16) / 16-byte (fp32) aligned at every 4th m
  // side job in one extra workgroup (the last): *aux_loss = aux_scale * sum of aux_rows
  const float *aux_rows;
  float *aux_loss;
  int aux_n;
  float aux_scale;
  // B's rows only 4-byte aligned (pitch and base): loaded in 4-byte pieces (NB <= 2), K even
  int b_dw4;
};

// Partial-sum layout: each workgroup's 64 x N tile is one contiguous block (a tile pitch
// of N*64 floats plus 64, a split pitch off powers of two), so the write-out and the
// reduce stream whole blocks.
inline int64_t sk_tile_pitch(int N) { return (int64_t)N * 64 + 64; }
inline int64_t sk_split_pitch(int M, int N) { return (int64_t)((M + 63) / 64) * sk_tile_pitch(N) + 1088; }

constexpr int CPOL_SC1 = 16;              // cache-policy operand of the raw buffer builtins: sc1
constexpr int SK_BM = 64;                 // rows of the output (W) per workgroup
constexpr int SK_KS = 64;                 // k per slab (128 bytes per row)
constexpr int SK_NW = 8;                  // W ring slots
constexpr int SK_NX = 3;                  // activation ring slots
constexpr int SK_WSLOT = 64 * 128;        // 8 KB: 64 rows (KC) or 64 k-rows (TR) x 128 B

// 16-byte chunk position of chunk c in row r of a slab read with 16-byte fragment reads
// (16 consecutive rows, one chunk): XOR with the row's low three bits. Measured on gfx950
// (SQ_LDS_BANK_CONFLICT) to be conflict-free for this read, at 4 LDS cycles per 1 KB.
__device__ __forceinline__ int swz_kc(int r) { return r & 7; }
// ... and of a W slab read with the transpose read (k-rows of 64 m-values); also measured
// conflict-free (2 LDS cycles per 512 B).
__device__ __forceinline__ int swz_tr(int r) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1); }

// Bytes of LDS a workgroup of the kernel uses.
template <int NB>
constexpr int sk_lds_bytes() { return SK_NX * 64 * NB * 128 + SK_NW * SK_WSLOT; }

// NB: the workgroup covers 64*NB samples; MMA wave w takes NB m-blocks and four
// 16-sample blocks. One workgroup's tile: bid is its index in the launch (the product's
// workgroups come first), smem its LDS (sk_lds_bytes<NB>() bytes). A function of its own
// so that a launch can also run it beside another product's workgroups.
template <bool A_TR, int NB>
__device__ __forceinline__ void skinny_body(const SkArgs &a, char *smem, int bid) {
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int XROWS = 64 * NB;
  constexpr int XSLOT = XROWS * 128;
  constexpr int XRING = SK_NX * XSLOT;
  static_assert(XRING + SK_NW * SK_WSLOT == sk_lds_bytes<NB>(), "LDS size");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.tiles_m * a.tiles_n * a.splits;  // product workgroups (an extra one carries aux)
  if (a.aux_loss && bid == G) {
    block_loss_mean(a.aux_n, a.aux_rows, a.aux_scale, a.aux_loss, reinterpret_cast<float *>(smem));
    return;
  }
  int b = bid;
  // consecutive logical blocks on one XCD: the sample tiles of one row tile, then the row
  // tiles of one K-range
  if ((G & 7) == 0) b = (b & 7) * (G >> 3) + (b >> 3);
  const int nt = b % a.tiles_n, mk = b / a.tiles_n;
  const int split = mk / a.tiles_m, m0 = (mk - split * a.tiles_m) * SK_BM, n0 = nt * XROWS;
  const int klo = split * a.k_split, krange = min(a.K, klo + a.k_split) - klo;
  const int nsl = (krange + SK_KS - 1) / SK_KS;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t ldsx = lds0, ldsw = lds0 + XRING;

  if (wave >= 6) {
    // -------------------------------------------------- activation loaders (6, 7)
    // Slab S: rows 0..XROWS-1 of the batch, k = klo + 64S ..; wave xw fills the 1 KB
    // blocks 4NB*xw .. 4NB*xw + 4NB-1 of the slot (8 rows x 128 B each).
    const int xw = wave - 6;
    const i32x4 rb = buf_rsrc(a.B, (uint32_t)((int64_t)a.N * a.ldb * 2));
    const uint32_t dst0 = ldsx + (uint32_t)(4 * NB * xw * 1024);
    uint32_t slot = 0;  // ring slot of the next slab to issue
    // B's rows 4-byte aligned only (NB <= 2): each 16-byte chunk of the layout below comes
    // as four 4-byte loads. Instruction i of a 1 KB block fills its bytes 256i .. 256i + 255:
    // lane l loads dword l%4 of the chunk that lane 16i + l/4 loads in the 16-byte form
    // (rows of block q are those of block 0 plus 8q, with the same swizzle). A dword past
    // the K-range (K even) reads as zero.
    constexpr bool DW4_OK = 4 * 4 * NB * (SK_NX - 2) <= 63;  // the memory counter's range
    if (DW4_OK && a.b_dw4) {
      uint32_t b4[4];
      int k4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int L = 16 * i + (lane >> 2), d = lane & 3;
        const int r = 8 * (4 * NB * xw) + (L >> 3);
        const int c = (L & 7) ^ swz_kc(r);
        b4[i] = (uint32_t)(((int64_t)(n0 + r) * a.ldb + klo + 8 * c) * 2 + 4 * d);
        k4[i] = 8 * c + 2 * d;
      }
      const uint32_t qstep = (uint32_t)(8 * a.ldb * 2);
      auto issue4 = [&](int S) {
#pragma unroll
        for (int q = 0; q < 4 * NB; ++q)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool ok = S * SK_KS + k4[i] < krange;
            dma4(rb, ok ? b4[i] + (uint32_t)q * qstep + (uint32_t)S * 128u : OOB,
                 dst0 + slot + (uint32_t)(q * 1024 + 256 * i));
          }
        slot = slot + XSLOT == XRING ? 0u : slot + XSLOT;
      };
#pragma unroll
      for (int S = 0; S < SK_NX - 1; ++S) issue4(S);
      for (int S = 0; S < nsl; ++S) {
        vm_barrier<(DW4_OK ? 4 : 1) * 4 * NB * (SK_NX - 2)>();  // slab S landed: B_S
        issue4(S + SK_NX - 1);                                 // into the slot of S-1
      }
      vm_barrier<0>();
    } else {
      uint32_t base[4 * NB];
      int kof[4 * NB];
#pragma unroll
      for (int q = 0; q < 4 * NB; ++q) {
        const int r = 8 * (4 * NB * xw + q) + (lane >> 3);
        const int c = (lane & 7) ^ swz_kc(r);
        base[q] = (uint32_t)(((int64_t)(n0 + r) * a.ldb + klo + 8 * c) * 2);  // rows past N: out of range
        kof[q] = 8 * c;
      }
      auto issue = [&](int S) {
#pragma unroll
        for (int q = 0; q < 4 * NB; ++q) {
          const bool ok = S * SK_KS + kof[q] < krange;
          dma16(rb, ok ? base[q] + (uint32_t)S * 128u : OOB, dst0 + slot + q * 1024);
        }
        slot = slot + XSLOT == XRING ? 0u : slot + XSLOT;
      };
#pragma unroll
      for (int S = 0; S < SK_NX - 1; ++S) issue(S);
      for (int S = 0; S < nsl; ++S) {
        vm_barrier<4 * NB * (SK_NX - 2)>();  // slab S landed: B_S
        issue(S + SK_NX - 1);                // into the slot of S-1
      }
      vm_barrier<0>();
    }
  } else if (wave >= 4) {
    // ------------------------------------------------------------ W loaders (4, 5)
    // KC slab: W rows m0..m0+63 x k = klo + 64S ..; TR slab: k-rows klo + 64S .. x
    // m0..m0+63. Wave lw fills the 1 KB blocks 4lw..4lw+3 (8 rows x 128 B each).
    const int lw = wave - 4;
    const i32x4 ra = buf_rsrc(a.A, (uint32_t)((A_TR ? (int64_t)a.K : (int64_t)a.M) * a.lda * 2));
    uint32_t base[4];
    int kof[4];
    bool okm[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = 8 * (4 * lw + q) + (lane >> 3);
      if constexpr (!A_TR) {
        const int c = (lane & 7) ^ swz_kc(r);
        base[q] = (uint32_t)(((int64_t)(m0 + r) * a.lda + klo + 8 * c) * 2);  // rows past M: out of range
        kof[q] = 8 * c;
        okm[q] = true;
      } else {
        const int c = (lane & 7) ^ swz_tr(r);
        base[q] = (uint32_t)(((int64_t)(klo + r) * a.lda + m0 + 8 * c) * 2);
        kof[q] = r;
        okm[q] = m0 + 8 * c < a.M;
      }
    }
    const uint32_t sstep = A_TR ? (uint32_t)((int64_t)SK_KS * a.lda * 2) : (uint32_t)(SK_KS * 2);
    const uint32_t dst0 = ldsw + (uint32_t)(4 * lw * 1024);
    auto issue = [&](int S) {
      const uint32_t dst = dst0 + (uint32_t)((S % SK_NW) * SK_WSLOT);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool ok = okm[q] && S * SK_KS + kof[q] < krange;
        dma16(ra, ok ? base[q] + (uint32_t)S * sstep : OOB, dst + q * 1024);
      }
    };
#pragma unroll
    for (int S = 0; S < SK_NW - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<4 * (SK_NW - 2)>();  // slab S landed: B_S
      issue(S + SK_NW - 1);           // into the slot of S-1
    }
    vm_barrier<0>();
  } else {
    // --------------------------------------------------------------- MMA group
    constexpr int FM = NB;  // m-blocks per wave
    const int fi = lane & 15, kg = lane >> 4;
    const int nw = wave % NB, mw = wave / NB;
    const int mb0 = FM * mw, nb0 = 4 * nw;  // first m-block and n-block of the wave
    // fragment addresses within a slot for k-step 0 (k-step s reads KC chunk 4s + kg,
    // TR k-rows 32s ..)
    uint32_t fa[FM], fx[4];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if constexpr (!A_TR) {
        fa[i] = (uint32_t)((16 * (mb0 + i) + fi) * 128);
      } else {
        // k-rows 8kg + fi/4 (+4) at columns 16i' + 4(fi%4) (i' = mb0 + i): the transpose
        // read hands lane fi the four consecutive k of column 16i' + fi
        const int r = 8 * kg + (fi >> 2);
        const int c = (2 * (mb0 + i) + ((fi >> 1) & 1)) ^ swz_tr(r);
        fa[i] = (uint32_t)(r * 128 + c * 16 + 8 * (fi & 1));
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) fx[j] = (uint32_t)((16 * (nb0 + j) + fi) * 128);
    const int sw = swz_kc(fi);  // rows 16i + fi all have this swizzle

    f32x4 acc[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    bf16x8 wa[2][FM], xb[2][4];
    auto read = [&](uint32_t ws, uint32_t xs, int s, bf16x8 (&wd)[FM], bf16x8 (&xd)[4]) {
      const uint32_t co = (uint32_t)(((4 * s + kg) ^ sw) * 16);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        if constexpr (!A_TR) {
          wd[i] = __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(ws + fa[i] + co));
        } else {
          lds_i16x4 *p = (lds_i16x4 *)(uintptr_t)(ws + fa[i] + (uint32_t)(s * 4096));
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p + 4 * 128 / 8);
          wd[i] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        xd[j] = __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(xs + fx[j] + co));
    };
    auto mma = [&](const bf16x8 (&wf)[FM], const bf16x8 (&xf)[4]) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[i], xf[j], acc[i][j], 0, 0, 0);
    };

    uint32_t ws = ldsw, xs = ldsx;  // slots of the slab being read
    lds_barrier();                  // B_0: slab 0 landed
    read(ws, xs, 0, wa[0], xb[0]);
    // Each k-step issues the fragment reads of the next one before its own MFMAs, so
    // that the reads land behind 16 MFMAs; the scheduling barriers keep that order.
    for (int S = 0; S < nsl; ++S) {
      read(ws, xs, 1, wa[1], xb[1]);
      __builtin_amdgcn_sched_barrier(0);
      mma(wa[0], xb[0]);
      __builtin_amdgcn_sched_barrier(0);
      // every read of slab S has landed: publish S+1, free S
      lds_barrier();  // B_{S+1}
      ws = ldsw + (uint32_t)(((S + 1) % SK_NW) * SK_WSLOT);
      xs = xs + XSLOT == ldsx + XRING ? ldsx : xs + XSLOT;
      read(ws, xs, 0, wa[0], xb[0]);  // past the last slab this reads a spent slot, unused
      __builtin_amdgcn_sched_barrier(0);
      mma(wa[1], xb[1]);
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- stage the tile: element (n, m) at float n*64 + 4*((m/4) ^ (n%16)) + m%4.
    // The activation ring is free: every wave has passed B_nsl.
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = 16 * (nb0 + j) + fi, u = 4 * (mb0 + i) + kg;
        *reinterpret_cast<f32x4 *>(stg + n * 64 + 4 * (u ^ (n & 15))) = acc[i][j];
      }
  }
  lds_barrier();
  const float *stg = reinterpret_cast<const float *>(smem);
  const int u = tid & 15;
  if (!a.fused) {
    // ---- partial tile out: the rows n0.. of one contiguous block, 16 threads per 256-byte
    // row. Device-scope stores (sc1) write through the XCD's L2, so the partials do not sit
    // there dirty until the end-of-kernel writeback (the AlexNet FC step is ~6 us faster
    // than with default stores).
    float *dst = a.partial + (int64_t)split * a.sstride + (int64_t)(m0 / SK_BM) * a.tpitch;
    const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(dst, 0, (int)(a.tpitch * 4), BUF_DW3);
#pragma unroll
    for (int p = 0; p < 2 * NB; ++p) {
      const int nl = 32 * p + (tid >> 4), n = n0 + nl;
      if (n < a.N) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + nl * 64 + 4 * (u ^ (nl & 15)));
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), prs, (uint32_t)((n * 64 + 4 * u) * 4), 0, CPOL_SC1);
      }
    }
    return;
  }
  {
    // ---- whole K in this workgroup: out(m, n) = [mask > 0] * relu?(alpha * acc + bias[m]),
    // four consecutive m of one sample per thread, the same arithmetic as the split reduce.
    const int m = m0 + 4 * u;
#pragma unroll
    for (int p = 0; p < 2 * NB; ++p) {
      const int nl = 32 * p + (tid >> 4), n = n0 + nl;
      if (n < a.N && m < a.M) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + nl * 64 + 4 * (u ^ (nl & 15)));
        const int cnt = min(4, a.M - m);
        const bool vec = a.vec && cnt == 4;
        float bb[4] = {0.f, 0.f, 0.f, 0.f};
        bool keep[4] = {true, true, true, true};
        if (vec) {
          if (a.bias) {
            const f32x4 t = *reinterpret_cast<const f32x4 *>(a.bias + m);
            bb[0] = t[0]; bb[1] = t[1]; bb[2] = t[2]; bb[3] = t[3];
          }
          if (a.mask) {
            const u32x2 mk = *reinterpret_cast<const u32x2 *>(a.mask + (int64_t)n * a.ldmask + m);
#pragma unroll
            for (int i = 0; i < 4; ++i) keep[i] = bf16_to_f32((uint16_t)((mk[i >> 1] >> (16 * (i & 1))) & 0xffffu)) > 0.0f;
          }
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (i < cnt) {
              if (a.bias) bb[i] = a.bias[m + i];
              if (a.mask) keep[i] = bf16_to_f32(a.mask[(int64_t)n * a.ldmask + m + i]) > 0.0f;
            }
        }
        float x[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float y = a.alpha * v[i] + bb[i];
          if (a.relu) y = y > 0.0f ? y : 0.0f;
          x[i] = keep[i] ? y : 0.0f;
        }
        if (a.out_bf16) {
          uint16_t *o = reinterpret_cast<uint16_t *>(a.out) + (int64_t)n * a.ldo + m;
          if (vec) {
            *reinterpret_cast<u32x2 *>(o) = u32x2{(uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16),
                                                  (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16)};
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (i < cnt) o[i] = f32_to_bf16(x[i]);
          }
        } else {
          float *o = reinterpret_cast<float *>(a.out) + (int64_t)n * a.ldo + m;
          if (vec) {
            *reinterpret_cast<f32x4 *>(o) = f32x4{x[0], x[1], x[2], x[3]};
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (i < cnt) o[i] = x[i];
          }
        }
      }
    }
  }
}

template <bool A_TR, int NB>
__global__ void __launch_bounds__(512, 1) skinny_kernel(SkArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[sk_lds_bytes<NB>()];
  skinny_body<A_TR, NB>(a, smem, (int)blockIdx.x);
}

// One launch for two independent products of a local backward pass (App. A): the Delta_X
// partial W^T Delta_Y on this kernel with K whole (workgroups 0 .. n_sk-1) and the Delta_W
// partial Delta_Y^T X stored as fp32 on the large-tile kernel (workgroups from n_pad, a
// multiple of 8, so that its launch order keeps its XCD mapping). Each workgroup runs one
// of the two bodies, so each product computes exactly what its own launch would.
template <int NB, int OH>
__global__ void __launch_bounds__(512, 1) dx_dw_pair_kernel(SkArgs sk, DlArgs dl, int n_sk, int n_pad, int g_dl) {
  constexpr int L1 = sk_lds_bytes<NB>(), L2 = dl_lds_bytes<OH, false>();
  __shared__ __attribute__((aligned(1024))) char smem[L1 > L2 ? L1 : L2];
  const int bid = (int)blockIdx.x;
  if (bid < n_sk) skinny_body<true, NB>(sk, smem, bid);
  else if (bid >= n_pad) dw_wide_body<false, OH, false>(dl, smem, bid - n_pad, g_dl);
}

template <bool VEC, int LANES>
__global__ void __launch_bounds__(256) skinny_reduce(SkReduceArgs g) {
  if (g.aux_loss && blockIdx.x == gridDim.x - 1) {
    __shared__ float part[256];
    block_loss_mean(g.aux_n, g.aux_rows, g.aux_scale, g.aux_loss, part);
    return;
  }
  sk_reduce_item<VEC, LANES>(g, (int64_t)blockIdx.x * 256 + threadIdx.x);
}

struct SkSoftmaxArgs {
  const float *partial;
  int64_t tpitch, sstride;
  int64_t ldp;    // > 0: partials laid out [split][row][ldp] (the wide-batch kernel's), else per tile
  int splits, B, C;
  float alpha;
  const float *bias;
  float *logits;  // [B][ldz] fp32
  int64_t ldz;
  const int32_t *labels;
  float inv_batch;
  float *row_loss;
  void *dz;       // [B][lddz] gradient of the batch-mean loss w.r.t. the logits
  int64_t lddz;
  int dz_bf16;
};

// Top layer, one workgroup per sample (one thread per class, C <= 1024): the logit is
// the splits' partials added in split order plus the bias (the same arithmetic as the
// reduce), stored; then softmax cross-entropy over the row: maximum, sum of
// exp(z - max) (each wave in the shuffle order of the row kernel, the waves' values
// added in wave order), per-sample loss lse - z[label] and the gradient
// inv_batch * (softmax - onehot); NaN loss and gradient row for a label outside [0, C).
__global__ void __launch_bounds__(1024) skinny_softmax_rows(SkSoftmaxArgs g) {
  __shared__ float red[2][16];
  const int row = blockIdx.x, c = threadIdx.x, lane = c & 63, w = c >> 6;
  const int nw = (g.C + 63) >> 6;
  const bool in = c < g.C;
  float z = -INFINITY;
  if (in) {
    const float *p = g.ldp > 0 ? g.partial + (int64_t)row * g.ldp + c
                               : g.partial + (int64_t)(c >> 6) * g.tpitch + row * 64 + (c & 63);
    float a = p[0];
    for (int q0 = 1; q0 < g.splits; q0 += 8) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = q0 + u < g.splits ? p[(int64_t)(q0 + u) * g.sstride] : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (q0 + u < g.splits) a += t[u];
    }
    z = g.alpha * a + (g.bias ? g.bias[c] : 0.0f);
    g.logits[(int64_t)row * g.ldz + c] = z;
  }
  float mx = z;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) red[0][w] = mx;
  __syncthreads();
  mx = red[0][0];
  for (int k = 1; k < nw; ++k) mx = fmaxf(mx, red[0][k]);
  const float e = in ? expf(z - mx) : 0.0f;
  float s = e;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) red[1][w] = s;
  __syncthreads();
  s = red[1][0];
  for (int k = 1; k < nw; ++k) s += red[1][k];
  const int lab = g.labels[row];
  const bool ok = lab >= 0 && lab < g.C;
  if (c == (ok ? lab : 0)) g.row_loss[row] = ok ? (mx + logf(s) - z) : __builtin_nanf("");
  if (in) {
    // a label outside [0, C) has no one-hot: its whole gradient row is NaN, like its loss
    const float gr = ok ? g.inv_batch * (e * (1.0f / s) - (c == lab ? 1.0f : 0.0f)) : __builtin_nanf("");
    if (g.dz_bf16)
      reinterpret_cast<uint16_t *>(g.dz)[(int64_t)row * g.lddz + c] = f32_to_bf16(gr);
    else
      reinterpret_cast<float *>(g.dz)[(int64_t)row * g.lddz + c] = gr;
  }
}

int nb_for(int N) { return N <= 64 ? 1 : N <= 128 ? 2 : 4; }


}  // namespace

bool skinny_dims_fit(const GemmProblem &p) {
  // K a multiple of 8 (whole 16-byte chunks), or B's rows zero-padded past K with A read by
  // k-rows (rows past K read as zero)
  // (or B read in 4-byte pieces with K even: pieces past K read as zero)
  return p.dtype == IMBD_BF16 && p.b_kc && p.epi.mode == EPI_STORE && p.db_mode == 0 && p.N >= 1 &&
         p.N <= (p.b_dw4 ? 128 : 256) && p.M >= 1 && p.K >= 1 &&
         (p.K % 8 == 0 || (p.b_kpad8 && !p.a_kc) || (p.b_dw4 && !p.a_kc && p.K % 2 == 0)) &&
         (p.a_kc || p.M % 8 == 0);
}

bool skinny_fits(const GemmProblem &p) {
  auto al = [](const void *q, int a) { return (reinterpret_cast<uintptr_t>(q) % a) == 0; };
  const int64_t arows = p.a_kc ? p.M : p.K;
  const bool bal = p.b_dw4 ? p.ldb % 2 == 0 && al(p.B, 4) : p.ldb % 8 == 0 && al(p.B, 16);
  return skinny_dims_fit(p) && p.lda % 8 == 0 && bal && al(p.A, 16) &&
         (arows + SK_KS + SK_BM) * p.lda * 2 < ((int64_t)1 << 31) &&
         ((int64_t)256 * p.ldb + p.K + SK_KS) * 2 < ((int64_t)1 << 31);
}

// Plan of a product: NB (64*NB samples per workgroup, tiles_n sample tiles) and the K
// split. Modelled time of a plan: the rounds of workgroups over 256 CUs times one
// workgroup's time (its 64-k slabs at a per-slab cost that grows with the bytes a slab
// brings into LDS, plus a fixed cost of start-up and tile write-out, which is larger
// for an fp32 partial tile than for the epilogue's output), bounded below by the HBM
// time of W, the activations and the partials; a split plan also pays the reduce launch
// (a slower reduce past four splits). Costs are the kernel's measured times on gfx950 in
// the 9216-4096-4096-1000 step at B = 256 (cycles at 2.1 GHz): per slab 567 / 677 / 1090
// cycles for 64 / 128 / 256 samples; fixed 7.6K (K whole, epilogue fused) and 7.1K /
// 13.7K cycles (128 / 256 samples, partial tile); the reduce ~4.4 us plus 0.045 us per MB
// of partials (0.116 us per MB past four splits, where four lanes share an output).
struct SkPlan {
  int nb, tiles_n, splits, k_split;
};

static bool sk_fused_ok(const GemmProblem &p) {
  return p.epi.mode == EPI_STORE && (p.epi.mask == nullptr || p.epi.mask_dtype == IMBD_BF16);
}

static SkPlan sk_plan(const GemmProblem &p) {
  const int tiles_m = (p.M + SK_BM - 1) / SK_BM;
  const double hbm = 5.0e12, clk = 2.1e9;
  const double slab_clk[5] = {0, 567.0, 677.0, 0, 1090.0};
  const double fix_fused[5] = {0, 7600.0, 7600.0, 0, 9000.0};
  const double fix_part[5] = {0, 7100.0, 7100.0, 0, 13700.0};
  const int forced_s = opt(IMBD_OPT_SKINNY_SPLITS), forced_nb = opt(IMBD_OPT_SKINNY_NB);
  const bool fusable = sk_fused_ok(p);
  SkPlan best{p.b_dw4 ? 2 : 4, 1, 1, p.K};
  double best_t = 1e30;
  for (int nb = 1; nb <= 4; nb *= 2) {
    if (forced_nb > 0 ? nb != forced_nb : nb > nb_for(p.N)) continue;
    if (p.b_dw4 && nb > 2) continue;  // 4-byte pieces: at most 128 samples per workgroup
    const int tiles_n = (p.N + 64 * nb - 1) / (64 * nb);
    for (int s = 1; s <= 64; ++s) {
      const int ks = ((p.K + s - 1) / s + SK_KS - 1) / SK_KS * SK_KS;
      if ((p.K + ks - 1) / ks != s) continue;
      const int64_t blocks = (int64_t)tiles_m * tiles_n * s;
      if (blocks > 65535) break;
      const bool fused = s == 1 && fusable;
      const double bytes = 2.0 * p.M * p.K + 2.0 * p.N * p.K + (fused ? 0.0 : 8.0 * s * (double)p.M * p.N);
      const int64_t rounds = (blocks + 255) / 256;
      const double t_cu = rounds * ((ks / SK_KS) * slab_clk[nb] + (fused ? fix_fused[nb] : fix_part[nb])) / clk;
      // past 16 splits the reduce's threads wait on their loads round after round (four
      // splits per round): ~0.6 us per extra round
      const double t_red = fused ? 0.0
                                 : 4.4e-6 + (s > 4 ? 0.116e-12 : 0.045e-12) * 4.0 * s * (double)p.M * p.N +
                                       0.6e-6 * (double)((s + 3) / 4 > 4 ? (s + 3) / 4 - 4 : 0);
      const double t = (bytes / hbm > t_cu ? bytes / hbm : t_cu) + t_red;
      const bool pick = forced_s > 0 ? s == forced_s && (best_t == 1e30 || t < best_t) : t < best_t * 0.98;
      if (pick) {
        best_t = t;
        best = SkPlan{nb, tiles_n, s, ks};
      }
    }
  }
  return best;
}

void skinny_plan(const GemmProblem &p, int *splits_out, int *k_split_out) {
  const SkPlan pl = sk_plan(p);
  *splits_out = pl.splits;
  *k_split_out = pl.k_split;
}

// Launches the product kernel (partials into ws, or the epilogue applied in the kernel
// when K is whole); returns its arguments in *out.
// The kernel's arguments for a problem and its plan; returns the number of workgroups.
static int prepare_skinny(const GemmProblem &p, const SkPlan &pl, void *ws, bool allow_fused, SkArgs *out) {
  SkArgs g{};
  g.A = reinterpret_cast<const uint16_t *>(p.A);
  g.B = reinterpret_cast<const uint16_t *>(p.B);
  g.lda = p.lda;
  g.ldb = p.ldb;
  g.M = p.M;
  g.N = p.N;
  g.K = p.K;
  g.k_split = pl.k_split;
  g.splits = pl.splits;
  g.tiles_m = (p.M + SK_BM - 1) / SK_BM;
  g.tiles_n = pl.tiles_n;
  g.partial = reinterpret_cast<float *>(ws);
  g.tpitch = sk_tile_pitch(p.N);
  g.sstride = sk_split_pitch(p.M, p.N);
  const Epilogue &e = p.epi;
  g.b_dw4 = p.b_dw4 ? 1 : 0;
  g.fused = allow_fused && pl.splits == 1 && sk_fused_ok(p);
  if (g.fused) {
    auto al = [](const void *q, int a) { return q == nullptr || (reinterpret_cast<uintptr_t>(q) % a) == 0; };
    g.alpha = e.alpha;
    g.bias = e.bias;
    g.relu = e.relu;
    g.mask = reinterpret_cast<const uint16_t *>(e.mask);
    g.ldmask = e.ldmask;
    g.out = e.out;
    g.ldo = e.ldo;
    g.out_bf16 = e.out_dtype == IMBD_BF16 ? 1 : 0;
    g.vec = al(e.bias, 16) && (e.mask == nullptr || (al(e.mask, 8) && e.ldmask % 4 == 0)) &&
            (g.out_bf16 ? al(e.out, 8) : al(e.out, 16)) && e.ldo % 4 == 0;
    if (p.aux_loss && p.aux_n > 0) {
      g.aux_rows = p.aux_rows;
      g.aux_loss = p.aux_loss;
      g.aux_n = p.aux_n;
      g.aux_scale = p.aux_scale;
    }
  }
  *out = g;
  return g.tiles_m * g.tiles_n * pl.splits + (g.aux_loss ? 1 : 0);
}

static int launch_skinny_product(const GemmProblem &p, void *ws, hipStream_t s, SkArgs *out, bool allow_fused) {
  const SkPlan pl = sk_plan(p);
  SkArgs g;
  const int grid = prepare_skinny(p, pl, ws, allow_fused, &g);
  {
    LaunchTimer t(p.kclass, p.layer, s);
    if (p.a_kc) {
      if (pl.nb == 1) hipLaunchKernelGGL((skinny_kernel<false, 1>), dim3(grid), dim3(512), 0, s, g);
      else if (pl.nb == 2) hipLaunchKernelGGL((skinny_kernel<false, 2>), dim3(grid), dim3(512), 0, s, g);
      else hipLaunchKernelGGL((skinny_kernel<false, 4>), dim3(grid), dim3(512), 0, s, g);
    } else {
      if (pl.nb == 1) hipLaunchKernelGGL((skinny_kernel<true, 1>), dim3(grid), dim3(512), 0, s, g);
      else if (pl.nb == 2) hipLaunchKernelGGL((skinny_kernel<true, 2>), dim3(grid), dim3(512), 0, s, g);
      else hipLaunchKernelGGL((skinny_kernel<true, 4>), dim3(grid), dim3(512), 0, s, g);
    }
  }
  *out = g;
  return check_launch("skinny");
}

// The split-K reduce of a product whose partials launch_skinny_product left in ws.
static SkReduceArgs skinny_reduce_args(const GemmProblem &p, const SkArgs &g, bool *vec, int *lanes,
                                       int64_t *threads) {
  SkReduceArgs r;
  r.partial = g.partial;
  r.tpitch = g.tpitch;
  r.sstride = g.sstride;
  r.M = p.M;
  r.N = p.N;
  r.splits = g.splits;
  r.epi = p.epi;
  r.aux_rows = p.aux_rows;
  r.aux_loss = p.aux_n > 0 ? p.aux_loss : nullptr;
  r.aux_n = p.aux_n;
  r.aux_scale = p.aux_scale;
  const Epilogue &e = p.epi;
  auto al = [](const void *q, int a) { return q == nullptr || (reinterpret_cast<uintptr_t>(q) % a) == 0; };
  *vec = p.M % 8 == 0 && al(e.out, 16) && e.ldo % 8 == 0 && al(e.bias, 16) &&
         (e.mask == nullptr || (al(e.mask, 16) && e.ldmask % 8 == 0));
  *lanes = g.splits > 4 ? 4 : 1;
  *threads = (int64_t)g.tiles_m * p.N * 8 * *lanes;
  return r;
}

static int launch_skinny_reduce(const SkReduceArgs &r, bool vec, int lanes, int64_t threads, int layer,
                                hipStream_t s) {
  const unsigned blocks = (unsigned)((threads + 255) / 256) + (r.aux_loss ? 1u : 0u);
  {
    LaunchTimer t(IMBD_K_SPLITK, layer, s);
    if (lanes == 4) {
      if (vec) hipLaunchKernelGGL((skinny_reduce<true, 4>), dim3(blocks), dim3(256), 0, s, r);
      else hipLaunchKernelGGL((skinny_reduce<false, 4>), dim3(blocks), dim3(256), 0, s, r);
    } else {
      if (vec) hipLaunchKernelGGL((skinny_reduce<true, 1>), dim3(blocks), dim3(256), 0, s, r);
      else hipLaunchKernelGGL((skinny_reduce<false, 1>), dim3(blocks), dim3(256), 0, s, r);
    }
  }
  return check_launch("skinny_reduce");
}

int run_skinny(const GemmProblem &p, void *ws, hipStream_t s) {
  ReduceTail tail;
  return run_skinny_split(p, ws, s, nullptr, &tail);
}

int run_skinny_split(const GemmProblem &p, void *ws, hipStream_t s, bool *deferred, ReduceTail *tail) {
  if (deferred) *deferred = false;
  SkArgs g;
  int rc = launch_skinny_product(p, ws, s, &g, true);
  if (rc != IMBD_OK || g.fused) return rc;
  bool vec;
  int lanes;
  int64_t threads;
  const SkReduceArgs r = skinny_reduce_args(p, g, &vec, &lanes, &threads);
  // a later launch may carry the reduce: one thread per item, the whole-vector form
  if (deferred && vec && lanes == 1 && r.aux_loss == nullptr) {
    tail->kind = 1;
    tail->sk = r;
    tail->items = threads;
    *deferred = true;
    return IMBD_OK;
  }
  return launch_skinny_reduce(r, vec, lanes, threads, p.layer, s);
}

int run_skinny_reduce_tail(const ReduceTail &tail, int layer, hipStream_t s) {
  return launch_skinny_reduce(tail.sk, true, 1, tail.items, layer, s);
}

bool skinny_softmax_fits(const GemmProblem &p) {
  return skinny_fits(p) && p.a_kc && p.M <= 1024 && p.epi.relu == 0 && p.epi.mask == nullptr &&
         p.epi.out_dtype == IMBD_F32 && opt(IMBD_OPT_TOP_UNFUSED) == 0;
}

int run_skinny_softmax(const GemmProblem &p, void *ws, const int32_t *labels, float inv_batch, float *row_loss,
                       void *dz, int64_t lddz, int dz_dtype, hipStream_t s) {
  SkArgs g;
  int rc = launch_skinny_product(p, ws, s, &g, false);
  if (rc != IMBD_OK) return rc;
  SkSoftmaxArgs a;
  a.partial = g.partial;
  a.tpitch = g.tpitch;
  a.sstride = g.sstride;
  a.ldp = 0;
  a.splits = g.splits;
  a.B = p.N;
  a.C = p.M;
  a.alpha = p.epi.alpha;
  a.bias = p.epi.bias;
  a.logits = reinterpret_cast<float *>(p.epi.out);
  a.ldz = p.epi.ldo;
  a.labels = labels;
  a.inv_batch = inv_batch;
  a.row_loss = row_loss;
  a.dz = dz;
  a.lddz = lddz;
  a.dz_bf16 = dz_dtype == IMBD_BF16 ? 1 : 0;
  {
    LaunchTimer t(IMBD_K_SOFTMAX, p.layer, s);
    const int threads = (p.M + 63) / 64 * 64;
    hipLaunchKernelGGL(skinny_softmax_rows, dim3(p.N), dim3(threads), 0, s, a);
  }
  return check_launch("skinny_softmax_rows");
}

int run_softmax_rows_from_partials(const GemmProblem &p, const float *partial, int64_t ldp, int64_t sstride,
                                   int splits, const int32_t *labels, float inv_batch, float *row_loss, void *dz,
                                   int64_t lddz, int dz_dtype, hipStream_t s) {
  SkSoftmaxArgs a;
  a.partial = partial;
  a.tpitch = 0;
  a.sstride = sstride;
  a.ldp = ldp;
  a.splits = splits;
  a.B = p.N;
  a.C = p.M;
  a.alpha = p.epi.alpha;
  a.bias = p.epi.bias;
  a.logits = reinterpret_cast<float *>(p.epi.out);
  a.ldz = p.epi.ldo;
  a.labels = labels;
  a.inv_batch = inv_batch;
  a.row_loss = row_loss;
  a.dz = dz;
  a.lddz = lddz;
  a.dz_bf16 = dz_dtype == IMBD_BF16 ? 1 : 0;
  {
    LaunchTimer t(IMBD_K_SOFTMAX, p.layer, s);
    const int threads = (p.M + 63) / 64 * 64;
    hipLaunchKernelGGL(skinny_softmax_rows, dim3(p.N), dim3(threads), 0, s, a);
  }
  return check_launch("softmax_rows_from_partials");
}

size_t skinny_ws_bytes(const GemmProblem &p) {
  // a plan that leaves K whole still needs its one partial when the caller reduces it
  // (the top layer's softmax pass reads the partials)
  const SkPlan pl = sk_plan(p);
  return (size_t)pl.splits * (size_t)sk_split_pitch(p.M, p.N) * sizeof(float);
}

int run_local_dx_dw_pair(const GemmProblem &dx, const GemmProblem &dw, void *ws, hipStream_t s) {
  constexpr int NOT_TAKEN = 1;
  if (opt(IMBD_OPT_LOCAL_PAIR) == 0 || opt(IMBD_OPT_SKINNY_OFF) != 0) return NOT_TAKEN;
  if (dx.M <= 0 || dx.N <= 0 || dw.M <= 0 || dw.N <= 0 || dx.aux_loss || !dx.b_kc || dx.a_kc) return NOT_TAKEN;
  if (dx.b_dw4 != dw.b_dw4) return NOT_TAKEN;
  if (!skinny_fits(dx) || !sk_fused_ok(dx) || !dw_wide_fits(dw) || dw.epi.mode != EPI_STORE) return NOT_TAKEN;
  const SkPlan pl = sk_plan(dx);
  if (pl.splits != 1) return NOT_TAKEN;  // its reduce would follow the pair
  if (dx.b_dw4 && pl.nb > 2) return NOT_TAKEN;
  // the large-tile product alone on two workgroups per CU (a launch of its own is faster)
  // or with its bias on the column-sum kernel: not paired
  DlArgs d;
  int oh, g_dl;
  bool dual;
  dw_wide_prepare(dw, 0, &d, &oh, &dual, &g_dl);
  if (dual || (dw.db_mode != 0 && d.db_mode == 0)) return NOT_TAKEN;
  SkArgs g;
  const int n_sk = prepare_skinny(dx, pl, ws, true, &g);
  const int n_pad = (n_sk + 7) / 8 * 8;
  dw_wide_prepare(dw, n_pad, &d, &oh, &dual, &g_dl);
  const int grid = n_pad + g_dl;
  {
    LaunchTimer t(dw.kclass, dw.layer, s);
    const int v = 4 * (oh == 256) + pl.nb;
    if (v == 1) hipLaunchKernelGGL((dx_dw_pair_kernel<1, 128>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
    else if (v == 2) hipLaunchKernelGGL((dx_dw_pair_kernel<2, 128>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
    else if (v == 4) hipLaunchKernelGGL((dx_dw_pair_kernel<4, 128>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
    else if (v == 5) hipLaunchKernelGGL((dx_dw_pair_kernel<1, 256>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
    else if (v == 6) hipLaunchKernelGGL((dx_dw_pair_kernel<2, 256>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
    else hipLaunchKernelGGL((dx_dw_pair_kernel<4, 256>), dim3(grid), dim3(512), 0, s, g, d, n_sk, n_pad, g_dl);
  }
  return check_launch("dx_dw_pair");
}

}  // namespace imbd
