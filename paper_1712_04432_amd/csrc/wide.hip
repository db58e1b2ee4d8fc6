// Forward and Delta_X products of a fully connected layer for batches above the skinny
// kernel's 256 samples (bf16 operands, fp32 accumulation), Sec. 1's first two products
// of a layer with the sample as the row index of every activation:
//   forward  Y[b][o]  = sum_i W[o][i] X[b][i]    (A = W read along its rows)
//   Delta_X  dX[b][i] = sum_o W[o][i] dY[b][o]   (A = W read as k-rows, o = k)
// In the notation of GemmProblem: D(m, n) = sum_k A(m, k) B(k, n) with n the sample and
// B stored [n][k].
//
// At these batch sizes the products are MFMA-bound (2 x batch flops per weight byte
// read), so a workgroup owns a 256 (m) x 128 (sample) tile and runs the large-tile
// structure of the conv tile kernels (csrc/conv.hip): both operands go through LDS in
// 64-k slabs written by buffer loads that land in LDS as whole 128-byte lines, loader
// waves with their own memory counters, one barrier per slab, XOR-swizzled 16-byte
// chunks:
//  * waves 8-9 stream the sample slab (128 rows x 64 k) through a 4-slot ring;
//  * waves 10-11 stream the weight slab (256 m x 64 k) through a 3-slot ring: W rows for
//    the forward product, k-rows of W (64 rows x 256 columns, as four 64-column quarters)
//    for Delta_X, whose fragments then come from the gfx950 LDS transpose read;
//  * waves 0-7, two per SIMD, each accumulate 64 samples x 64 m in registers.
// When the tiles alone cannot fill the chip, K is split and each split writes fp32
// partials that the split-K reduce adds in split order and finishes (bias, ReLU, ReLU'
// mask, bf16 or fp32 store); otherwise the kernel finishes the tile itself, the same way.
//
// Ragged edges: rows past M (forward) or N, and k-rows past K (Delta_X), are past the end
// of their buffer descriptors and read as zero; chunks at or past K inside a row are
// masked explicitly (they would read the next row). Outputs past M or N are not stored.

#include <stdlib.h>

#include "cdna4.h"
#include "loss_mean.h"

namespace imbd {
namespace {

constexpr int WD_BM = 256;             // m per workgroup (weight rows or columns)
constexpr int WD_BN = 128;             // samples per workgroup
constexpr int WD_KS = 64;              // k per slab
constexpr int WD_NB = 4;               // sample ring slots
constexpr int WD_NA = 3;               // weight ring slots
constexpr int WD_BSLOT = WD_BN * 128;  // 16 KB
constexpr int WD_ASLOT = WD_BM * 128;  // 32 KB
constexpr int WD_QSLOT = 64 * 128;     // one 64-column quarter of a k-row slab
constexpr int WD_PITCH = WD_BM + 4;    // staging row pitch in floats (1040 B)
constexpr int WD_GM = 8;               // m tiles per launch-order group
constexpr int WD_NT = 768;

struct WdArgs {
  const uint16_t *A;    // W
  const uint16_t *B;    // X or Delta_Y: [N][ldb]
  int64_t lda, ldb;
  uint32_t a_bytes, b_bytes;  // buffer extents
  int M, N, K;
  int tiles_m, tiles_n, splits, kps, nsl;  // kps: slabs per split; nsl: slabs of K
  Epilogue epi;                             // finish when splits == 1
  float *partial;                           // [split][n][ldp] fp32 when splits > 1
  int64_t ldp, sstride;
  int gmain;                                // product workgroups (a multiple of 8)
  // side job in one extra workgroup (the last): *aux_loss = aux_scale * sum of aux_rows
  const float *aux_rows;
  float *aux_loss;
  int aux_n;
  float aux_scale;
};

__device__ __forceinline__ int wd_swz_kc(int r) { return r & 7; }
__device__ __forceinline__ int wd_swz_tr(int r) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1); }

// TR: A is stored as k-rows (Delta_X); else as m-rows (forward).
template <bool TR>
__global__ void __launch_bounds__(WD_NT, 1) wide_kernel(WdArgs a) {
  constexpr int NMW = 8;
  constexpr int FM = 8;    // 16-sample blocks of the tile
  constexpr int FMW = 4;   // sample blocks per MMA wave
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int ARING = WD_NA * WD_ASLOT, BRING = WD_NB * WD_BSLOT;
  __shared__ __attribute__((aligned(1024))) char smem[ARING + BRING];
  static_assert(ARING + BRING <= 160 * 1024, "LDS");
  static_assert(WD_BN * WD_PITCH * 4 <= ARING + BRING, "staging");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (a.aux_loss && (int)blockIdx.x == a.gmain) {
    block_loss_mean(a.aux_n, a.aux_rows, a.aux_scale, a.aux_loss, reinterpret_cast<float *>(smem));
    return;
  }
  // The product's grid is padded to a multiple of 8 and each XCD takes a contiguous range
  // of the launch order, in which the tiles of one split come in groups of WD_GM m tiles x
  // all sample tiles: the workgroups resident on an XCD share weight and sample slabs in L2.
  const int G = a.gmain;
  int L = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  const int per_split = a.tiles_m * a.tiles_n;
  if (L >= per_split * a.splits) return;
  const int split = L / per_split;
  L -= split * per_split;
  const int mg = L / (WD_GM * a.tiles_n);
  const int gsz = min(WD_GM, a.tiles_m - mg * WD_GM);
  L -= mg * WD_GM * a.tiles_n;
  const int nt = L / gsz, mt = mg * WD_GM + (L - (L / gsz) * gsz);
  const int m0 = mt * WD_BM, n0 = nt * WD_BN;
  const int s0 = split * a.kps;
  const int nsl = min(a.kps, a.nsl - s0);  // slabs of this split
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t ldsw = lds0, ldsb = lds0 + ARING;

  if (wave >= NMW + 2) {
    // --------------------------------------------------------------- weight loaders
    const int ww = wave - NMW - 2;
    const i32x4 rw = buf_rsrc(a.A, a.a_bytes);
    uint32_t base[16], dst[16];
    // forward: the source chunk (lane%8) ^ (row%8) of every row a lane loads is the same
    const int kc = 8 * ((lane & 7) ^ (lane >> 3));
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int blk = 16 * ww + q;  // 1 KB block of the slot
      if constexpr (!TR) {
        const int r = 8 * blk + (lane >> 3);  // W row m0 + r
        base[q] = (uint32_t)(((int64_t)(m0 + r) * a.lda + kc) * 2);
        dst[q] = (uint32_t)(blk * 1024);
      } else {
        // quarter h (columns m0 + 64h ..), k-row r of the slab
        const int h = blk >> 3, g = blk & 7;
        const int r = 8 * g + (lane >> 3);
        const int c = (lane & 7) ^ wd_swz_tr(r);
        base[q] = (uint32_t)(((int64_t)r * a.lda + m0 + 64 * h + 8 * c) * 2);
        dst[q] = (uint32_t)(h * WD_QSLOT + g * 1024);
      }
    }
    auto issue = [&](int S) {
      const uint32_t slot = ldsw + (uint32_t)((S % WD_NA) * WD_ASLOT);
      const int k0 = (s0 + S) * WD_KS;
      uint32_t off = OOB;
      if (S < nsl) {
        if constexpr (!TR) off = (k0 + kc < a.K) ? (uint32_t)(k0 * 2) : OOB;
        else off = (uint32_t)((int64_t)k0 * a.lda * 2);
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) dma16(rw, off == OOB ? OOB : base[q] + off, slot + dst[q]);
    };
#pragma unroll
    for (int S = 0; S < WD_NA - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<16 * (WD_NA - 2)>();  // slab S landed: B_S
      issue(S + WD_NA - 1);            // into the slot of S-1
    }
    vm_barrier<0>();
  } else if (wave >= NMW) {
    // --------------------------------------------------------------- sample loaders
    // rows n0 ..; wave bw fills the 1 KB blocks FM*bw .. FM*bw + FM-1 (8 rows each)
    const int bw = wave - NMW;
    const i32x4 rb = buf_rsrc(a.B, a.b_bytes);
    const int kc = 8 * ((lane & 7) ^ (lane >> 3));
    uint32_t base[FM];
#pragma unroll
    for (int q = 0; q < FM; ++q) {
      const int r = 8 * (FM * bw + q) + (lane >> 3);
      base[q] = (uint32_t)(((int64_t)(n0 + r) * a.ldb + kc) * 2);
    }
    const uint32_t d0 = ldsb + (uint32_t)(FM * bw * 1024);
    auto issue = [&](int S) {
      const uint32_t slot = d0 + (uint32_t)((S % WD_NB) * WD_BSLOT);
      const int k0 = (s0 + S) * WD_KS;
      const uint32_t off = (S < nsl && k0 + kc < a.K) ? (uint32_t)(k0 * 2) : OOB;
#pragma unroll
      for (int q = 0; q < FM; ++q) dma16(rb, off == OOB ? OOB : base[q] + off, slot + (uint32_t)(q * 1024));
    };
#pragma unroll
    for (int S = 0; S < WD_NB - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<FM * (WD_NB - 2)>();  // slab S landed: B_S
      issue(S + WD_NB - 1);            // into the slot of S-1
    }
    vm_barrier<0>();
  } else {
    // --------------------------------------------------------------- MMA group
    const int fi = lane & 15, kg = lane >> 4;
    const int nq = wave >> 1;          // m quarter of the wave
    const int mb0 = FMW * (wave & 1);  // first sample block
    const int nb0 = 4 * nq;            // first 16-wide m block
    uint32_t fa[FMW], fx[4];
#pragma unroll
    for (int i = 0; i < FMW; ++i) fa[i] = (uint32_t)((16 * (mb0 + i) + fi) * 128);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (!TR) {
        fx[j] = (uint32_t)((16 * (nb0 + j) + fi) * 128);
      } else {
        // k-rows 8kg + fi/4 (+4) at columns 16j + 4(fi%4) of quarter nq: the transpose
        // read hands lane fi the four consecutive k of column 16j + fi
        const int r = 8 * kg + (fi >> 2);
        const int c = (2 * j + ((fi >> 1) & 1)) ^ wd_swz_tr(r);
        fx[j] = (uint32_t)(nq * WD_QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
      }
    }
    const int sw = wd_swz_kc(fi);

    f32x4 acc[FMW][4];
#pragma unroll
    for (int i = 0; i < FMW; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    bf16x8 bv[2][FMW], wv[2][4];
    auto read = [&](uint32_t bs, uint32_t ws, int s, bf16x8 (&bd)[FMW], bf16x8 (&wd)[4]) {
      const uint32_t co = (uint32_t)(((4 * s + kg) ^ sw) * 16);
#pragma unroll
      for (int i = 0; i < FMW; ++i)
        bd[i] = __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(bs + fa[i] + co));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (!TR) {
          wd[j] = __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(ws + fx[j] + co));
        } else {
          lds_i16x4 *p = (lds_i16x4 *)(uintptr_t)(ws + fx[j] + (uint32_t)(s * 4096));
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p + 4 * 128 / 8);
          wd[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
      }
    };
    auto mma = [&](const bf16x8 (&bf)[FMW], const bf16x8 (&wf)[4]) {
#pragma unroll
      for (int i = 0; i < FMW; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bf[i], wf[j], acc[i][j], 0, 0, 0);
    };

    uint32_t bs = ldsb, ws = ldsw;  // slots of the slab being read
    lds_barrier();                  // B_0: slab 0 landed
    read(bs, ws, 0, bv[0], wv[0]);
    for (int S = 0; S < nsl; ++S) {
      read(bs, ws, 1, bv[1], wv[1]);
      __builtin_amdgcn_sched_barrier(0);
      mma(bv[0], wv[0]);
      __builtin_amdgcn_sched_barrier(0);
      lds_barrier();  // B_{S+1}: every read of slab S has landed; publish S+1, free S
      bs = ldsb + (uint32_t)(((S + 1) % WD_NB) * WD_BSLOT);
      ws = ldsw + (uint32_t)(((S + 1) % WD_NA) * WD_ASLOT);
      read(bs, ws, 0, bv[0], wv[0]);  // past the last slab this reads a spent slot, unused
      __builtin_amdgcn_sched_barrier(0);
      mma(bv[1], wv[1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // ---- stage the tile as [sample][m] fp32 (pitch 260 floats). All of LDS is free:
    // every wave has passed B_nsl, and every loader had drained its loads before it.
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FMW; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) stg[(16 * (mb0 + i) + 4 * kg + e) * WD_PITCH + 16 * (nb0 + j) + fi] = acc[i][j][e];
  }
  lds_barrier();
  const float *stg = reinterpret_cast<const float *>(smem);
  if (a.splits > 1) {
    // ---- fp32 partial rows, written through to the device (the reduce reads them next)
    const __amdgpu_buffer_rsrc_t prs =
        __builtin_amdgcn_make_buffer_rsrc(a.partial + split * a.sstride, 0, (int)(a.sstride * 4), BUF_DW3);
    const int ch = tid & 63, sub = tid >> 6;  // 4 m per thread, 12 rows per pass
    if (m0 + 4 * ch < a.M) {
      for (int r = sub; r < WD_BN && n0 + r < a.N; r += WD_NT / 64) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + r * WD_PITCH + 4 * ch);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), prs,
                                               (uint32_t)(((n0 + r) * a.ldp + m0 + 4 * ch) * 4), 0, 16);
      }
    }
    return;
  }
  // ---- finish the tile: alpha, bias, ReLU, ReLU' mask; 8 m (bf16) or 4 m (fp32) per thread
  const Epilogue &e = a.epi;
  if (e.out_dtype == IMBD_BF16) {
    const int ch = tid & 31, sub = tid >> 5;  // 24 rows per pass
    const int m = m0 + 8 * ch;
    if (m >= a.M) return;
    float bb[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (e.bias) {
      const f32x4 b0 = *reinterpret_cast<const f32x4 *>(e.bias + m);
      const f32x4 b1 = *reinterpret_cast<const f32x4 *>(e.bias + m + 4);
      bb[0] = b0[0]; bb[1] = b0[1]; bb[2] = b0[2]; bb[3] = b0[3];
      bb[4] = b1[0]; bb[5] = b1[1]; bb[6] = b1[2]; bb[7] = b1[3];
    }
    for (int r = sub; r < WD_BN && n0 + r < a.N; r += WD_NT / 32) {
      const int n = n0 + r;
      const f32x4 v0 = *reinterpret_cast<const f32x4 *>(stg + r * WD_PITCH + 8 * ch);
      const f32x4 v1 = *reinterpret_cast<const f32x4 *>(stg + r * WD_PITCH + 8 * ch + 4);
      float x[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        x[i] = e.alpha * x[i] + bb[i];
        if (e.relu) x[i] = x[i] > 0.f ? x[i] : 0.f;
      }
      if (e.mask) {
        const u32x4 mk = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(e.mask) +
                                                          (int64_t)n * e.ldmask + m);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint16_t h = (uint16_t)((mk[i >> 1] >> (16 * (i & 1))) & 0xffffu);
          if (!(bf16_to_f32(h) > 0.f)) x[i] = 0.f;
        }
      }
      u32x4 pk;
#pragma unroll
      for (int i = 0; i < 4; ++i) pk[i] = cvt_pk_bf16(x[2 * i], x[2 * i + 1]);
      *reinterpret_cast<u32x4 *>(reinterpret_cast<uint16_t *>(e.out) + (int64_t)n * e.ldo + m) = pk;
    }
  } else {
    const int ch = tid & 63, sub = tid >> 6;  // 12 rows per pass
    const int m = m0 + 4 * ch;
    if (m >= a.M) return;
    float bb[4] = {0.f, 0.f, 0.f, 0.f};
    if (e.bias) {
      const f32x4 b0 = *reinterpret_cast<const f32x4 *>(e.bias + m);
      bb[0] = b0[0]; bb[1] = b0[1]; bb[2] = b0[2]; bb[3] = b0[3];
    }
    for (int r = sub; r < WD_BN && n0 + r < a.N; r += WD_NT / 64) {
      const int n = n0 + r;
      const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + r * WD_PITCH + 4 * ch);
      float x[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = e.alpha * x[i] + bb[i];
        if (e.relu) x[i] = x[i] > 0.f ? x[i] : 0.f;
      }
      if (e.mask) {
        const u32x2 mk = *reinterpret_cast<const u32x2 *>(reinterpret_cast<const uint16_t *>(e.mask) +
                                                          (int64_t)n * e.ldmask + m);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint16_t h = (uint16_t)((mk[i >> 1] >> (16 * (i & 1))) & 0xffffu);
          if (!(bf16_to_f32(h) > 0.f)) x[i] = 0.f;
        }
      }
      *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m) =
          f32x4{x[0], x[1], x[2], x[3]};
    }
  }
}

int64_t a_extent(const GemmProblem &p) {
  // elements from A to one past the last one a product reads
  return p.a_kc ? (int64_t)(p.M - 1) * p.lda + p.K : (int64_t)(p.K - 1) * p.lda + p.M;
}

}  // namespace

bool wide_dims_fit(const GemmProblem &p) {
  if (opt(IMBD_OPT_WIDE_OFF) != 0) return false;  // the tiled GEMM template instead
  return p.dtype == IMBD_BF16 && p.b_kc && p.db_mode == 0 && p.epi.mode == EPI_STORE && p.M >= 128 &&
         p.N > 256 && p.K >= WD_KS && p.M % 8 == 0 && p.K % 8 == 0;
}

bool wide_fits(const GemmProblem &p) {
  auto al = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) % 16) == 0; };
  const Epilogue &e = p.epi;
  if (!wide_dims_fit(p) || p.lda % 8 || p.ldb % 8 || !al(p.A) || !al(p.B)) return false;
  if (p.a_kc ? p.lda < p.K : p.lda < p.M) return false;
  if (p.ldb < p.K) return false;
  const int64_t lim = (int64_t)1 << 30;  // elements: 2 GiB of bf16 in a buffer descriptor
  if (a_extent(p) >= lim || (int64_t)(p.N - 1) * p.ldb + p.K >= lim || (int64_t)p.N * partial_ld(p.M) >= lim / 2)
    return false;
  if (!e.out || e.ldo % 8 || !al(e.out) || (e.bias && !al(e.bias))) return false;
  return !e.mask || (e.mask_dtype == IMBD_BF16 && e.ldmask % 8 == 0 && al(e.mask));
}

void wide_plan(const GemmProblem &p, int *splits, int *kps) {
  const int tiles = ((p.M + WD_BM - 1) / WD_BM) * ((p.N + WD_BN - 1) / WD_BN);
  const int nsl = (p.K + WD_KS - 1) / WD_KS;
  // split K while the tiles cover fewer than 256 CUs, keeping >= 8 slabs per split
  int s = (256 + tiles / 2) / tiles;
  if (s > nsl / 8) s = nsl / 8;
  if (s < 1) s = 1;
  const int forced = opt(IMBD_OPT_WIDE_SPLITS);
  if (forced >= 1) s = forced < nsl ? forced : nsl;
  *kps = (nsl + s - 1) / s;
  *splits = (nsl + *kps - 1) / *kps;
}

int run_wide(const GemmProblem &p, float *partial, int64_t ldp, int64_t sstride, hipStream_t s) {
  WdArgs a;
  a.A = reinterpret_cast<const uint16_t *>(p.A);
  a.B = reinterpret_cast<const uint16_t *>(p.B);
  a.lda = p.lda;
  a.ldb = p.ldb;
  a.a_bytes = (uint32_t)(a_extent(p) * 2);
  a.b_bytes = (uint32_t)(((int64_t)(p.N - 1) * p.ldb + p.K) * 2);
  a.M = p.M;
  a.N = p.N;
  a.K = p.K;
  a.tiles_m = (p.M + WD_BM - 1) / WD_BM;
  a.tiles_n = (p.N + WD_BN - 1) / WD_BN;
  a.nsl = (p.K + WD_KS - 1) / WD_KS;
  wide_plan(p, &a.splits, &a.kps);
  a.epi = p.epi;
  a.partial = partial;
  a.ldp = ldp;
  a.sstride = sstride;
  a.gmain = (a.tiles_m * a.tiles_n * a.splits + 7) / 8 * 8;
  a.aux_rows = p.aux_rows;
  a.aux_loss = p.aux_n > 0 ? p.aux_loss : nullptr;
  a.aux_n = p.aux_n;
  a.aux_scale = p.aux_scale;
  const int grid = a.gmain + (a.aux_loss ? 1 : 0);
  {
    LaunchTimer t(p.kclass, p.layer, s);
    if (p.a_kc) hipLaunchKernelGGL(wide_kernel<false>, dim3(grid), dim3(WD_NT), 0, s, a);
    else hipLaunchKernelGGL(wide_kernel<true>, dim3(grid), dim3(WD_NT), 0, s, a);
  }
  return check_launch("wide");
}

}  // namespace imbd
