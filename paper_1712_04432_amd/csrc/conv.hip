// Forward and input-gradient passes of the domain-parallel 3x3 conv tile (Sec. 2.2, pure
// domain parallelism: each process convolves its spatial tile with the halo supplied;
// the input gradient takes the output gradient with its own halo), for 256 output
// channels, as implicit GEMMs on the zero-padded (H+2) x (W+2) grid:
//   forward   D(P, o) = sum_{tap, c} x_pad[P + r*(W+2) + s][c] * W[o][tap][c]
//   input grad D(P, c) = sum_{tap, o} dy_pad[P + (2-r)*(W+2) + 2-s][o] * W[o][tap][c]
// with tap = 3r + s and P = (n (H+2) + h) (W+2) + w the row of the padded grid whose
// D(P, .) is the output at position (n, h, w). Each tap is a row shift of a dense
// [positions][channels] matrix, so a k-slab (64 channels of one tap) of the activation
// operand is 64 contiguous channels of shifted rows.
//
// The products are MFMA-bound (2 x 9 x C flops per output), so a workgroup owns a large
// tile: 128 (or 112) output positions x all 256 channels over the whole K = 9 C (no split,
// no partials; the epilogue writes the outputs). With one workgroup per CU, the tiles of a
// short last round run as two 128-channel halves each (the loader and MMA waves of the
// other half only keep the slab barriers). The kernel keeps the layout of the skinny-batch
// kernel (csrc/skinny.hip): both operands travel through LDS in 64-k slabs written by
// buffer loads that go straight to LDS in whole 128-byte lines, loader waves with their
// own memory counters, one barrier per slab, XOR-swizzled 16-byte chunks:
//  * waves 8-9 stream the activation slab (128 or 112 shifted rows x 128 B) through a
//    4-slot ring;
//  * waves 10-11 stream the weight slab (256 channels x 64 k) through a 3-slot ring: rows
//    of W for the forward pass, k-rows of W (64 output channels of one tap x 256 input
//    channels, as four 64-channel quarters) for the input gradient, whose fragments then
//    come from the gfx950 LDS transpose read;
//  * waves 0-7, two per SIMD, each accumulate 64 (or 48) positions x 64 channels in
//    registers.
// After the last slab the tile goes through LDS ([position][channel], fp32) and is written
// as whole 512-byte (bf16) or 1 KB (fp32) output rows.

#include <stdlib.h>

#include "cdna4.h"

namespace imbd {
namespace {

constexpr int CV_BM = 128;             // positions per workgroup (at most; 112 with FM = 7)
constexpr int CV_BN = 256;             // channels of the output per workgroup
constexpr int CV_KS = 64;              // k per slab: 64 channels of one tap
constexpr int CV_NA = 4;               // activation ring slots
constexpr int CV_NW = 3;               // weight ring slots
constexpr int CV_WSLOT = CV_BN * 128;  // 32 KB
constexpr int CV_QSLOT = 64 * 128;     // one 64-channel quarter of a transposed weight slab
constexpr int CV_PITCH = CV_BN + 4;    // staging row pitch in floats (1040 B)
constexpr int CV_CUS = 256;            // compute units of the chip: one workgroup each per round

struct CvArgs {
  const uint16_t *act;  // x_pad (forward) or dy_pad (input gradient): [N][H+2][W+2][Ck]
  const uint16_t *w;    // [C_out][3][3][C_in]
  void *out;            // [N][H][W][256]
  int out_bf16;
  int N, H, W, Ck, Cw;  // Ck: channels of act (the reduction); Cw: C_in (the W row's channel stride)
  int M, tiles;         // output positions N*H*W, tiles of 128 of them
  int tfull, gfull;     // tiles run whole (the first tfull), their workgroups (a multiple of 8)
};

__device__ __forceinline__ int cv_swz_kc(int r) { return r & 7; }
__device__ __forceinline__ int cv_swz_tr(int r) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1); }

// TR: input gradient (W read transposed); else forward. FM: 16-position blocks per tile
// (8: 128 positions; 7: 112, whose tile count fills the chip's rounds better for some
// grids). Eight MMA waves, two per SIMD, so that one computes while the other waits for
// its fragments or the slab barrier (with one per SIMD the matrix pipe was busy ~40% of
// the time); each takes one position half (blocks 0-3 or 4..FM-1) and one channel
// quarter. Waves w and w+4 share a SIMD: with FM = 8 wave w takes position half w%2 and
// quarter w/2; with FM = 7 the two waves of a SIMD take different position halves (4 + 3
// blocks on every SIMD), and each channel half (the quarters of a half tile) still spans
// all four SIMDs. The loader waves follow the MMA waves.
//
// Slab order: for each kernel row r of the taps and each 64-channel chunk, the three taps
// (r, 0), (r, 1), (r, 2) in turn (1-2% faster than all channels of one tap in turn).
template <bool TR, int FM>
__global__ void __launch_bounds__(768, 1) conv_nt_kernel(CvArgs a) {
  static_assert(FM == 8 || FM == 7, "tile");
  constexpr int NMW = 8;
  constexpr int BM = 16 * FM;
  constexpr int NT = 64 * (NMW + 4);
  constexpr int FMW = 4;               // position blocks per MMA wave (at most)
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int ASLOT = BM * 128;
  constexpr int WRING = CV_NW * CV_WSLOT, ARING = CV_NA * ASLOT;
  __shared__ __attribute__((aligned(1024))) char smem[WRING + ARING];
  static_assert(WRING + ARING <= 160 * 1024, "LDS");
  static_assert(BM * CV_PITCH * 4 <= WRING + ARING, "staging");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // The first gfull workgroups take whole tiles (padded to a multiple of 8; consecutive
  // tiles, which share shifted activation rows, run on one XCD). The workgroups after
  // them take the last tiles in 128-channel halves, two per tile, so that the chip's last
  // round of workgroups is a short one.
  int b, hc = -1;
  if ((int)blockIdx.x < a.gfull) {
    b = (int)((blockIdx.x & 7) * (a.gfull >> 3) + (blockIdx.x >> 3));
    if (b >= a.tfull) return;
  } else {
    const int j = (int)blockIdx.x - a.gfull;
    b = a.tfull + (j >> 1);
    hc = j & 1;
  }
  if (b >= a.tiles) return;
  const int m0 = b * BM;
  const int Hp = a.H + 2, Wp = a.W + 2;
  const int nsl = 9 * a.Ck / CV_KS;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t ldsw = lds0, ldsa = lds0 + WRING;
  // tap (3 r + s) and channel offset of slab S: triple q = S / 3 is kernel row q / nch and
  // channel chunk q % nch, and S % 3 the tap's column s
  const int nch = a.Ck / CV_KS;
  auto tap_of = [&](int S, int *c0) {
    const int q = S / 3, r = q / nch;
    *c0 = (q - r * nch) * CV_KS;
    return 3 * r + (S - 3 * q);
  };

  if (wave >= NMW + 2) {
    // --------------------------------------------------------------- weight loaders
    const int ww = wave - NMW - 2;  // loads the slab rows of channels 128 ww .. 128 ww + 127
    const bool on = hc < 0 || ww == hc;
    const i32x4 rw = buf_rsrc(a.w, (uint32_t)((int64_t)9 * a.Ck * CV_BN * 2));
    uint32_t base[16];
    uint32_t dst[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int blk = 16 * ww + q;  // 1 KB block of the slot
      if constexpr (!TR) {
        // W row o = 8 blk + lane/8, 16-byte chunk (lane%8) ^ swz
        const int r = 8 * blk + (lane >> 3);
        const int c = (lane & 7) ^ cv_swz_kc(r);
        base[q] = (uint32_t)(((int64_t)r * 9 * a.Ck + 8 * c) * 2);
        dst[q] = (uint32_t)(blk * 1024);
      } else {
        // quarter h (input channels 64h..64h+63), k-row (output channel) r of the slab
        const int h = blk >> 3, g = blk & 7;
        const int r = 8 * g + (lane >> 3);
        const int c = (lane & 7) ^ cv_swz_tr(r);
        base[q] = (uint32_t)(((int64_t)r * 9 * a.Cw + 64 * h + 8 * c) * 2);
        dst[q] = (uint32_t)(h * CV_QSLOT + g * 1024);
      }
    }
    auto issue = [&](int S) {
      if (!on) return;  // a half tile's other channels: no loads, the same barriers
      const uint32_t slot = ldsw + (uint32_t)((S % CV_NW) * CV_WSLOT);
      uint32_t off = OOB;
      if (S < nsl) {
        int c0;
        const int t = tap_of(S, &c0);
        if constexpr (!TR) off = (uint32_t)((t * a.Ck + c0) * 2);
        else off = (uint32_t)(((int64_t)c0 * 9 + t) * a.Cw * 2);
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) dma16(rw, off == OOB ? OOB : base[q] + off, slot + dst[q]);
    };
#pragma unroll
    for (int S = 0; S < CV_NW - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<16 * (CV_NW - 2)>();  // slab S landed: B_S
      issue(S + CV_NW - 1);            // into the slot of S-1
    }
    vm_barrier<0>();
  } else if (wave >= NMW) {
    // ----------------------------------------------------------- activation loaders
    // The rows of the tile's BM output positions in the padded grid, shifted by the slab's
    // tap; positions past the last one read as zero. Wave aw fills the 1 KB blocks
    // FM*aw .. FM*aw + FM-1 (8 rows each).
    const int aw = wave - NMW;
    const i32x4 ra = buf_rsrc(a.act, (uint32_t)((int64_t)a.N * Hp * Wp * a.Ck * 2));
    uint32_t base[FM];
#pragma unroll
    for (int q = 0; q < FM; ++q) {
      const int r = 8 * (FM * aw + q) + (lane >> 3);
      const int c = (lane & 7) ^ cv_swz_kc(r);
      const int p = m0 + r;
      uint32_t bq = OOB;  // OOB + any slab offset stays past the buffer's end
      if (p < a.M) {
        const int n = p / (a.H * a.W), rem = p - n * a.H * a.W, h = rem / a.W, w = rem - h * a.W;
        bq = (uint32_t)(((int64_t)((n * Hp + h) * Wp + w) * a.Ck + 8 * c) * 2);
      }
      base[q] = bq;
    }
    const uint32_t d0 = ldsa + (uint32_t)(FM * aw * 1024);
    auto issue = [&](int S) {
      const uint32_t slot = d0 + (uint32_t)((S % CV_NA) * ASLOT);
      uint32_t off = OOB;
      if (S < nsl) {
        int c0;
        const int t = tap_of(S, &c0);
        const int r = t / 3, s = t - 3 * r;
        const int shift = TR ? (2 - r) * Wp + 2 - s : r * Wp + s;
        off = (uint32_t)(((int64_t)shift * a.Ck + c0) * 2);
      }
#pragma unroll
      for (int q = 0; q < FM; ++q) dma16(ra, off == OOB ? OOB : base[q] + off, slot + (uint32_t)(q * 1024));
    };
#pragma unroll
    for (int S = 0; S < CV_NA - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<FM * (CV_NA - 2)>();  // slab S landed: B_S
      issue(S + CV_NA - 1);           // into the slot of S-1
    }
    vm_barrier<0>();
  } else if (hc >= 0 && (wave >> 2) != hc) {
    // ------------------------------- MMA waves of a half tile's other channels: the slab
    // barriers B_0 .. B_nsl only
    for (int S = 0; S <= nsl; ++S) lds_barrier();
  } else {
    // --------------------------------------------------------------- MMA group
    const int fi = lane & 15, kg = lane >> 4;
    const int sim = wave & 3, j4 = wave >> 2;
    const int nq = FM == 8 ? wave >> 1 : 2 * j4 + (sim >> 1);    // channel quarter of the wave
    const int ph = FM == 8 ? wave & 1 : (sim & 1) ^ j4;          // position half
    const int mb0 = FMW * ph;                                    // first position block
    const int nbw = ph == 0 ? FMW : FM - FMW;                    // its position blocks
    const int nb0 = 4 * nq;                                      // first 16-channel block
    uint32_t fa[FMW], fx[4];
#pragma unroll
    for (int i = 0; i < FMW; ++i) fa[i] = (uint32_t)((16 * (mb0 + i) + fi) * 128);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (!TR) {
        fx[j] = (uint32_t)((16 * (nb0 + j) + fi) * 128);
      } else {
        // k-rows 8kg + fi/4 (+4) at channels 16j + 4(fi%4) of quarter nq: the transpose
        // read hands lane fi the four consecutive k of channel 16j + fi
        const int r = 8 * kg + (fi >> 2);
        const int c = (2 * j + ((fi >> 1) & 1)) ^ cv_swz_tr(r);
        fx[j] = (uint32_t)(nq * CV_QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
      }
    }
    const int sw = cv_swz_kc(fi);

    f32x4 acc[FMW][4];
#pragma unroll
    for (int i = 0; i < FMW; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    bf16x8 av[2][FMW], wv[2][4];
    auto read = [&](uint32_t as, uint32_t ws, int s, bf16x8 (&ad)[FMW], bf16x8 (&wd)[4]) {
      const uint32_t co = (uint32_t)(((4 * s + kg) ^ sw) * 16);
#pragma unroll
      for (int i = 0; i < FMW; ++i)
        if (i < nbw)
          ad[i] = __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(as + fa[i] + co));
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
    auto mma = [&](const bf16x8 (&af)[FMW], const bf16x8 (&wf)[4]) {
#pragma unroll
      for (int i = 0; i < FMW; ++i)
        if (i < nbw)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], wf[j], acc[i][j], 0, 0, 0);
    };

    uint32_t as = ldsa, ws = ldsw;  // slots of the slab being read
    lds_barrier();                  // B_0: slab 0 landed
    read(as, ws, 0, av[0], wv[0]);
    for (int S = 0; S < nsl; ++S) {
      read(as, ws, 1, av[1], wv[1]);
      __builtin_amdgcn_sched_barrier(0);
      mma(av[0], wv[0]);
      __builtin_amdgcn_sched_barrier(0);
      lds_barrier();  // B_{S+1}: every read of slab S has landed; publish S+1, free S
      as = ldsa + (uint32_t)(((S + 1) % CV_NA) * ASLOT);
      ws = ldsw + (uint32_t)(((S + 1) % CV_NW) * CV_WSLOT);
      read(as, ws, 0, av[0], wv[0]);  // past the last slab this reads a spent slot, unused
      __builtin_amdgcn_sched_barrier(0);
      mma(av[1], wv[1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // ---- stage the tile as [position][channel] fp32 (pitch 260 floats: the 64 lanes of
    // one store hit 64 different banks). All of LDS is free: every wave has passed B_nsl,
    // and every loader had drained its loads before it.
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FMW; ++i)
      if (i < nbw)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) stg[(16 * (mb0 + i) + 4 * kg + e) * CV_PITCH + 16 * (nb0 + j) + fi] = acc[i][j][e];
  }
  lds_barrier();
  // ---- write the tile's rows (output position p is row p of the output); a half tile
  // its 128 channels
  const float *stg = reinterpret_cast<const float *>(smem);
  if (a.out_bf16) {
    // 8 channels per thread, 32 (16) threads per row
    const int ch = hc < 0 ? (tid & 31) : 16 * hc + (tid & 15), sub = hc < 0 ? tid >> 5 : tid >> 4;
    const int step = hc < 0 ? NT / 32 : NT / 16;
    for (int m = sub; m < BM; m += step) {
      const int p = m0 + m;
      if (p < a.M) {
        const f32x4 v0 = *reinterpret_cast<const f32x4 *>(stg + m * CV_PITCH + 8 * ch);
        const f32x4 v1 = *reinterpret_cast<const f32x4 *>(stg + m * CV_PITCH + 8 * ch + 4);
        u32x4 pk;
        pk[0] = cvt_pk_bf16(v0[0], v0[1]);
        pk[1] = cvt_pk_bf16(v0[2], v0[3]);
        pk[2] = cvt_pk_bf16(v1[0], v1[1]);
        pk[3] = cvt_pk_bf16(v1[2], v1[3]);
        uint16_t *o = reinterpret_cast<uint16_t *>(a.out) + (int64_t)p * CV_BN + 8 * ch;
        *reinterpret_cast<u32x4 *>(o) = pk;
      }
    }
  } else {
    // 4 channels per thread, 64 (32) threads per row
    const int ch = hc < 0 ? (tid & 63) : 32 * hc + (tid & 31), sub = hc < 0 ? tid >> 6 : tid >> 5;
    const int step = hc < 0 ? NT / 64 : NT / 32;
    for (int m = sub; m < BM; m += step) {
      const int p = m0 + m;
      if (p < a.M) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + m * CV_PITCH + 4 * ch);
        float *o = reinterpret_cast<float *>(a.out) + (int64_t)p * CV_BN + 4 * ch;
        *reinterpret_cast<f32x4 *>(o) = v;
      }
    }
  }
}


// ------------------------------------------------------------------ weight gradient
// dW[o][tap][c] = sum_p dy[p][o] * x_pad[P(p) + r*(W+2) + s][c] over the tile's output
// positions p = (n, h, w), P(p) = (n (H+2) + h) (W+2) + w (Sec. 2.2: the tile's partial of
// the weight gradient, which the all-reduce over the domain completes). Both operands are
// position-major, so K = positions and both fragments come from k-row-major LDS slabs
// through the transpose read. A workgroup owns 256 output channels x 128 input channels
// of one tap over one range of output positions; the ranges are K splits whose fp32
// partials the split-K reduce adds in split order. Slabs of 64 positions, each row's
// padded-grid row P(p) kept incrementally by the loader lane that fetches it:
//  * waves 6-7 load the Delta_Y slab (64 positions x 256 channels, four 64-channel
//    quarters);
//  * waves 4-5 load the shifted activation slab (64 positions x 128 channels);
//  * waves 0-3 each accumulate 128 output channels x 64 input channels.
// Rows past the split's range read as zero (their loads are out of range).
struct CwArgs {
  const uint16_t *x;    // x_pad [N][H+2][W+2][Ci]
  const uint16_t *dy;   // interior start of dy_pad: dy_pad + ((W+2) + 1) * Co
  float *partial;       // [split][Co][ldp]: element (tap*Ci + c, o) at o*ldp + tap*Ci + c
  int64_t ldp, sstride;
  int H, W, Ci, Co;
  int M, k_split, splits, tiles;  // output positions N*H*W; tiles = 9 * Ci / 128
  int Mp;                         // padded-grid rows up to the last output position's
};

constexpr int CW_XSLOT = 64 * 256;   // 16 KB: 64 positions x 128 channels
constexpr int CW_DSLOT = 64 * 512;   // 32 KB: 64 positions x 256 channels
constexpr int CW_NX = 4, CW_ND = 3;  // ring slots
constexpr int CW_PITCH = 128 + 4;    // staging row pitch in floats

// Output position p as (h, w) and its padded-grid row P(p); the step to position p + 64
// without a division (the rows that wrap past an image row or an image are counted).
__device__ __forceinline__ void cw_row_init(const CwArgs &a, int p, int *h, int *w, int *P) {
  const int HW = a.H * a.W, n = p / HW, rem = p - n * HW;
  *h = rem / a.W;
  *w = rem - *h * a.W;
  *P = (n * (a.H + 2) + *h) * (a.W + 2) + *w;
}
__device__ __forceinline__ void cw_row_next(const CwArgs &a, int *h, int *w, int *P) {
  const int Wp = a.W + 2, dh = 64 / a.W, dw = 64 - dh * a.W;
  *w += dw;
  *h += dh;
  *P += dh * Wp + dw;
  if (*w >= a.W) {
    *w -= a.W;
    ++*h;
    *P += 2;
  }
  while (*h >= a.H) {
    *h -= a.H;
    *P += 2 * Wp;
  }
}

__global__ void __launch_bounds__(512, 1) conv_wg_kernel(CwArgs a) {
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int DRING = CW_ND * CW_DSLOT, XRING = CW_NX * CW_XSLOT;
  __shared__ __attribute__((aligned(1024))) char smem[DRING + XRING];
  static_assert(DRING + XRING <= 160 * 1024, "LDS");
  static_assert(256 * CW_PITCH * 4 <= DRING + XRING, "staging");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // padded to a multiple of 8: the tiles of one split (which read the same positions) run
  // on one XCD
  const int G = gridDim.x;
  const int b = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  if (b >= a.tiles * a.splits) return;
  const int split = b / a.tiles, tile = b - split * a.tiles;
  const int tap = tile / (a.Ci / 128), c0 = (tile - tap * (a.Ci / 128)) * 128;
  const int klo = split * a.k_split, krange = min(a.M, klo + a.k_split) - klo;
  const int nsl = krange > 0 ? (krange + 63) / 64 : 0;
  const int Wp = a.W + 2;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t ldsd = lds0, ldsx = lds0 + DRING;

  if (wave >= 6) {
    // ---------------------------------------------------- Delta_Y loaders (6, 7)
    // blocks 16dw..16dw+15 of a slot: quarter h = blk/8, k-rows 8(blk%8)..+7
    const int dw = wave - 6;
    const i32x4 rd = buf_rsrc(a.dy, (uint32_t)((int64_t)a.Mp * a.Co * 2));
    // the wave's blocks cover quarters 2dw, 2dw+1 of the same 8 row groups g (k-rows
    // 8g + lane/8)
    uint32_t col[2][8];
    int hh[8], ww[8], pp[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int r = 8 * g + (lane >> 3);
      const int c = (lane & 7) ^ cv_swz_tr(r);
      col[0][g] = (uint32_t)((64 * (2 * dw) + 8 * c) * 2);
      col[1][g] = (uint32_t)((64 * (2 * dw + 1) + 8 * c) * 2);
      cw_row_init(a, klo + r, &hh[g], &ww[g], &pp[g]);
    }
    auto issue = [&](int S) {
      const uint32_t slot = ldsd + (uint32_t)((S % CW_ND) * CW_DSLOT);
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        const int r = 8 * g + (lane >> 3);
        const bool ok = S < nsl && S * 64 + r < krange;
        const uint32_t off = (uint32_t)pp[g] * (uint32_t)(a.Co * 2);
#pragma unroll
        for (int hq = 0; hq < 2; ++hq)
          dma16(rd, ok ? off + col[hq][g] : OOB, slot + (uint32_t)((2 * dw + hq) * CV_QSLOT + g * 1024));
        cw_row_next(a, &hh[g], &ww[g], &pp[g]);
      }
    };
#pragma unroll
    for (int S = 0; S < CW_ND - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<16 * (CW_ND - 2)>();  // slab S landed: B_S
      issue(S + CW_ND - 1);            // into the slot of S-1
    }
    vm_barrier<0>();
  } else if (wave >= 4) {
    // --------------------------------------------------- activation loaders (4, 5)
    // quarter h = blk/8 (channels c0 + 64h ..), k-rows 8(blk%8).. of positions shifted by tap
    const int xw = wave - 4;
    const int r3 = tap / 3, s3 = tap - 3 * r3, shift = r3 * Wp + s3;
    const i32x4 rx = buf_rsrc(a.x, (uint32_t)((int64_t)(a.Mp + 2 * Wp + 2) * a.Ci * 2));
    // block q of the wave's quarter: k-rows 8q + lane/8
    uint32_t col[8];
    int hh[8], ww[8], pp[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = 8 * q + (lane >> 3);
      const int c = (lane & 7) ^ cv_swz_tr(r);
      col[q] = (uint32_t)((c0 + 64 * xw + 8 * c) * 2);
      cw_row_init(a, klo + r, &hh[q], &ww[q], &pp[q]);
    }
    auto issue = [&](int S) {
      const uint32_t slot = ldsx + (uint32_t)((S % CW_NX) * CW_XSLOT) + (uint32_t)(xw * CV_QSLOT);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int r = 8 * q + (lane >> 3);
        const bool ok = S < nsl && S * 64 + r < krange;
        const uint32_t off = (uint32_t)(pp[q] + shift) * (uint32_t)(a.Ci * 2);
        dma16(rx, ok ? off + col[q] : OOB, slot + (uint32_t)(q * 1024));
        cw_row_next(a, &hh[q], &ww[q], &pp[q]);
      }
    };
#pragma unroll
    for (int S = 0; S < CW_NX - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<8 * (CW_NX - 2)>();  // slab S landed: B_S
      issue(S + CW_NX - 1);           // into the slot of S-1
    }
    vm_barrier<0>();
  } else {
    // --------------------------------------------------------------- MMA group
    // wave (wm, wn): output channels 128wm.. (Delta_Y quarters 2wm, 2wm+1), input channels
    // 64wn.. (activation quarter wn)
    constexpr int FM = 8;
    const int fi = lane & 15, kg = lane >> 4;
    const int wm = wave & 1, wn = wave >> 1;
    const int r = 8 * kg + (fi >> 2);
    uint32_t fa[FM], fx[4];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int mb = 8 * wm + i, h = mb >> 2, ib = mb & 3;
      const int c = (2 * ib + ((fi >> 1) & 1)) ^ cv_swz_tr(r);
      fa[i] = (uint32_t)(h * CV_QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = (2 * j + ((fi >> 1) & 1)) ^ cv_swz_tr(r);
      fx[j] = (uint32_t)(wn * CV_QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
    }
    f32x4 acc[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto tr8 = [&](uint32_t addr) {
      lds_i16x4 *p = (lds_i16x4 *)(uintptr_t)addr;
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p + 4 * 128 / 8);
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    bf16x8 dv[2][FM], xv[2][4];
    auto read = [&](uint32_t ds, uint32_t xs, int s, bf16x8 (&dd)[FM], bf16x8 (&xd)[4]) {
#pragma unroll
      for (int i = 0; i < FM; ++i) dd[i] = tr8(ds + fa[i] + (uint32_t)(s * 4096));
#pragma unroll
      for (int j = 0; j < 4; ++j) xd[j] = tr8(xs + fx[j] + (uint32_t)(s * 4096));
    };
    // One 32-k step: its 32 MFMAs in eight groups (row block g against the four column
    // blocks), with the next step's twelve fragments (24 transpose reads) read two per group
    // in the first six, the column blocks and the first row blocks first (the next step's
    // first groups use them). Reading all 24 ahead of the MFMAs made every step wait for ten
    // of them: the LDS counter tracks at most 15 operations, so the wait that the older
    // fragments need also covers the oldest of the new reads. The last two groups' MFMAs
    // cover the reads before the next step or the slab barrier.
    auto step = [&](const bf16x8 (&df)[FM], const bf16x8 (&xf)[4], uint32_t dsn, uint32_t xsn, int sn,
                    bf16x8 (&dd)[FM], bf16x8 (&xd)[4]) {
#pragma unroll
      for (int g = 0; g < FM; ++g) {
        if (g < 6) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int f = 2 * g + h;
            if (f < 4) xd[f] = tr8(xsn + fx[f] + (uint32_t)(sn * 4096));
            else dd[f - 4] = tr8(dsn + fa[f - 4] + (uint32_t)(sn * 4096));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[g][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(df[g], xf[j], acc[g][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    uint32_t ds = ldsd, xs = ldsx;
    if (nsl > 0) {
      lds_barrier();  // B_0
      read(ds, xs, 0, dv[0], xv[0]);
    }
    for (int S = 0; S < nsl; ++S) {
      step(dv[0], xv[0], ds, xs, 1, dv[1], xv[1]);
      lds_barrier();  // B_{S+1}
      ds = ldsd + (uint32_t)(((S + 1) % CW_ND) * CW_DSLOT);
      xs = ldsx + (uint32_t)(((S + 1) % CW_NX) * CW_XSLOT);
      step(dv[1], xv[1], ds, xs, 0, dv[0], xv[0]);  // past the last slab this reads a spent slot, unused
    }
    if (nsl == 0) lds_barrier();  // the loaders' B_0 (they pass vm_barrier<0> once)
    // ---- stage the tile as [output channel][input channel] fp32
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          stg[(16 * (8 * wm + i) + 4 * kg + e) * CW_PITCH + 16 * (4 * wn + j) + fi] = acc[i][j][e];
  }
  lds_barrier();
  // ---- partial tile out: 256 rows of 128 floats (512 B), device-scope stores
  const float *stg = reinterpret_cast<const float *>(smem);
  float *dst = a.partial + (int64_t)split * a.sstride + tap * a.Ci + c0;
  const __amdgpu_buffer_rsrc_t prs =
      __builtin_amdgcn_make_buffer_rsrc(dst, 0, (int)(((int64_t)(a.Co - 1) * a.ldp + 128) * 4), BUF_DW3);
  const int ch = tid & 31, sub = tid >> 5;
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int o = 16 * p + sub;
    const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + o * CW_PITCH + 4 * ch);
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), prs, (uint32_t)((o * a.ldp + 4 * ch) * 4), 0, 16);
  }
}

}  // namespace

bool conv_nt_fits(int pass, int N, int H, int W, int Ci, int Co, const void *act, const void *w, const void *out) {
  if (opt(IMBD_OPT_CONV_NT) == 0) return false;  // the tiled GEMM template instead
  const int Cn = pass == 1 ? Co : Ci, Ck = pass == 1 ? Ci : Co;
  auto al = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) % 16) == 0; };
  const int64_t rows = (int64_t)N * (H + 2) * (W + 2) + 2 * (W + 2) + 2 + CV_BM;
  return (pass == 1 || pass == 2) && N >= 1 && H >= 1 && W >= 1 && Cn == CV_BN && Ck >= 64 && Ck % 64 == 0 &&
         al(act) && al(w) && al(out) && rows * Ck * 2 < ((int64_t)1 << 31) &&
         (int64_t)9 * Ci * Co * 2 < ((int64_t)1 << 31);
}

bool conv_wg_fits(int N, int H, int W, int Ci, int Co, const void *x, const void *dy, const void *dw) {
  if (opt(IMBD_OPT_CONV_NT) == 0) return false;
  auto al = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) % 16) == 0; };
  const int64_t rows = (int64_t)N * (H + 2) * (W + 2) + 2 * (W + 2) + 2 + 64;
  return N >= 1 && H >= 1 && W >= 1 && Co == 256 && Ci >= 128 && Ci % 128 == 0 && al(x) && al(dy) && al(dw) &&
         rows * (Ci > Co ? Ci : Co) * 2 < ((int64_t)1 << 31);
}

void conv_wg_plan(int N, int H, int W, int Ci, int *splits, int *k_split) {
  const int64_t M = (int64_t)N * H * W;
  const int tiles = 9 * Ci / 128;
  int s = 256 / tiles;
  if (s < 1) s = 1;
  int ks = (int)((M + s - 1) / s + 63) / 64 * 64;
  if (ks < 64) ks = 64;
  *k_split = ks;
  *splits = (int)((M + ks - 1) / ks);
}

int run_conv_wg(int N, int H, int W, int Ci, int Co, const void *x, const void *dy_pad, float *partial,
                int64_t ldp, int64_t sstride, hipStream_t s) {
  CwArgs a;
  a.x = reinterpret_cast<const uint16_t *>(x);
  a.dy = reinterpret_cast<const uint16_t *>(dy_pad) + (int64_t)(W + 3) * Co;
  a.partial = partial;
  a.ldp = ldp;
  a.sstride = sstride;
  a.H = H;
  a.W = W;
  a.Ci = Ci;
  a.Co = Co;
  a.M = N * H * W;
  a.Mp = (int)((int64_t)(N - 1) * (H + 2) * (W + 2) + (int64_t)(H - 1) * (W + 2) + W);
  conv_wg_plan(N, H, W, Ci, &a.splits, &a.k_split);
  a.tiles = 9 * Ci / 128;
  const int grid = (a.tiles * a.splits + 7) / 8 * 8;
  {
    LaunchTimer t(IMBD_K_CONV_WGRAD, 0, s);
    hipLaunchKernelGGL(conv_wg_kernel, dim3(grid), dim3(512), 0, s, a);
  }
  return check_launch("conv_wg");
}

int run_conv_nt(int pass, int N, int H, int W, int Ci, int Co, const void *act, const void *w, void *out,
                int out_dtype, hipStream_t s) {
  CvArgs a;
  a.act = reinterpret_cast<const uint16_t *>(act);
  a.w = reinterpret_cast<const uint16_t *>(w);
  a.out = out;
  a.out_bf16 = out_dtype == IMBD_BF16 ? 1 : 0;
  a.N = N;
  a.H = H;
  a.W = W;
  a.Ck = pass == 1 ? Ci : Co;
  a.Cw = Ci;
  a.M = N * H * W;
  // One workgroup per CU (160 KB of LDS): past one round, the tiles of a short last round
  // run as 128-channel halves on twice as many CUs, which ends that round sooner. The tile
  // height (128 or 112 positions) is the one whose rounds (a round of halves counted as
  // half a round) take fewer position blocks per CU: on the 32 x 56 x 56 grid, 784 tiles
  // of 128 (3 rounds and a short one) against 896 of 112 (3 rounds and a full round of
  // halves).
  auto plan = [&](int fm, int *tiles, int *last, bool *halves) {
    *tiles = (a.M + 16 * fm - 1) / (16 * fm);
    *last = *tiles > CV_CUS ? *tiles % CV_CUS : 0;
    *halves = *last > 0 && 2 * *last <= CV_CUS;
    const int rounds = (*tiles + CV_CUS - 1) / CV_CUS;
    return (*halves ? 2 * rounds - 1 : 2 * rounds) * fm;  // in half rounds x blocks
  };
  int t8, l8, t7, l7;
  bool h8, h7;
  const int c8 = plan(8, &t8, &l8, &h8), c7 = plan(7, &t7, &l7, &h7);
  const int o = opt(IMBD_OPT_CONV_NT);
  const int fm = o == 2 ? 8 : o == 3 ? 7 : (c7 < c8 ? 7 : 8);
  a.tiles = fm == 8 ? t8 : t7;
  const int last = fm == 8 ? l8 : l7;
  const bool halves = fm == 8 ? h8 : h7;
  a.tfull = halves ? a.tiles - last : a.tiles;
  a.gfull = (a.tfull + 7) / 8 * 8;
  const int grid = a.gfull + (halves ? 2 * last : 0);
  {
    LaunchTimer t(pass == 1 ? IMBD_K_CONV_FWD : IMBD_K_CONV_DGRAD, 0, s);
    if (pass == 1) {
      if (fm == 8) hipLaunchKernelGGL((conv_nt_kernel<false, 8>), dim3(grid), dim3(768), 0, s, a);
      else hipLaunchKernelGGL((conv_nt_kernel<false, 7>), dim3(grid), dim3(768), 0, s, a);
    } else {
      if (fm == 8) hipLaunchKernelGGL((conv_nt_kernel<true, 8>), dim3(grid), dim3(768), 0, s, a);
      else hipLaunchKernelGGL((conv_nt_kernel<true, 7>), dim3(grid), dim3(768), 0, s, a);
    }
  }
  return check_launch("conv_nt");
}

}  // namespace imbd
