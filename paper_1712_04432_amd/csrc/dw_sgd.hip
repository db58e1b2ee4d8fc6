// Fused weight gradient + SGD update of one fully connected layer, bf16 operands.
//
// Delta_W = Delta_Y^T X (Sec. 1: the third product of a layer's backward pass; K = the
// batch, both operands stored with the sample as the row index) with the update of
// Eq. (1) applied in place: w -= lr * alpha * Delta_W (alpha = 1/B), w16 = bf16(w), and
// the bias gradient (column sums of Delta_Y) applied the same way.
//
// The update streams 10 bytes per weight through HBM (fp32 master read and written, bf16
// copy written) while the product itself is small (K = batch), so the kernel is built
// around that stream. Persistent workgroups, one per CU, of eight waves in two groups:
//  * waves 0-3 (MMA group) keep the workgroup's Delta_Y column block resident in LDS
//    (the grid is a multiple of the column-block count, so all tiles of a workgroup
//    share it), stream 32-sample slabs of X through a four-slot LDS ring with buffer
//    loads that write LDS directly (out-of-range lanes read as zero), gather MFMA
//    fragments with the LDS transpose read and accumulate a 128 x 128 tile in registers;
//  * waves 4-7 (update group) finish the previous tile out of a separate LDS staging
//    buffer: read-modify-write of the fp32 masters, bf16 copy.
// Each wave keeps its own memory counter, so the groups do not wait on each other's
// traffic; they meet at one barrier per slab and two per tile (staging free / full).
// Past 256 samples the Delta_Y block no longer fits beside the X ring and the staging
// buffer: Delta_Y then streams through a ring of its own in the X slabs' layout (the
// streamed variant), or, with IMBD_DW_STREAM=0, the resident block is reloaded per
// 256-sample chunk. On the VGG FC stack at B = 512 the streamed update takes the step
// from 623 to 568 us.

#include <hip/hip_ext.h>
#include <stdlib.h>

#include <type_traits>

#include "cdna4.h"
#include "skinny_reduce.h"

namespace imbd {
namespace {

// Cache policies (the aux operand of the raw buffer builtins: 2 = nt, 16 = sc1).
//  * fp32 master loads: non-temporal. The masters are touched once per step; keeping them
//    out of the caches leaves the bf16 copy this kernel writes (which the next step's
//    forward product reads) resident in the 256 MB MALL. In the AlexNet FC step that took
//    the layer-1 forward from 39 to 29 us.
//  * fp32 master stores: non-temporal and device scope (write-through past the XCD's L2),
//    for the same reason, and so that the L2s hold no dirty lines for the end-of-kernel
//    writeback, which otherwise delays the next launch by ~5 us.
//  * bf16 copy stores: device scope, allocated in the MALL for the next forward.
// Together the stores take the AlexNet FC step from 245 to 233 us, although the layer-1
// launch itself runs ~2 us longer than with default stores.
constexpr int CPOL_MASTER_LD = 2;
constexpr int CPOL_MASTER_ST = 2 | 16;
constexpr int CPOL_COPY_ST = 16;

constexpr int KMAX_SAMPLES = 256;  // samples of the Delta_Y block resident at a time

struct DwArgs {
  const uint16_t *X;   // [K][ldx]  rows are samples, M = d_in columns
  const uint16_t *DY;  // [K][lddy] N = d_out columns
  int64_t ldx, lddy;
  int M, N, K;
  float *w;            // [N][ldw] fp32 masters (read-modify-write)
  int64_t ldw;
  uint16_t *w16;       // [N][ldw16] bf16 copy
  int64_t ldw16;
  float lr, alpha;
  int db_mode;         // 0 none, 1 store db_out, 2 bias -= bias_lr * db
  float *db_out, *bias;
  float db_alpha, bias_lr;
  int tiles_m, tiles_n;
  int spread;          // row-block order (see the kernel)
  SkReduceArgs tail;   // a skinny product's split-K reduce carried by this launch
  int64_t tail_items;  // its items (0: none)
};

// STREAM (batches past 256): Delta_Y travels in 32-sample slabs through a ring of its own,
// beside the X slabs and with the same row layout, instead of the resident block; the
// update group spreads its chunks over all of a tile's slab barriers.
template <bool STREAM>
__global__ void __launch_bounds__(512, 1) dw_sgd_kernel(DwArgs a) {
  constexpr int BM = 128, BN = 128, BK = 32, NS = 4, NTM = 256, NTU = 256, KMAX = 256;
  constexpr int ROWB = 256;                 // bytes per LDS row: 128 bf16 columns
  constexpr int XSLAB = BK * ROWB;          // 8 KB X slab
  constexpr int DYB = STREAM ? NS * XSLAB : KMAX * ROWB;  // Delta_Y ring, or the 64 KB resident block
  constexpr int FM = 4, FN = 4;             // 16 x 16 fragments per wave (64 x 64)
  constexpr int RPP = NTU / (BM / 4), PASSES = BN / RPP;
  constexpr int CHUNKS = 8, CP = PASSES / CHUNKS;
  constexpr int DMA_PER_SLAB = STREAM ? 4 : 2;  // per wave: 2 x 1 KB of X (and of Delta_Y)
  constexpr uint32_t OOB = 0x80000000u;
  // [X ring][Delta_Y ring or resident block][staging, 128 x 128 fp32 with 16-byte units swizzled]
  __shared__ __attribute__((aligned(1024))) char smem[NS * XSLAB + DYB + BN * BM * 4];
  char *dyres = smem + NS * XSLAB;
  float *stg = reinterpret_cast<float *>(dyres + DYB);

  const int tid = threadIdx.x;
  const int tiles = a.tiles_m * a.tiles_n;
  const int G = gridDim.x;  // a multiple of tiles_n: every tile of a workgroup has the same column block
  int b = blockIdx.x;
  if ((G & 7) == 0) b = (b & 7) * (G >> 3) + (b >> 3);
  // The gpb workgroups of a column block share its row blocks; the k-th row block of the
  // one with index grp is gpb*k + (grp + k) % gpb, so that every workgroup visits every
  // column offset modulo gpb row blocks. (A fixed offset per workgroup left some of them
  // on slow address classes: layer-1 finish times spread 53-73 us, now 62-70 us.) The gpb
  // row blocks in flight at once are then adjacent, one 4 KB run of each master row; when
  // the row pitch is a multiple of 8 KB those runs fall in at most two of the four 4 KB
  // pages modulo 16 KB, and the update streams slower (4096 x 4096: 41 us). With spread
  // set, the k-th row block is full*((grp + k) % gpb) + k instead: the blocks in flight
  // are full blocks apart (34 us). The rem extra blocks come last either way.
  const int gpb = G / a.tiles_n, grp = b / a.tiles_n;
  const int full = a.tiles_m / gpb, rem = a.tiles_m % gpb;
  const int nmy = b < tiles ? full + ((grp + full) % gpb < rem ? 1 : 0) : 0;
  const int TK = (a.K + BK - 1) / BK;
  // Batches past 256 samples without streaming: the Delta_Y block holds one chunk of 256
  // samples (8 slabs) at a time and is reloaded whenever the next slab starts another
  // chunk (the first of every tile included), 2 barriers per reload.
  const int nch = (TK + 7) / 8;
  const bool multi = !STREAM && nch > 1;
  auto reloads = [&](int it) { return multi ? nch - (it == nmy - 1 ? 1 : 0) : 0; };
  const int n0 = (b % a.tiles_n) * BN;
  auto tile_m0 = [&](int it) {
    const int r = (grp + it) % gpb;
    return (it < full && a.spread ? r * full + it : gpb * it + r) * BM;
  };

  if (tid < NTM) {
    // ------------------------------------------------------------------ MMA group
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm0 = (wave & 1) * 64, wn0 = (wave >> 1) * 64;
    // Rows past the batch fall outside the descriptors' ranges and read as zero.
    const i32x4 rx = buf_rsrc(a.X, (uint32_t)(a.K * a.ldx * 2));
    const i32x4 rdy = buf_rsrc(a.DY, (uint32_t)(a.K * a.lddy * 2));
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
    const uint32_t ldy = lds0 + NS * XSLAB;
    // LDS row layout (X slabs and the Delta_Y block alike): row r (sample r of the slab or
    // block) holds 128 columns as 16 chunks of 16 bytes, chunk c stored at position
    // c ^ swz(r), swz(r) = 2*(r & 3) + 8*((r >> 3) & 1): the 16 rows that one transpose
    // read touches then cover every bank exactly twice. A wave's 1 KB load covers 4 rows:
    // lane i fills row 4q + i/16, stored chunk i%16, from source chunk (i%16) ^ swz(row).
    const int dr = lane >> 4, dc = lane & 15;
    // resident Delta_Y block (samples 256 ch .. 256 ch + 255): wave w loads rows
    // 64w..64w+63, 16 loads of 4 rows
    auto load_dy = [&](int ch) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int r = 64 * wave + 4 * q + dr;
        const int scol = 8 * (dc ^ (2 * dr + 8 * ((q >> 1) & 1)));  // source column of the lane's chunk
        const uint32_t off = n0 + scol < a.N ? (uint32_t)(((KMAX * ch + r) * a.lddy + n0 + scol) * 2) : OOB;
        dma16(rdy, off, __builtin_amdgcn_readfirstlane(ldy + (uint32_t)((64 * wave + 4 * q) * ROWB)));
      }
    };
    if constexpr (!STREAM) load_dy(0);
    // X slabs (and in STREAM mode Delta_Y slabs, same layout): wave w fills rows 8w..8w+7
    // of each slab (two 4-row loads)
    const int dcol = 8 * (dc ^ (2 * dr + 8 * (wave & 1)));
    const uint32_t xstep = (uint32_t)(BK * a.ldx * 2), xh = (uint32_t)(4 * a.ldx * 2);
    const uint32_t ystep = (uint32_t)(BK * a.lddy * 2), yh = (uint32_t)(4 * a.lddy * 2);
    // the workgroup's Delta_Y columns are the same for all its tiles
    const uint32_t yb0 = n0 + dcol < a.N ? (uint32_t)(((8 * wave + dr) * a.lddy + n0 + dcol) * 2) : OOB;
    int i_it = 0, i_ks = 0;
    uint32_t i_slot = 0, xk = 0, xb = OOB, yb = OOB;
    auto i_tile = [&]() {
      xb = OOB;
      yb = OOB;
      if (i_it < nmy) {
        const int m0 = tile_m0(i_it);
        if (m0 + dcol < a.M) xb = (uint32_t)(((8 * wave + dr) * a.ldx + m0 + dcol) * 2);
        yb = yb0;
      }
      xk = 0;
    };
    auto issue = [&]() {
      const uint32_t dst = lds0 + i_slot + (uint32_t)(8 * wave * ROWB);
      dma16(rx, xb + xk, dst);
      dma16(rx, xb + xh + xk, dst + 4 * ROWB);
      if constexpr (STREAM) {
        const uint32_t yk = (uint32_t)i_ks * ystep;
        dma16(rdy, yb == OOB ? OOB : yb + yk, dst + (uint32_t)(NS * XSLAB));
        dma16(rdy, yb == OOB ? OOB : yb + yh + yk, dst + (uint32_t)(NS * XSLAB) + 4 * ROWB);
      }
      i_slot = i_slot + XSLAB == NS * XSLAB ? 0u : i_slot + XSLAB;
      xk += xstep;
      if (++i_ks == TK) {
        i_ks = 0;
        ++i_it;
        i_tile();
      }
    };

    // Fragment reads: lane (kg = lane/16, s = lane%16) addresses row 8kg + s/4 (+4 for
    // the second half of its 8 samples) at column c0 + 4*(s%4); the transpose read then
    // hands lane s the 4 consecutive samples of column c0 + s.
    const int kg = lane >> 4, fs = lane & 15;
    const int fsw = 2 * (fs >> 2) + 8 * (kg & 1);
    const uint32_t frow = (uint32_t)((8 * kg + (fs >> 2)) * ROWB + 8 * (fs & 1));
    uint32_t fa_off[FM], fb_off[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa_off[i] = lds0 + frow + (uint32_t)((((wm0 >> 3) + 2 * i + ((fs >> 1) & 1)) ^ fsw) * 16);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb_off[j] = ldy + frow + (uint32_t)((((wn0 >> 3) + 2 * j + ((fs >> 1) & 1)) ^ fsw) * 16);

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto read_slab = [&](uint32_t slot, uint32_t krow, i16x4 (&xa)[FM][2], i16x4 (&xb2)[FN][2]) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        lds_i16x4 *p = (lds_i16x4 *)(uintptr_t)(fa_off[i] + slot);
        xa[i][0] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
        xa[i][1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p + 4 * ROWB / 8);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        lds_i16x4 *p = (lds_i16x4 *)(uintptr_t)(fb_off[j] + krow);
        xb2[j][0] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
        xb2[j][1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p + 4 * ROWB / 8);
      }
    };
    auto mma = [&](const i16x4 (&xa)[FM][2], const i16x4 (&xb2)[FN][2]) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, __builtin_shufflevector(xa[i][0], xa[i][1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const bf16x8 bv = __builtin_bit_cast(bf16x8, __builtin_shufflevector(xb2[j][0], xb2[j][1], 0, 1, 2, 3, 4, 5, 6, 7));
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[i][j], 0, 0, 0);
        }
      }
    };
    // Staging layout: element (n, m) at float n*128 + 4*((m/4) ^ (n % 32)) + m%4.
    auto handoff = [&]() {
      lds_barrier();  // staging free (the update group is done with the previous tile)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int n = wn0 + j * 16 + fs, m4 = (wm0 >> 2) + i * 4 + kg;
          *reinterpret_cast<f32x4 *>(stg + n * BM + 4 * (m4 ^ (n & 31))) = acc[i][j];
          acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      lds_barrier();  // staging full
    };

    const int total = nmy * TK;
    i_tile();
#pragma unroll
    for (int s = 0; s < NS; ++s) issue();
    vm_barrier<(NS - 1) * DMA_PER_SLAB>();  // Delta_Y block and slab 0 landed

    // Bias gradient: the column sums of the resident Delta_Y block, once per column block,
    // by the workgroup with index 0 in the block's group (it always has a tile). Wave w
    // sums rows 64w..64w+63: lane l reads 16-byte chunk l%16 (columns 8(l%16)..+7) of rows
    // 64w + l/16 + 4i, i < 16, and the four row phases are added across lanes. The waves'
    // sums go to the staging buffer (unused until the first tile is handed off) and wave 0
    // adds them in wave order after the next slab barrier, which every wave reaches only
    // after writing its sums.
    bool bias_pending = !STREAM && a.db_mode != 0 && b < tiles && grp == 0;
    if (bias_pending) {
      const int j = lane & 15, q = lane >> 4;
      float cs[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) cs[e] = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = 64 * wave + q + 4 * i;
        const int sw = 2 * (r & 3) + 8 * ((r >> 3) & 1);
        const u32x4 v = *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(ldy + (uint32_t)(r * ROWB + ((j ^ sw) << 4)));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          cs[2 * e] += bf16_to_f32((uint16_t)(v[e] & 0xffffu));
          cs[2 * e + 1] += bf16_to_f32((uint16_t)(v[e] >> 16));
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        cs[e] += __shfl_xor(cs[e], 16, 64);
        cs[e] += __shfl_xor(cs[e], 32, 64);
      }
      if (q == 0) {
        float *dst = stg + wave * BN + 8 * j;
        *reinterpret_cast<f32x4 *>(dst) = f32x4{cs[0], cs[1], cs[2], cs[3]};
        *reinterpret_cast<f32x4 *>(dst + 4) = f32x4{cs[4], cs[5], cs[6], cs[7]};
      }
    }
    auto bias_finish = [&]() {
      if (wave == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int c = lane + 64 * h, n = n0 + c;
          const float sum = stg[c] + stg[BN + c] + stg[2 * BN + c] + stg[3 * BN + c];
          if (n < a.N) {
            const float g = a.db_alpha * sum;
            if (a.db_mode == 1) a.db_out[n] = g;
            else a.bias[n] = fmaf(-a.bias_lr, g, a.bias[n]);
          }
        }
      }
      bias_pending = false;
    };

    int c_ks = 0, c_it = 0;
    uint32_t c_slot = 0, c_krow = 0;
    i16x4 fa[FM][2], fb[FN][2], ga[FM][2], gb[FN][2];
    // Delta_Y fragments: the resident block's k-rows of the slab, or the slab's own slot
    auto yrow = [&]() { return STREAM ? c_slot : c_krow; };
    read_slab(c_slot, yrow(), fa, fb);
    auto step = [&](const i16x4 (&ca)[FM][2], const i16x4 (&cb)[FN][2], i16x4 (&na)[FM][2], i16x4 (&nb)[FN][2]) {
      // Slab s+1 landed once at most the later NS-2 slabs' loads are outstanding; every
      // wave has read slab s, so its slot takes the next slab in line.
      vm_barrier<(NS - 2) * DMA_PER_SLAB>();
      if (bias_pending) bias_finish();  // before any handoff can reuse the staging buffer
      issue();
      c_slot = c_slot + XSLAB == NS * XSLAB ? 0u : c_slot + XSLAB;
      const bool tile_end = ++c_ks == TK;
      if (tile_end) c_ks = 0;
      c_krow = (uint32_t)((c_ks & 7) * BK * ROWB);
      // The MFMAs of slab s go first: the transpose reads of slab s+1 then run while
      // the matrix pipe works, with no wait between them.
      mma(ca, cb);
      __builtin_amdgcn_sched_barrier(0);
      if (multi && (c_ks & 7) == 0 && !(tile_end && c_it == nmy - 1)) {
        lds_barrier();        // every wave is done reading the current chunk
        load_dy(c_ks >> 3);   // the next slab's chunk
        vm_barrier<0>();      // landed in every wave
      }
      read_slab(c_slot, yrow(), na, nb);
      if (tile_end) {
        ++c_it;
        handoff();
      }
    };
    // Two steps per trip so that the fragment sets alternate without copies.
    for (int s = 0; s < total; s += 2) {
      step(fa, fb, ga, gb);
      if (s + 1 >= total) break;
      step(ga, gb, fa, fb);
    }
    // Drain the ring's trailing loads (they target slots nobody reads again).
    asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
    // The reduce this launch carries (another layer's Delta_X partials into its Delta_Y),
    // spread over the workgroups' MMA waves while their update waves finish the last tile.
    for (int64_t t = (int64_t)blockIdx.x * NTM + tid; t < a.tail_items; t += (int64_t)gridDim.x * NTM)
      sk_reduce_item<true, 1>(a.tail, t);
  } else {
    // --------------------------------------------------------------- update group
    // Branch-free buffer loads and stores on per-tile descriptors. Rows past the matrix
    // fall outside the descriptor's range and a lane whose columns are past it gets an
    // out-of-range base, so the hardware drops those stores and reads those loads as
    // zero; with no conditional memory operation the compiler counts each master load
    // exactly and never drains the store stream. Iteration it finishes tile it-1 (at
    // it = 0 every store is dropped: empty range) while loading the masters of tile it,
    // pass by pass, spread over the tile's slab barriers; the last iteration runs after
    // the MMA group is done and passes no barrier.
    const int et = tid - NTM;
    const int er = et / (BM / 4), ec = (et % (BM / 4)) * 4;
    const float c = -a.lr * a.alpha;
    const uint32_t wrow = (uint32_t)(RPP * a.ldw * 4), hrow = (uint32_t)(RPP * a.ldw16 * 2);
    // staging row pp*RPP + er, 16-byte unit (ec/4) ^ ((pp*RPP + er) % 32): four lane bases
    uint32_t sb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      sb[q] = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)stg + (uint32_t)(er * BM * 4 + (((ec >> 2) ^ (er + 8 * q)) << 4));
    const int nrows = min(BN, a.N - n0);
    // A master vector is loaded CHUNKS - LAG chunks (slab barriers) before the pass that
    // needs it: far enough ahead to cover the HBM latency, near enough that the CU's queue
    // of outstanding requests stays short and the operand loads are not stuck behind it.
    // The first two iterations are peeled (PH 0 and 1, the rest PH 2) so that tile 0's
    // masters are all loaded during its product, chunk ch at chunk ch of iteration 0, with
    // no conditional load in any iteration: iteration 0 stores nothing, iteration 1 skips
    // the loads of tile 0's second half, which are already in the registers.
    constexpr int LAG = 4;
    f32x4 wold[PASSES];
    int pm0 = 0;
    lds_barrier();  // matches the MMA group's "Delta_Y block and slab 0 landed"
    auto iteration = [&](auto phase, int it) {
      constexpr int PH = decltype(phase)::value;
      const bool have = it < nmy;
      const int m0 = have ? tile_m0(it) : 0;
      // rn: tile it (masters for passes loaded late in this iteration), rq: tile it-1
      // (loaded early in this iteration), rp/rh: tile it-1 (finished in this iteration)
      const float *wn_base = a.w + (int64_t)n0 * a.ldw + m0;
      const float *wq_base = a.w + (int64_t)n0 * a.ldw + pm0;
      float *wp_base = a.w + (int64_t)n0 * a.ldw + pm0;
      uint16_t *hp_base = a.w16 + (int64_t)n0 * a.ldw16 + pm0;
      const int rn_rows = have ? nrows : 0, rp_rows = it > 0 ? nrows : 0;
      const __amdgpu_buffer_rsrc_t rn = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(wn_base), 0, rn_rows * (int)a.ldw * 4, BUF_DW3);
      const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(wq_base), 0, rp_rows * (int)a.ldw * 4, BUF_DW3);
      const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(wp_base, 0, rp_rows * (int)a.ldw * 4, BUF_DW3);
      const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(hp_base, 0, rp_rows * (int)a.ldw16 * 2, BUF_DW3);
      const uint32_t vp = pm0 + ec < a.M ? (uint32_t)(er * a.ldw + ec) * 4u : OOB;
      const uint32_t vh = pm0 + ec < a.M ? (uint32_t)(er * a.ldw16 + ec) * 2u : OOB;
      const uint32_t vn = m0 + ec < a.M ? (uint32_t)(er * a.ldw + ec) * 4u : OOB;
#pragma unroll
      for (int ch = 0; ch < CHUNKS; ++ch) {
#pragma unroll
        for (int q = 0; q < CP; ++q) {
          if constexpr (PH == 0) break;  // no tile before tile 0
          const int pp = ch * CP + q;
          const f32x4 v = *(const __attribute__((address_space(3))) f32x4 *)(uintptr_t)(sb[pp & 3] + pp * RPP * BM * 4);
          f32x4 nw;
#pragma unroll
          for (int e = 0; e < 4; ++e) nw[e] = fmaf(c, v[e], wold[pp][e]);
          u32x2 pk;
          pk[0] = cvt_pk_bf16(nw[0], nw[1]);
          pk[1] = cvt_pk_bf16(nw[2], nw[3]);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, nw), rp, vp + pp * wrow, 0, CPOL_MASTER_ST);
          __builtin_amdgcn_raw_buffer_store_b64(pk, rh, vh + pp * hrow, 0, CPOL_COPY_ST);
        }
        // refill the registers of chunk ch - LAG (tile it) or ch - LAG + CHUNKS (tile it-1)
#pragma unroll
        for (int q = 0; q < CP; ++q) {
          if constexpr (PH == 0) {
            const int pp = ch * CP + q;
            wold[pp] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rn, vn + pp * wrow, 0, CPOL_MASTER_LD));
          } else if (ch >= LAG) {
            const int pp = (ch - LAG) * CP + q;
            wold[pp] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rn, vn + pp * wrow, 0, CPOL_MASTER_LD));
          } else if constexpr (PH == 2) {
            const int pp = (ch - LAG + CHUNKS) * CP + q;
            wold[pp] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, vp + pp * wrow, 0, CPOL_MASTER_LD));
          }
        }
        if constexpr (STREAM) {
          // chunk ch spans slab barriers ch*TK/CHUNKS .. (ch+1)*TK/CHUNKS - 1 (TK > CHUNKS)
          if (have)
            for (int q = (ch * TK) / CHUNKS; q < ((ch + 1) * TK) / CHUNKS; ++q) lds_barrier();
        } else {
          if (have && ch < TK) lds_barrier();
        }
      }
      if (have) {
        if constexpr (!STREAM) {
          for (int ch = CHUNKS; ch < TK; ++ch) lds_barrier();
          for (int q = 0; q < 2 * reloads(it); ++q) lds_barrier();  // the MMA group's Delta_Y reloads
        }
        lds_barrier();  // staging free
        lds_barrier();  // staging full
      }
      pm0 = m0;
    };
    iteration(std::integral_constant<int, 0>{}, 0);
    if (nmy >= 1) iteration(std::integral_constant<int, 1>{}, 1);
    for (int it = 2; it <= nmy; ++it) iteration(std::integral_constant<int, 2>{}, it);
  }
}

}  // namespace

bool dw_sgd_fits(const GemmProblem &p) {
  const Epilogue &e = p.epi;
  auto al = [](const void *q, int a) { return (reinterpret_cast<uintptr_t>(q) % a) == 0; };
  return p.dtype == IMBD_BF16 && !p.a_kc && !p.b_kc && e.mode == EPI_SGD && e.out2 && !e.mask && !e.bias &&
         !e.relu && p.K > 0 && p.K <= 2048 && p.M > 0 && p.N > 0 && p.N <= 256 * 128 && p.M % 8 == 0 &&
         p.N % 8 == 0 && al(p.A, 16) && al(p.B, 16) && p.lda % 8 == 0 && p.ldb % 8 == 0 &&
         al(e.out, 16) && e.ldo % 4 == 0 && al(e.out2, 8) && e.ldo2 % 4 == 0 && e.ldo < (1 << 21) &&
         e.ldo2 < (1 << 21) && (int64_t)p.K * p.lda * 2 < ((int64_t)1 << 31) &&
         (int64_t)p.K * p.ldb * 2 < ((int64_t)1 << 31);
}

int run_dw_sgd(const GemmProblem &p, hipStream_t s, const ReduceTail *tail) {
  DwArgs d;
  const bool carry = tail && tail->kind == 1;
  d.tail = carry ? tail->sk : SkReduceArgs{};
  d.tail_items = carry ? tail->items : 0;
  d.X = reinterpret_cast<const uint16_t *>(p.A);
  d.DY = reinterpret_cast<const uint16_t *>(p.B);
  d.ldx = p.lda;
  d.lddy = p.ldb;
  d.M = p.M;
  d.N = p.N;
  d.K = p.K;
  d.w = reinterpret_cast<float *>(p.epi.out);
  d.ldw = p.epi.ldo;
  d.w16 = p.epi.out2;
  d.ldw16 = p.epi.ldo2;
  d.lr = p.epi.lr;
  d.alpha = p.epi.alpha;
  // past 256 samples the Delta_Y block is never whole in LDS: the bias gradient gets the
  // column-sum kernel instead
  const bool bias_apart = p.K > KMAX_SAMPLES && p.db_mode != 0;
  d.db_mode = bias_apart ? 0 : p.db_mode;
  d.db_out = p.db_out;
  d.bias = p.bias;
  d.db_alpha = p.db_alpha;
  d.bias_lr = p.bias_lr;
  d.tiles_m = (p.M + 127) / 128;
  d.tiles_n = (p.N + 127) / 128;
  d.spread = (p.epi.ldo * 4) % 8192 == 0;
  // past 256 samples Delta_Y streams in slabs beside X (option IMBD_OPT_DW_STREAM = 0:
  // the resident block reloaded per 256-sample chunk instead)
  const bool stream = p.K > KMAX_SAMPLES && opt(IMBD_OPT_DW_STREAM) != 0;
  // One workgroup per CU at most, and a multiple of the column-block count so that a
  // workgroup's tiles share one Delta_Y column block (kept in LDS).
  const int tiles = d.tiles_m * d.tiles_n;
  const int grid = tiles < 256 ? tiles : (256 / d.tiles_n) * d.tiles_n;
  {
    LaunchTimer t(p.kclass, p.layer, s, true);
    if (stream) hipExtLaunchKernelGGL(dw_sgd_kernel<true>, dim3(grid), dim3(512), 0, s, t.start(), t.stop(), 0, d);
    else hipExtLaunchKernelGGL(dw_sgd_kernel<false>, dim3(grid), dim3(512), 0, s, t.start(), t.stop(), 0, d);
  }
  const int rc = check_launch("dw_sgd");
  if (rc != IMBD_OK || !bias_apart) return rc;
  return run_bias_grad(IMBD_BF16, p.N, p.K, p.B, p.ldb, p.db_alpha, p.db_mode == 1 ? p.db_out : nullptr,
                       p.db_mode == 2 ? p.bias : nullptr, p.bias_lr, s, p.layer);
}

}  // namespace imbd
