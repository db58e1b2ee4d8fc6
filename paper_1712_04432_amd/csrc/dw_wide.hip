// Fused weight gradient + SGD update of a fully connected layer for batches above 256
// samples (bf16 operands, fp32 masters):
//   Delta_W[o][i] = sum_b Delta_Y[b][o] X[b][i]      (Sec. 1, K = the batch)
//   w[o][i] -= lr * alpha * Delta_W[o][i];  w16[o][i] = bf16(w[o][i])   (Eq. (1))
// (or, for the unfused and local backward passes, alpha * Delta_W stored as fp32). The
// bias gradient (column sums of Delta_Y) comes from the workgroups of the first column
// tile up to 512 samples, else from the column-sum kernel.
//
// At these batch sizes the product (2 x batch flops per weight) outweighs the update's
// 10 bytes per weight, so the kernel takes the large-tile layout of the conv tile's
// weight-gradient kernel (csrc/conv.hip), with the update done by the epilogue of each
// tile (K is never split: the update needs the whole sum). A workgroup owns 256 (or 128) output
// rows o x 128 input columns i; both operands are sample-major, so K = samples and both
// fragments come from k-row slabs through the gfx950 LDS transpose read. Slabs of 64
// samples:
//  * waves 6-7 load the Delta_Y slab (64 samples x 256 (128) columns, four (two) 64-column
//    quarters) through a 3-slot ring;
//  * waves 4-5 load the X slab (64 samples x 128 columns, two quarters) through a 4-slot
//    ring;
//  * waves 0-3 each accumulate 128 (64) rows o x 64 columns i in registers.
// Samples past the batch are past the end of the buffer descriptors and read as zero;
// columns past M or N only reach outputs that are not stored.
// Then the tile goes through LDS ([o][i], fp32) and all eight waves update it: non-
// temporal master loads, non-temporal device-scope master stores and device-scope stores
// of the bf16 copy, as in the small-batch update kernel (csrc/dw_sgd.hip), which keeps
// the masters out of the caches and the new copy in the MALL for the next forward.

#include <stdlib.h>

#include "dw_wide_body.h"
#include "lean_reduce.h"

namespace imbd {
namespace {

// the kernel: one tile per workgroup
template <bool SGD, int OH, bool DUAL>
__global__ void __launch_bounds__(512, DUAL ? 2 : 1) dw_wide_kernel(DlArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[dl_lds_bytes<OH, DUAL>()];
  dw_wide_body<SGD, OH, DUAL>(a, smem, (int)blockIdx.x, (int)gridDim.x);
  if constexpr (SGD) {
    // the reduce this launch carries (another layer's Delta_X partials into its Delta_Y):
    // eight outputs of one sample per item, a share of them per workgroup after its tile
    const int mq = a.tail.M / 8;
    for (int64_t t = (int64_t)blockIdx.x * 512 + threadIdx.x; t < a.tail_items; t += (int64_t)gridDim.x * 512) {
      const int n = (int)(t / mq);
      lean_reduce_item<true, true>(a.tail, n, (int)(t - (int64_t)n * mq) * 8);
    }
  }
}

}  // namespace

bool dw_wide_fits(const GemmProblem &p) {
  const Epilogue &e = p.epi;
  // the fused update: batches above 256 (smaller ones run on the persistent kernel with its
  // Delta_Y block resident, the faster of the two there on the AlexNet and VGG FC stacks;
  // from 257 samples this kernel, with two workgroups per CU where the tiles take more than
  // one round, beats the persistent one with Delta_Y streamed); the fp32 store: any batch
  const int min_k = e.mode == EPI_STORE ? 1 : opt(IMBD_OPT_DW_WIDE_MIN_K);
  auto al = [](const void *q, int a) { return (reinterpret_cast<uintptr_t>(q) % a) == 0; };
  const int64_t lim = (int64_t)1 << 31;  // bytes in one buffer descriptor
  if (p.dtype != IMBD_BF16 || p.a_kc || p.b_kc || e.mask || e.bias || e.relu || p.K < min_k || p.K <= 0 ||
      p.M <= 0 || p.N <= 0 || p.M % 8 || !al(p.A, 16) || p.lda % 8 ||
      (p.b_dw4 ? !al(p.B, 4) || p.ldb % 2 || p.N % 2 : !al(p.B, 16) || p.ldb % 8) ||
      p.lda < p.M || p.ldb < p.N || !al(e.out, 16) || e.ldo % 4 || e.ldo < p.M)
    return false;
  if (((int64_t)(p.K - 1) * p.lda + p.M) * 2 >= lim || ((int64_t)(p.K - 1) * p.ldb + (p.N + 7) / 8 * 8) * 2 >= lim ||
      ((int64_t)(p.N - 1) * e.ldo + p.M) * 4 >= lim)
    return false;
  if (e.mode == EPI_STORE) return e.out_dtype == IMBD_F32;  // alpha * Delta_W, fp32
  return e.mode == EPI_SGD && e.out2 && al(e.out2, 8) && e.ldo2 % 4 == 0 && e.ldo2 >= p.M &&
         ((int64_t)(p.N - 1) * e.ldo2 + p.M) * 2 < lim;
}

void dw_wide_prepare(const GemmProblem &p, int extra_blocks, DlArgs *out, int *oh_out, bool *dual_out,
                     int *grid_out) {
  DlArgs a;
  a.X = reinterpret_cast<const uint16_t *>(p.A);
  a.DY = reinterpret_cast<const uint16_t *>(p.B);
  a.ldx = p.lda;
  a.lddy = p.ldb;
  a.x_bytes = (uint32_t)(((int64_t)(p.K - 1) * p.lda + p.M) * 2);
  // the descriptor ends at the last sample's row rounded up to whole 16-byte chunks: with
  // a 16-byte aligned base and ldb a multiple of 8 that is still inside the caller's row,
  // and a chunk that crossed a tighter end would read as zero whole (columns of the last
  // sample dropped); columns past N only feed outputs that are not stored
  a.dy_bytes = (uint32_t)(((int64_t)(p.K - 1) * p.ldb + (p.N + 7) / 8 * 8) * 2);
  // rows read in 4-byte pieces: the descriptor ends at the last sample's column N (even)
  a.dy_dw4 = p.b_dw4 ? 1 : 0;
  if (p.b_dw4) a.dy_bytes = (uint32_t)(((int64_t)(p.K - 1) * p.ldb + p.N) * 2);
  a.M = p.M;
  a.N = p.N;
  a.K = p.K;
  a.w = reinterpret_cast<float *>(p.epi.out);
  a.w16 = p.epi.out2;
  a.ldw = p.epi.ldo;
  a.ldw16 = p.epi.ldo2;
  a.w_bytes = (uint32_t)(((int64_t)(p.N - 1) * p.epi.ldo + p.M) * 4);
  const bool sgd = p.epi.mode == EPI_SGD;
  a.w16_bytes = sgd ? (uint32_t)(((int64_t)(p.N - 1) * p.epi.ldo2 + p.M) * 2) : 0;
  a.lr = p.epi.lr;
  a.alpha = p.epi.alpha;
  // 128-row tiles where they finish the launch in fewer tile-heights of time: the time
  // of a launch is about its rounds of workgroups over 256 CUs times the tile height
  // (256-row tiles keep a 10% preference: fewer, larger tiles amortise each tile's start);
  // workgroups of another product in the same launch count in the rounds
  const int64_t ti = (p.M + 127) / 128;
  const int64_t t256 = (p.N + 255) / 256 * ti + extra_blocks, t128 = (p.N + 127) / 128 * ti + extra_blocks;
  // two workgroups per CU when the 128-row tiles take more than one round of the 256 CUs:
  // one workgroup's update (or store) then streams while the other computes (alone in
  // its launch only)
  const int dual_opt = opt(IMBD_OPT_DW_WIDE_DUAL);
  const bool dual = extra_blocks == 0 && (dual_opt == 1 || (dual_opt == -1 && t128 > 256));
  // (4-byte pieces: 128-row tiles, whose loads in flight fit the memory counter)
  const bool half = dual || p.b_dw4 || ((t128 + 255) / 256) * 128 * 11 < ((t256 + 255) / 256) * 256 * 10;
  const int oh = half ? 128 : 256;
  a.tiles_o = (p.N + oh - 1) / oh;
  a.tiles_i = (p.M + 127) / 128;
  // the bias gradient in the kernel up to 512 samples (a few microseconds of one column
  // tile's workgroups); past that the column-sum kernel spreads it over more workgroups
  const bool db_here = p.db_mode != 0 && p.K <= 512;
  a.db_mode = db_here ? p.db_mode : 0;
  a.db_alpha = p.db_alpha;
  a.bias_lr = p.bias_lr;
  a.db_out = p.db_out;
  a.bias = p.bias;
  a.tail = LeanReduceArgs{};
  a.tail_items = 0;
  *out = a;
  *oh_out = oh;
  *dual_out = dual;
  *grid_out = (a.tiles_o * a.tiles_i + 7) / 8 * 8;
}

int run_dw_wide(const GemmProblem &p, hipStream_t s, const ReduceTail *tail) {
  DlArgs a;
  int oh, grid;
  bool dual;
  dw_wide_prepare(p, 0, &a, &oh, &dual, &grid);
  const bool sgd = p.epi.mode == EPI_SGD, half = oh == 128;
  if (tail && tail->kind == 2 && sgd) {
    a.tail = tail->lean;
    a.tail_items = tail->items;
  } else if (tail && tail->kind != 0) {
    set_error("the large-tile update carries only a wide-batch product's reduce");
    return IMBD_EINVAL;
  }
  {
    LaunchTimer t(p.kclass, p.layer, s);
    if (dual) {
      if (sgd) hipLaunchKernelGGL((dw_wide_kernel<true, 128, true>), dim3(grid), dim3(512), 0, s, a);
      else hipLaunchKernelGGL((dw_wide_kernel<false, 128, true>), dim3(grid), dim3(512), 0, s, a);
    } else if (sgd) {
      if (half) hipLaunchKernelGGL((dw_wide_kernel<true, 128, false>), dim3(grid), dim3(512), 0, s, a);
      else hipLaunchKernelGGL((dw_wide_kernel<true, 256, false>), dim3(grid), dim3(512), 0, s, a);
    } else {
      if (half) hipLaunchKernelGGL((dw_wide_kernel<false, 128, false>), dim3(grid), dim3(512), 0, s, a);
      else hipLaunchKernelGGL((dw_wide_kernel<false, 256, false>), dim3(grid), dim3(512), 0, s, a);
    }
  }
  int rc = check_launch("dw_wide");
  if (rc != IMBD_OK || p.db_mode == 0 || a.db_mode != 0) return rc;
  return run_bias_grad(IMBD_BF16, p.N, p.K, p.B, p.ldb, p.db_alpha, p.db_mode == 1 ? p.db_out : nullptr,
                       p.db_mode == 2 ? p.bias : nullptr, p.bias_lr, s, p.layer);
}

}  // namespace imbd
