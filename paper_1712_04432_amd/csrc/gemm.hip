// MFMA products of a fully connected layer on gfx950 (Sec. 1 of the paper: training
// needs three matrix products per layer -- Y = W X, Delta_X = W^T Delta_Y and
// Delta_W = Delta_Y X^T; Appendix A for their block forms).
//
// One kernel template covers all three. A workgroup owns a BM x BN tile of the output
// D(m, n) = sum_k A(m, k) B(k, n) and walks K in tiles of 128 bytes per row (64 bf16 or
// 32 fp32 elements), double-buffered in LDS. Operands are always stored in LDS with k
// contiguous ([row][k], rows padded to 144 bytes), so every MFMA fragment is a single
// 16-byte LDS read. Operands whose k index is strided in memory (W in Delta_X, both
// operands of Delta_W) are transposed inside the tile loader: each thread reads a
// VEC x VEC block with coalesced 16-byte loads along the contiguous index and
// transposes it in registers before the LDS write, so no transposed copy is ever
// written to HBM.
//
// Matrix cores: bf16 uses v_mfma_f32_16x16x32_bf16 (8 k-values per lane), fp32 uses
// v_mfma_f32_16x16x4_f32 four times per 16-byte fragment. Since a dot product does not
// depend on the order of its k terms, the k-values a lane hands to the instruction are
// simply the 8 (or 4) contiguous ones of its 16-byte fragment.
//
// Long-K products with few output tiles split K over workgroups; every split writes
// fp32 partial sums and a second kernel adds them in split order (deterministic) and
// applies the epilogue. Workgroup ids are remapped so that the tiles of one split (which
// share that K-slice of the activation operand) run on one XCD and share its L2.

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>

#include "common.h"
#include "lean_reduce.h"

namespace imbd {

namespace {

constexpr int LDS_PITCH = 144;  // bytes per LDS row: 128 bytes of k plus 16 bytes of pad
constexpr int KT_BYTES = 128;   // bytes of k per row per K tile

template <typename T> struct Elem;
template <> struct Elem<uint16_t> { static constexpr int VEC = 8; };  // bf16 bit patterns
template <> struct Elem<float> { static constexpr int VEC = 4; };

// 16 bytes = VEC consecutive elements starting at p; elements at index >= valid read as 0.
template <typename T>
__device__ __forceinline__ u32x4 load16(const T *p, int valid, bool vec_ok) {
  constexpr int VEC = Elem<T>::VEC;
  if (valid >= VEC && vec_ok) return *reinterpret_cast<const u32x4 *>(p);
  T tmp[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) tmp[e] = (e < valid) ? p[e] : T(0);
  u32x4 r;
  __builtin_memcpy(&r, tmp, 16);
  return r;
}

// Padded-grid geometry for masked k rows (convolution weight gradient).
struct KMask {
  int wp = 1, hp = 1, w = 1, h = 1;
};

// Operand with k contiguous in memory: the tile is R rows x 128 bytes, 8 chunks per row.
template <typename T, int R, int NT>
struct KcLoader {
  static constexpr int VEC = Elem<T>::VEC;
  static constexpr int CH = R * 8;
  static constexpr int PER = (CH + NT - 1) / NT;
  u32x4 v[PER];

  // G: guarded (edge tile: masked, possibly unaligned); !G: interior tile, plain loads
  template <bool G, bool KM = false>
  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int rows, int k0,
                                       int kend, bool vec_ok, int tid, KMask = KMask{}) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (CH % NT == 0 || c < CH) {
        const int r = c >> 3, kc = c & 7;
        const int grow = row0 + r;
        const int kk = k0 + kc * VEC;
        if constexpr (G) {
          const int valid = (grow < rows) ? (kend - kk) : 0;
          v[i] = load16<T>(base + (int64_t)grow * ld + kk, valid, vec_ok);
        } else {
          // fast path: chunks are whole (kend % VEC == 0); out-of-range chunks load a
          // clamped in-range address and are zeroed, without a branch
          const bool ok = grow < rows && kk < kend;
          const T *p = base + (int64_t)min(grow, rows - 1) * ld + min(kk, kend - VEC);
          const u32x4 x = *reinterpret_cast<const u32x4 *>(p);
          v[i] = ok ? x : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (CH % NT == 0 || c < CH) {
        const int r = c >> 3, kc = c & 7;
        *reinterpret_cast<u32x4 *>(lds + r * LDS_PITCH + kc * 16) = v[i];
      }
    }
  }
};

// Operand whose rows are contiguous and k is strided: the tile is 128 bytes of k (8 blocks
// of VEC k-rows) by R contiguous elements. Thread blocks are VEC (k) x VEC (r); lanes with
// consecutive ids take consecutive k-blocks, so one wave reads 8 rows x 128 contiguous
// bytes per load and writes 8 distinct 16-byte slots of one LDS row per store.
template <typename T, int R, int NT>
struct TrLoader {
  static constexpr int VEC = Elem<T>::VEC;
  static constexpr int NB = 8 * (R / VEC);
  static constexpr int PER = (NB + NT - 1) / NT;
  u32x4 v[PER][VEC];

  // KM: k indexes positions of a zero-padded (hp x wp) image grid; rows whose position
  // falls outside the inner (h x w) image read as zero.
  template <bool G, bool KM = false>
  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int rows, int k0,
                                       int kend, bool vec_ok, int tid, KMask km = KMask{}) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int blk = tid + i * NT;
      if (NB % NT == 0 || blk < NB) {
        const int kb = blk & 7, rb = blk >> 3;
        const int col = row0 + rb * VEC;
        int wpos = 0, hpos = 0;
        if constexpr (KM) {
          const int kf = k0 + kb * VEC;
          const int q = kf / km.wp;
          wpos = kf - q * km.wp;
          hpos = q % km.hp;
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const int k = k0 + kb * VEC + j;
          bool inside = true;
          if constexpr (KM) {
            int w = wpos + j, h = hpos;
            if (w >= km.wp) {  // VEC < wp: at most one wrap into the next grid row
              w -= km.wp;
              h = (h + 1 == km.hp) ? 0 : h + 1;
            }
            inside = (w < km.w) && (h < km.h);
          }
          if constexpr (G) {
            const int valid = (k < kend && inside) ? (rows - col) : 0;
            v[i][j] = load16<T>(base + (int64_t)k * ld + col, valid, vec_ok);
          } else {
            // fast path: rows % VEC == 0, so a chunk is whole or entirely out of range;
            // out-of-range rows/columns load a clamped address and are zeroed
            const bool ok = inside && k < kend && col < rows;
            const T *p = base + (int64_t)min(k, kend - 1) * ld + min(col, rows - VEC);
            const u32x4 x = *reinterpret_cast<const u32x4 *>(p);
            v[i][j] = ok ? x : u32x4{0u, 0u, 0u, 0u};
          }
        }
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int blk = tid + i * NT;
      if (NB % NT == 0 || blk < NB) {
        const int kb = blk & 7, rb = blk >> 3;
        u32x4 o[VEC];
        if constexpr (VEC == 8) {
          // 8x8 transpose of 16-bit elements: o[r] word q = (v[2q][r], v[2q+1][r]).
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            const int w = r >> 1;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const uint32_t x = v[i][2 * q][w], y = v[i][2 * q + 1][w];
              o[r][q] = (r & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
            }
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) o[r][q] = v[i][q][r];
        }
#pragma unroll
        for (int r = 0; r < VEC; ++r)
          *reinterpret_cast<u32x4 *>(lds + (rb * VEC + r) * LDS_PITCH + kb * 16) = o[r];
      }
    }
  }
};

template <typename T, int R, int NT, bool KC>
struct LoaderSel;
template <typename T, int R, int NT>
struct LoaderSel<T, R, NT, true> { using type = KcLoader<T, R, NT>; };
template <typename T, int R, int NT>
struct LoaderSel<T, R, NT, false> { using type = TrLoader<T, R, NT>; };

template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

struct KArgs {
  const void *A;
  const void *B;
  int64_t lda, ldb;
  int M, N, K;
  int k_split, splits, tiles_m, tiles_n;
  int a_vec, b_vec, out_vec, mask_vec, bias_vec;
  Epilogue epi;
  float *partial;  // [splits][sstride] of [N][ldp] rows when splits > 1
  int64_t ldp, sstride;
  int db_mode;     // see GemmProblem
  float *db_out;
  float *bias;
  float db_alpha, bias_lr;
  int cH, cW, cCi, cCo;  // 3x3 conv tile geometry (conv launches only)
  int fast_ok;           // operand extents allow the clamped fast path (see the kernel)
};

// ------------------------------------------------------------------------- epilogue
__device__ __forceinline__ float mask_at(const Epilogue &e, int m, int n) {
  const int64_t off = (int64_t)n * e.ldmask + m;
  return (e.mask_dtype == IMBD_BF16) ? bf16_to_f32(reinterpret_cast<const uint16_t *>(e.mask)[off])
                                     : reinterpret_cast<const float *>(e.mask)[off];
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}

// Finish up to 4 consecutive outputs (m..m+3, n); v holds the accumulated sums.
__device__ __forceinline__ void epilogue4(const KArgs &g, int m, int n, const float v[4]) {
  const Epilogue &e = g.epi;
  const int cnt = (g.M - m) < 4 ? (g.M - m) : 4;
  const bool vec = cnt == 4 && g.out_vec;
  if (e.mode == EPI_SGD) {
    float *w = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    if (vec) {
      const f32x4 old = *reinterpret_cast<const f32x4 *>(w);
      f32x4 nw;
#pragma unroll
      for (int i = 0; i < 4; ++i) nw[i] = fmaf(-e.lr, e.alpha * v[i], old[i]);
      *reinterpret_cast<f32x4 *>(w) = nw;
      if (e.out2) {
        u32x2 pk;
        pk[0] = pack_bf16x2(nw[0], nw[1]);
        pk[1] = pack_bf16x2(nw[2], nw[3]);
        *reinterpret_cast<u32x2 *>(e.out2 + (int64_t)n * e.ldo2 + m) = pk;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < cnt) {
          const float nw = fmaf(-e.lr, e.alpha * v[i], w[i]);
          w[i] = nw;
          if (e.out2) e.out2[(int64_t)n * e.ldo2 + m + i] = f32_to_bf16(nw);
        }
    }
    return;
  }
  float x[4], bias[4] = {0.f, 0.f, 0.f, 0.f}, keep[4] = {1.f, 1.f, 1.f, 1.f};
  if (e.bias) {
    if (cnt == 4 && g.bias_vec) {
      const f32x4 b4 = *reinterpret_cast<const f32x4 *>(e.bias + m);
      bias[0] = b4[0]; bias[1] = b4[1]; bias[2] = b4[2]; bias[3] = b4[3];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < cnt) bias[i] = e.bias[m + i];
    }
  }
  if (e.mask) {
    if (cnt == 4 && g.mask_vec) {
      const int64_t off = (int64_t)n * e.ldmask + m;
      if (e.mask_dtype == IMBD_BF16) {
        const u32x2 mk = *reinterpret_cast<const u32x2 *>(reinterpret_cast<const uint16_t *>(e.mask) + off);
        keep[0] = bf16_to_f32((uint16_t)(mk[0] & 0xffffu)) > 0.f;
        keep[1] = bf16_to_f32((uint16_t)(mk[0] >> 16)) > 0.f;
        keep[2] = bf16_to_f32((uint16_t)(mk[1] & 0xffffu)) > 0.f;
        keep[3] = bf16_to_f32((uint16_t)(mk[1] >> 16)) > 0.f;
      } else {
        const f32x4 mk = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(e.mask) + off);
#pragma unroll
        for (int i = 0; i < 4; ++i) keep[i] = mk[i] > 0.f;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < cnt) keep[i] = mask_at(e, m + i, n) > 0.f;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = e.alpha * v[i] + bias[i];
    if (e.relu) t = t > 0.0f ? t : 0.0f;
    x[i] = keep[i] != 0.f ? t : 0.0f;
  }
  if (e.out_dtype == IMBD_BF16) {
    uint16_t *o = reinterpret_cast<uint16_t *>(e.out) + (int64_t)n * e.ldo + m;
    if (vec) {
      u32x2 pk;
      pk[0] = pack_bf16x2(x[0], x[1]);
      pk[1] = pack_bf16x2(x[2], x[3]);
      *reinterpret_cast<u32x2 *>(o) = pk;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < cnt) o[i] = f32_to_bf16(x[i]);
    }
  } else {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    if (vec) {
      *reinterpret_cast<f32x4 *>(o) = f32x4{x[0], x[1], x[2], x[3]};
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < cnt) o[i] = x[i];
    }
  }
}

// Position P of the padded grid (n, h, w) -> output pixel row (n*H + h)*W + w, or -1 when
// (h, w) lies in the padding (those positions are computed and dropped).
__device__ __forceinline__ int conv_out_row(const KArgs &g, int P) {
  const int Wp = g.cW + 2, Hp = g.cH + 2;
  const int n = P / (Hp * Wp);
  const int rem = P - n * Hp * Wp;
  const int h = rem / Wp;
  const int w = rem - h * Wp;
  if (h >= g.cH || w >= g.cW) return -1;
  return (n * g.cH + h) * g.cW + w;
}

// --------------------------------------------------------------------------- kernel
// CONV selects how operands are addressed: 0 plain matrices; 1/2/3 the forward, input-
// gradient and weight-gradient passes of a 3x3 conv tile, computed on the positions of
// the zero-padded (H+2) x (W+2) grid so that every tap is a row shift of a dense matrix.
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, bool A_KC, bool B_KC, int CONV = 0>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N, 2)
    gemm_kernel(KArgs g) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int VEC = Elem<T>::VEC;
  constexpr int BK = KT_BYTES / (int)sizeof(T);
  constexpr int STAGE_A = BM * LDS_PITCH, STAGE = (BM + BN) * LDS_PITCH;
  // Transposed loaders use a fraction of the threads; when both fit in half the block,
  // the B loader runs on the other half.
  constexpr int NB_A = A_KC ? BM * 8 : 8 * (BM / VEC);
  constexpr int NB_B = B_KC ? BN * 8 : 8 * (BN / VEC);
  constexpr int XOR_B = (NB_A <= NT / 2 && NB_B <= NT / 2) ? NT / 2 : 0;
  // The weight-gradient product (both operands strided) is the one that carries the
  // fused update; its old master tile is fetched before the K loop so the read half of
  // the read-modify-write overlaps the products.
  constexpr bool PREFETCH_W = !A_KC && !B_KC && CONV == 0;
  // Row sums of the B tile (the bias gradient), NT/BN threads per row.
  constexpr int TPR = NT / BN;
  constexpr int CPT = 8 / TPR;  // 16-byte chunks per thread per K tile
  static_assert(WM % 16 == 0 && WN % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(NT % BN == 0 && (TPR == 1 || TPR == 2 || TPR == 4 || TPR == 8), "row-sum split");
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const int tid = threadIdx.x;
  const int tid_b = tid ^ XOR_B;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave % WAVES_M) * WM, wn0 = (wave / WAVES_M) * WN;

  // Consecutive workgroup ids are dealt round-robin to the 8 XCDs; give each XCD a
  // contiguous range of logical tiles (which share a K-slice of the B operand).
  int bid = blockIdx.x;
  const int G = gridDim.x;
  if ((G & 7) == 0) bid = (bid & 7) * (G >> 3) + (bid >> 3);
  const int per_split = g.tiles_m * g.tiles_n;
  const int s = bid / per_split;
  const int rem = bid - s * per_split;
  // n fastest: the tiles that share an A tile (a W row block, or an X column block in
  // the weight gradient) run back to back on one XCD and share its L2
  const int tm = rem / g.tiles_n;
  const int tn = rem - tm * g.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = s * g.k_split;
  const int kend = min(g.K, kbeg + g.k_split);
  const int nk = (kend > kbeg) ? (kend - kbeg + BK - 1) / BK : 0;
  const int fr = lane & 15, fg = lane >> 4;

  // Full tiles finish through LDS (see the end of the kernel): 32 threads cover one row of
  // BM outputs, so every store instruction writes whole contiguous rows.
  constexpr int TPRW = BM / 4;            // threads per output row (4 outputs each)
  constexpr int RPP = NT / TPRW;          // rows per pass
  constexpr int PASSES = BN / RPP;
  static_assert(NT % TPRW == 0 && BN % RPP == 0, "staged epilogue shape");
  const int er = tid / TPRW, ec = (tid % TPRW) * 4;
  // Staged when the outputs allow 16-byte stores; ragged tiles guard each row and each
  // group of 4 columns.
  const bool staged = g.out_vec;
  const bool sgd_fast = PREFETCH_W && staged && g.splits == 1 && g.epi.mode == EPI_SGD;
  f32x4 wold[PREFETCH_W ? PASSES : 1];
  if constexpr (PREFETCH_W) {
    if (sgd_fast) {
      const float *w = reinterpret_cast<const float *>(g.epi.out);
#pragma unroll
      for (int p = 0; p < PASSES; ++p) {
        const int n = n0 + p * RPP + er;
        const int m = m0 + ec;
        wold[p] = (n < g.N && m + 4 <= g.M)
                      ? *reinterpret_cast<const f32x4 *>(w + (int64_t)n * g.epi.ldo + m)
                      : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  const bool do_db = g.db_mode != 0 && tm == 0 && g.splits == 1;
  float dbsum = 0.f;

  const T *A = reinterpret_cast<const T *>(g.A);
  const T *Bp = reinterpret_cast<const T *>(g.B);
  // Two register stages: while tile kt is multiplied out of LDS, the global loads of
  // tiles kt+1 and kt+2 are both in flight. The weight-gradient product (short K, its
  // registers taken by the prefetched master tile) keeps one stage.
  constexpr int NSTAGE = PREFETCH_W ? 1 : 2;
  typename LoaderSel<T, BM, NT, A_KC>::type la[NSTAGE];
  typename LoaderSel<T, BN, NT, B_KC>::type lb[NSTAGE];

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Interior tiles (every row, column and K tile in range, 16-byte aligned operands) run
  // the main loop with plain vector loads and no branches around them, so the compiler's
  // wait counts cover exactly the tile being stored (the last iterations re-load the last
  // tile instead of skipping the load). Edge tiles run it with masked, conditional loads.
  // Fast path: aligned operands, whole 16-byte chunks (K ends and transposed-operand
  // widths are multiples of VEC); ragged M/N/K edges are handled by clamped, zeroed loads
  // and an odd tile count is padded with one all-zero tile.
  const bool interior = g.a_vec && g.b_vec && nk > 0 && (kend % VEC == 0) &&
                        (A_KC || g.M % VEC == 0) && (B_KC || g.N % VEC == 0) && g.fast_ok;
  const int nk_fast = (nk + NSTAGE - 1) / NSTAGE * NSTAGE;

  auto compute = [&](int kt) {
    const char *sa = smem + (kt & 1) * STAGE;
    const char *sb = sa + STAGE_A;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      u32x4 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *reinterpret_cast<const u32x4 *>(sa + (wm0 + i * 16 + fr) * LDS_PITCH + kk * 64 + fg * 16);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *reinterpret_cast<const u32x4 *>(sb + (wn0 + j * 16 + fr) * LDS_PITCH + kk * 64 + fg * 16);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (sizeof(T) == 2) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, fa[i]), __builtin_bit_cast(bf16x8, fb[j]), acc[i][j], 0, 0, 0);
          } else {
            // the whole 16-byte fragment is reinterpreted once; element-wise casts of a
            // vector lane were lowered to a single repeated lane
            const f32x4 af = __builtin_bit_cast(f32x4, fa[i]);
            const f32x4 bf = __builtin_bit_cast(f32x4, fb[j]);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af.x, bf.x, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af.y, bf.y, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af.z, bf.z, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af.w, bf.w, acc[i][j], 0, 0, 0);
          }
        }
    }
    if (do_db) {
      // this thread's share of row tid/TPR of the B tile, in k order
      const char *row = sb + (tid / TPR) * LDS_PITCH + (tid % TPR) * CPT * 16;
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const u32x4 q = *reinterpret_cast<const u32x4 *>(row + c * 16);
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            dbsum += bf16_to_f32((uint16_t)(q[w] & 0xffffu));
            dbsum += bf16_to_f32((uint16_t)(q[w] >> 16));
          }
        } else {
          const f32x4 qf = __builtin_bit_cast(f32x4, q);  // whole-vector cast (see above)
          dbsum += qf.x;
          dbsum += qf.y;
          dbsum += qf.z;
          dbsum += qf.w;
        }
      }
    }
  };
  auto buf = [&](int kt) { return smem + (kt & 1) * STAGE; };

  // Operand sources of K tile kt of this split.
  const int Wp = g.cW + 2;
  const T *A_rs = A;
  if constexpr (CONV == 3) {
    // rows of A are m = tap*C_in + c; a tile lies within one tap (C_in % BM == 0)
    const int rs = m0 / g.cCi, r = rs / 3, sx = rs - 3 * r;
    A_rs = A + (int64_t)(r * Wp + sx - rs) * g.cCi;
  }
  KMask km;
  if constexpr (CONV == 3) {
    km.wp = Wp;
    km.hp = g.cH + 2;
    km.w = g.cW;
    km.h = g.cH;
  }
  auto issueA = [&](auto &L, int kt, auto gtag) {
    constexpr bool G = decltype(gtag)::value;
    const int kg = kbeg + kt * BK;
    if constexpr (CONV == 2) {
      // W[o][tap][c] read as A(c, o) for one tap; a tile past the K range reads nothing
      const bool live = kg < kend;
      const int rs = live ? kg / g.cCo : 0, o0 = live ? kg - rs * g.cCo : g.cCo;
      L.template load<G>(A + (int64_t)rs * g.cCi, g.lda, m0, g.M, o0, g.cCo, g.a_vec, tid);
    } else {
      L.template load<G>(A_rs, g.lda, m0, g.M, kg, kend, g.a_vec, tid);
    }
  };
  auto issueB = [&](auto &L, int kt, auto gtag) {
    constexpr bool G = decltype(gtag)::value;
    const int kg = kbeg + kt * BK;
    if constexpr (CONV == 1) {
      // x_pad shifted by tap (r, s): B(c, P) = x_pad_flat[P + r*Wp + s][c]
      const bool live = kg < kend;
      const int rs = live ? kg / g.cCi : 0, c0 = live ? kg - rs * g.cCi : g.cCi, r = rs / 3, sx = rs - 3 * r;
      L.template load<G>(Bp + (int64_t)(r * Wp + sx) * g.cCi, g.ldb, n0, g.N, c0, g.cCi, g.b_vec, tid_b);
    } else if constexpr (CONV == 2) {
      // dy_pad shifted by (2-r, 2-s): B(o, P) = dy_pad_flat[P + (2-r)*Wp + 2-s][o]
      const bool live = kg < kend;
      const int rs = live ? kg / g.cCo : 0, o0 = live ? kg - rs * g.cCo : g.cCo, r = rs / 3, sx = rs - 3 * r;
      L.template load<G>(Bp + (int64_t)((2 - r) * Wp + 2 - sx) * g.cCo, g.ldb, n0, g.N, o0, g.cCo, g.b_vec,
                         tid_b);
    } else if constexpr (CONV == 3) {
      // interior of dy_pad, rows outside the inner image masked to zero
      L.template load<G, true>(Bp, g.ldb, n0, g.N, kg, kend, g.b_vec, tid_b, km);
    } else {
      L.template load<G>(Bp, g.ldb, n0, g.N, kg, kend, g.b_vec, tid_b);
    }
  };
  const BoolTag<false> plain{};
  const BoolTag<true> guarded{};

  if (interior) {
    auto kc = [&](int kt) { return kt; };
    issueA(la[0], 0, plain);
    issueB(lb[0], 0, plain);
    la[0].store(buf(0), tid);
    lb[0].store(buf(0) + STAGE_A, tid_b);
    if constexpr (NSTAGE == 2) {
      issueA(la[NSTAGE - 1], kc(1), plain);
      issueB(lb[NSTAGE - 1], kc(1), plain);
    }
    __syncthreads();
    for (int kt = 0; kt < nk_fast; kt += NSTAGE) {
      if constexpr (NSTAGE == 2) {
        // step kt: set 1 holds tile kt+1; set 0 receives tile kt+2
        issueA(la[0], kc(kt + 2), plain);
        issueB(lb[0], kc(kt + 2), plain);
        compute(kt);
        la[NSTAGE - 1].store(buf(kt + 1), tid);
        lb[NSTAGE - 1].store(buf(kt + 1) + STAGE_A, tid_b);
        __syncthreads();
        // step kt+1: set 0 holds tile kt+2; set 1 receives tile kt+3
        issueA(la[NSTAGE - 1], kc(kt + 3), plain);
        issueB(lb[NSTAGE - 1], kc(kt + 3), plain);
        compute(kt + 1);
        la[0].store(buf(kt + 2), tid);
        lb[0].store(buf(kt + 2) + STAGE_A, tid_b);
        __syncthreads();
      } else {
        issueA(la[0], kc(kt + 1), plain);
        issueB(lb[0], kc(kt + 1), plain);
        compute(kt);
        la[0].store(buf(kt + 1), tid);
        lb[0].store(buf(kt + 1) + STAGE_A, tid_b);
        __syncthreads();
      }
    }
  } else {
    // edge tiles: masked loads, one register stage
    if (nk > 0) {
      issueA(la[0], 0, guarded);
      issueB(lb[0], 0, guarded);
      la[0].store(buf(0), tid);
      lb[0].store(buf(0) + STAGE_A, tid_b);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const bool more = kt + 1 < nk;
      if (more) {
        issueA(la[0], kt + 1, guarded);
        issueB(lb[0], kt + 1, guarded);
      }
      compute(kt);
      if (more) {
        la[0].store(buf(kt + 1), tid);
        lb[0].store(buf(kt + 1) + STAGE_A, tid_b);
      }
      __syncthreads();
    }
  }

  if (do_db) {
    // combine the TPR consecutive threads of a row (commutative pairwise adds: every
    // lane of the group gets the same bits)
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) dbsum += __shfl_xor(dbsum, o, 64);
    const int n = n0 + tid / TPR;
    if (tid % TPR == 0 && n < g.N) {
      const float gb = g.db_alpha * dbsum;
      if (g.db_mode == 1) g.db_out[n] = gb;
      else g.bias[n] = fmaf(-g.bias_lr, gb, g.bias[n]);
    }
  }

  if (staged) {
    // Stage the accumulator tile in LDS as [n][m] (pitch BM+4 floats), then let each group
    // of TPRW threads finish one whole row per pass.
    constexpr int PT = BM + 4;
    static_assert(BN * PT * 4 <= 2 * STAGE, "staged tile must fit the operand buffers");
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        *reinterpret_cast<f32x4 *>(stg + (wn0 + j * 16 + fr) * PT + wm0 + i * 16 + fg * 4) = acc[i][j];
    __syncthreads();
    const int m = m0 + ec;
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int nl = p * RPP + er;
      int n = n0 + nl;
      if (n >= g.N || m >= g.M) continue;
      const f32x4 a = *reinterpret_cast<const f32x4 *>(stg + nl * PT + ec);
      if constexpr (CONV == 1 || CONV == 2) {
        n = conv_out_row(g, n);
        if (n < 0) continue;
      }
      if (g.splits > 1) {
        *reinterpret_cast<f32x4 *>(g.partial + (int64_t)s * g.sstride + (int64_t)n * g.ldp + m) = a;
        continue;
      }
      if constexpr (PREFETCH_W) {
        if (sgd_fast && m + 4 <= g.M) {
          const Epilogue &e = g.epi;
          f32x4 nw;
#pragma unroll
          for (int q = 0; q < 4; ++q) nw[q] = fmaf(-e.lr, e.alpha * a[q], wold[p][q]);
          *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m) = nw;
          if (e.out2) {
            u32x2 pk;
            pk[0] = pack_bf16x2(nw[0], nw[1]);
            pk[1] = pack_bf16x2(nw[2], nw[3]);
            *reinterpret_cast<u32x2 *>(e.out2 + (int64_t)n * e.ldo2 + m) = pk;
          }
          continue;
        }
      }
      const float v[4] = {a[0], a[1], a[2], a[3]};
      epilogue4(g, m, n, v);
    }
    return;
  }

  // Accumulator layout of a 16x16 block: lane holds rows 4*(lane/16)..+3 of column lane%16.
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int m = m0 + wm0 + i * 16 + fg * 4;
      const int n = n0 + wn0 + j * 16 + fr;
      if (m >= g.M || n >= g.N) continue;
      const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if (g.splits == 1) {
        int on = n;
        if constexpr (CONV == 1 || CONV == 2) {
          on = conv_out_row(g, n);
          if (on < 0) continue;
        }
        epilogue4(g, m, on, v);
      } else {
        float *p = g.partial + (int64_t)s * g.sstride + (int64_t)n * g.ldp + m;
        *reinterpret_cast<f32x4 *>(p) = f32x4{v[0], v[1], v[2], v[3]};
      }
    }
}

// Sum the split partials in split order, then apply the epilogue.
__global__ void __launch_bounds__(256) splitk_reduce_kernel(KArgs g) {
  const int m4 = (g.M + 3) >> 2;
  const int64_t total = (int64_t)g.N * m4;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int n = (int)(t / m4);
    const int m = (int)(t - (int64_t)n * m4) * 4;
    // loads of up to 8 splits are issued together; the adds keep split order
    const float *p0 = g.partial + (int64_t)n * g.ldp + m;
    const int64_t sstride = g.sstride;
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < g.splits; s0 += 8) {
      f32x4 q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < g.splits) q[u] = *reinterpret_cast<const f32x4 *>(p0 + (s0 + u) * sstride);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < g.splits) a = (s0 + u == 0) ? q[u] : a + q[u];
    }
    const float v[4] = {a[0], a[1], a[2], a[3]};
    epilogue4(g, m, n, v);
  }
}

// Lean split-K reduction for the epilogues the layer products use (store with optional
// bias/ReLU, or store with the ReLU mask), 8 outputs per thread on a 2-D grid
// (blockIdx.y = n). Splits are added in split order, as in the generic kernel.
template <bool OUT_BF16, bool MASK>
__global__ void __launch_bounds__(256) splitk_reduce_fast(KArgs g) {
  const int n = blockIdx.y;
  const int m = (blockIdx.x * 256 + threadIdx.x) * 8;
  if (m >= g.M) return;
  lean_reduce_item<OUT_BF16, MASK>(LeanReduceArgs{g.partial, g.ldp, g.sstride, g.M, g.N, g.splits, g.epi}, n, m);
}

// ------------------------------------------------------------- configurations
typedef void (*KernelFn)(KArgs);

struct TileCfg {
  int bm, bn, nt;
  KernelFn fn[2][2][2];  // [bf16?][a_kc][b_kc]
};

template <int BM, int BN, int WMW, int WNW>
constexpr TileCfg make_cfg() {
  return TileCfg{BM, BN, 64 * WMW * WNW,
                 {{{gemm_kernel<float, BM, BN, WMW, WNW, false, false>,
                    gemm_kernel<float, BM, BN, WMW, WNW, false, true>},
                   {gemm_kernel<float, BM, BN, WMW, WNW, true, false>,
                    gemm_kernel<float, BM, BN, WMW, WNW, true, true>}},
                  {{gemm_kernel<uint16_t, BM, BN, WMW, WNW, false, false>,
                    gemm_kernel<uint16_t, BM, BN, WMW, WNW, false, true>},
                   {gemm_kernel<uint16_t, BM, BN, WMW, WNW, true, false>,
                    gemm_kernel<uint16_t, BM, BN, WMW, WNW, true, true>}}}};
}

const TileCfg kCfgs[] = {
    make_cfg<64, 64, 2, 2>(),    // 0: small products and ragged edges
    make_cfg<128, 128, 2, 2>(),  // 1: large products
    make_cfg<128, 64, 2, 2>(),   // 2: tall
    make_cfg<64, 128, 2, 2>(),   // 3: wide
};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

// Conv launches (bf16): [cfg 0 = 64x64, cfg 1 = 128x128][pass 1..3]
const KernelFn kConvFns[2][3] = {
    {gemm_kernel<uint16_t, 64, 64, 2, 2, true, true, 1>, gemm_kernel<uint16_t, 64, 64, 2, 2, false, true, 2>,
     gemm_kernel<uint16_t, 64, 64, 2, 2, false, false, 3>},
    {gemm_kernel<uint16_t, 128, 128, 2, 2, true, true, 1>, gemm_kernel<uint16_t, 128, 128, 2, 2, false, true, 2>,
     gemm_kernel<uint16_t, 128, 128, 2, 2, false, false, 3>}};


inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Split-K partial sums: [split][n][ldp] fp32. Row pitch and split pitch are kept off powers
// of two (+256 B and +4.25 KiB) so the splits of one output do not all map to the same
// DRAM bank.

}  // namespace

// The tiled template's plan.
static GemmPlan tiled_plan(const GemmProblem &p) {
  GemmPlan pl{};
  const int esz = p.dtype == IMBD_BF16 ? 2 : 4;
  const int BK = KT_BYTES / esz;
  // Tile: the largest configuration that still gives a reasonable number of tiles.
  int cfg = 0;
  if (p.M >= 128 && p.N >= 128) cfg = 1;
  else if (p.M >= 128) cfg = 2;
  else if (p.N >= 128) cfg = 3;
  const int ktiles = cdiv(p.K, BK);
  // A short product whose large tiles cannot fill 256 CUs takes 64 x 64 tiles instead
  // (splitting its few K tiles could not fill them either).
  if (cfg != 0 && ktiles < 16 && cdiv(p.M, kCfgs[cfg].bm) * cdiv(p.N, kCfgs[cfg].bn) < 256) cfg = 0;
  const int forced = opt(IMBD_OPT_GEMM_CFG);
  if (forced >= 0 && forced < kNumCfgs) cfg = forced;
  pl.cfg = cfg;
  pl.bm = kCfgs[cfg].bm;
  pl.bn = kCfgs[cfg].bn;
  const int tiles = cdiv(p.M, pl.bm) * cdiv(p.N, pl.bn);
  // Split K while there are too few tiles to fill 256 CUs twice, keeping >= 4 K tiles
  // per split (>= 2 for products of 4..15 K tiles); a product of fewer K tiles is left
  // whole (a second launch would cost more).
  int splits = 1;
  if (tiles < 512 && ktiles >= 4) {
    splits = cdiv(512, tiles);
    const int max_s = ktiles >= 16 ? ktiles / 4 : ktiles / 2;
    if (splits > max_s) splits = max_s;
    if (splits < 1) splits = 1;
  }
  const int forced_s = opt(IMBD_OPT_GEMM_SPLITS);
  if (forced_s >= 1) splits = forced_s < ktiles ? forced_s : (ktiles > 0 ? ktiles : 1);
  int k_split = cdiv(cdiv(p.K > 0 ? p.K : 1, splits), BK) * BK;
  splits = p.K > 0 ? cdiv(p.K, k_split) : 1;
  pl.splits = splits;
  pl.k_split = k_split;
  pl.ws_bytes = splits > 1 ? (size_t)splits * (size_t)partial_split_stride(p.M, p.N) * sizeof(float) : 0;
  return pl;
}

GemmPlan gemm_plan(const GemmProblem &p) {
  // Workspace sizes are computed from the dimensions alone, while the skinny and wide
  // kernels also check leading dimensions and alignment when they run; a run that fails
  // those checks falls back to the tiled template. So a plan whose dimensions admit a
  // special kernel asks for the larger of that kernel's partials and the template's, and
  // any run fits the workspace that the same dimensions were given.
  const GemmPlan tp = tiled_plan(p);
  GemmPlan pl{};
  if (skinny_dims_fit(p) && opt(IMBD_OPT_SKINNY_OFF) == 0) {
    if (skinny_fits(p)) {
      // the skinny-batch product always goes through fp32 partials (one per K split)
      skinny_plan(p, &pl.splits, &pl.k_split);
      pl.cfg = PLAN_SKINNY;
      pl.bm = 64;
      pl.bn = 256;
    } else {
      pl = tp;
    }
    pl.ws_bytes = std::max(skinny_ws_bytes(p), tp.ws_bytes);
    return pl;
  }
  if (wide_dims_fit(p)) {
    int splits, kps;
    wide_plan(p, &splits, &kps);
    const size_t wws = splits > 1 ? (size_t)splits * (size_t)partial_split_stride(p.M, p.N) * sizeof(float) : 0;
    if (wide_fits(p)) {
      pl.cfg = PLAN_WIDE;
      pl.bm = 256;
      pl.bn = 128;
      pl.splits = splits;
      pl.k_split = 64 * kps;
    } else {
      pl = tp;
    }
    pl.ws_bytes = std::max(wws, tp.ws_bytes);
    return pl;
  }
  return tp;
}

// Adds the split partials in split order and applies the epilogue.
// the lean reduce needs 8-aligned rows (M, ld and pointers) and a store epilogue
static bool lean_ok(const GemmProblem &p, int64_t ldp, int64_t sstride) {
  const Epilogue &e = p.epi;
  const int oes = e.out_dtype == IMBD_BF16 ? 2 : 4;
  return e.mode == EPI_STORE && p.M % 8 == 0 && e.ldo % 8 == 0 && (uintptr_t)e.out % (8 * oes) == 0 &&
         (!e.bias || (uintptr_t)e.bias % 32 == 0) &&
         (!e.mask || (e.ldmask % 8 == 0 && (uintptr_t)e.mask % (e.mask_dtype == IMBD_BF16 ? 16 : 32) == 0)) &&
         ldp % 8 == 0 && sstride % 8 == 0 && p.N <= 65535;
}

static int launch_reduce(const GemmProblem &p, const KArgs &g, hipStream_t s) {
  const Epilogue &e = p.epi;
  const bool lean = lean_ok(p, g.ldp, g.sstride);
  LaunchTimer t(IMBD_K_SPLITK, p.layer, s);
  if (lean) {
    const dim3 grid((unsigned)((p.M / 8 + 255) / 256), (unsigned)p.N);
    const bool bf = e.out_dtype == IMBD_BF16;
    if (e.mask) {
      if (bf) hipLaunchKernelGGL((splitk_reduce_fast<true, true>), grid, dim3(256), 0, s, g);
      else hipLaunchKernelGGL((splitk_reduce_fast<false, true>), grid, dim3(256), 0, s, g);
    } else {
      if (bf) hipLaunchKernelGGL((splitk_reduce_fast<true, false>), grid, dim3(256), 0, s, g);
      else hipLaunchKernelGGL((splitk_reduce_fast<false, false>), grid, dim3(256), 0, s, g);
    }
  } else {
    const int64_t total = (int64_t)p.N * ((p.M + 3) / 4);
    int blocks = (int)((total + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, g);
  }
  return check_launch("splitk_reduce");
}

bool wide_softmax_fits(const GemmProblem &p) {
  const GemmPlan pl = gemm_plan(p);
  return pl.cfg == PLAN_WIDE && pl.splits > 1 && p.a_kc && p.M <= 1024 && p.epi.mode == EPI_STORE &&
         p.epi.relu == 0 && p.epi.mask == nullptr && p.epi.out_dtype == IMBD_F32 && p.aux_loss == nullptr &&
         opt(IMBD_OPT_TOP_UNFUSED) == 0;
}

// The wide-batch product's split partials, then one pass per sample that adds them in split
// order with the bias (the split reduce's arithmetic), stores the logits and takes the
// softmax cross-entropy: the reduce launch and the softmax launch in one.
int run_wide_softmax(const GemmProblem &p, void *ws, size_t ws_bytes, const int32_t *labels, float inv_batch,
                     float *row_loss, void *dz, int64_t lddz, int dz_dtype, hipStream_t s) {
  const GemmPlan pl = gemm_plan(p);
  if (ws == nullptr || ws_bytes < pl.ws_bytes || (uintptr_t)ws % 16 != 0) {
    set_error("top-layer product %dx%dx%d needs %zu bytes of 16-byte aligned workspace, got %zu", p.M, p.N, p.K,
              pl.ws_bytes, ws_bytes);
    return IMBD_EWORKSPACE;
  }
  float *partial = reinterpret_cast<float *>(ws);
  const int64_t ldp = partial_ld(p.M), sstride = partial_split_stride(p.M, p.N);
  const int rc = run_wide(p, partial, ldp, sstride, s);
  if (rc != IMBD_OK) return rc;
  return run_softmax_rows_from_partials(p, partial, ldp, sstride, pl.splits, labels, inv_batch, row_loss, dz, lddz,
                                        dz_dtype, s);
}

// A fused-SGD weight-gradient problem that gemm_run sends to the persistent update kernel.
bool dw_sgd_route(const GemmProblem &p) {
  if (p.M <= 0 || p.N <= 0 || p.aux_loss || (p.db_mode != 0 && p.b_kc)) return false;
  const GemmPlan pl = gemm_plan(p);
  if (pl.cfg == PLAN_SKINNY || pl.cfg == PLAN_WIDE) return false;
  return !dw_wide_fits(p) && dw_sgd_fits(p) && opt(IMBD_OPT_DW_GENERIC) == 0;
}

bool dw_wide_route(const GemmProblem &p) {
  if (p.M <= 0 || p.N <= 0 || p.aux_loss || (p.db_mode != 0 && p.b_kc) || p.epi.mode != EPI_SGD) return false;
  const GemmPlan pl = gemm_plan(p);
  if (pl.cfg == PLAN_SKINNY || pl.cfg == PLAN_WIDE) return false;
  return dw_wide_fits(p);
}

static int check_plan_ws(const GemmPlan &pl, const GemmProblem &p, const void *ws, size_t ws_bytes) {
  if (pl.ws_bytes > 0 && (ws == nullptr || ws_bytes < pl.ws_bytes)) {
    set_error("product %dx%dx%d needs %zu bytes of workspace for split-K partials, got %zu",
              p.M, p.N, p.K, pl.ws_bytes, ws_bytes);
    return IMBD_EWORKSPACE;
  }
  if (pl.ws_bytes > 0 && (uintptr_t)ws % 16 != 0) {
    set_error("workspace must be 16-byte aligned");
    return IMBD_EINVAL;
  }
  return IMBD_OK;
}

int gemm_run_defer(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s, bool *deferred,
                   ReduceTail *tail) {
  *deferred = false;
  // (a loss-mean side job stays where gemm_run puts it: in the wide-batch product launch,
  // or in the skinny reduce, which is then not deferred)
  if (opt(IMBD_OPT_REDUCE_TAIL) != 0 && p.M > 0 && p.N > 0 && !(p.db_mode != 0 && p.b_kc)) {
    const GemmPlan pl = gemm_plan(p);
    if (pl.cfg == PLAN_SKINNY) {
      const int rc = check_plan_ws(pl, p, ws, ws_bytes);
      if (rc != IMBD_OK) return rc;
      return run_skinny_split(p, ws, s, deferred, tail);
    }
    const Epilogue &e = p.epi;
    if (pl.cfg == PLAN_WIDE && pl.splits > 1 && e.mask && e.mask_dtype == IMBD_BF16 && e.out_dtype == IMBD_BF16) {
      int rc = check_plan_ws(pl, p, ws, ws_bytes);
      if (rc != IMBD_OK) return rc;
      LeanReduceArgs r{reinterpret_cast<float *>(ws), partial_ld(p.M), partial_split_stride(p.M, p.N), p.M, p.N,
                       pl.splits, e};
      if (lean_ok(p, r.ldp, r.sstride)) {
        rc = run_wide(p, reinterpret_cast<float *>(ws), r.ldp, r.sstride, s);
        if (rc != IMBD_OK) return rc;
        tail->kind = 2;
        tail->lean = r;
        tail->items = (int64_t)p.N * (p.M / 8);
        *deferred = true;
        return IMBD_OK;
      }
    }
  }
  return gemm_run(p, ws, ws_bytes, s);
}

int run_reduce_tail(const ReduceTail &tail, int layer, hipStream_t s) {
  if (tail.kind == 1) return run_skinny_reduce_tail(tail, layer, s);
  if (tail.kind != 2) return IMBD_OK;
  KArgs g{};
  g.M = tail.lean.M;
  g.N = tail.lean.N;
  g.splits = tail.lean.splits;
  g.epi = tail.lean.epi;
  g.partial = const_cast<float *>(tail.lean.partial);
  g.ldp = tail.lean.ldp;
  g.sstride = tail.lean.sstride;
  LaunchTimer t(IMBD_K_SPLITK, layer, s);
  const dim3 grid((unsigned)((g.M / 8 + 255) / 256), (unsigned)g.N);
  hipLaunchKernelGGL((splitk_reduce_fast<true, true>), grid, dim3(256), 0, s, g);
  return check_launch("splitk_reduce");
}

int gemm_run_dw_tail(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s, const ReduceTail &tail) {
  if (tail.kind == 1 && dw_sgd_route(p)) return run_dw_sgd(p, s, &tail);
  if (tail.kind == 2 && dw_wide_route(p)) return run_dw_wide(p, s, &tail);
  // another route may use ws, where the partials are: the reduce goes first
  const int rc = run_reduce_tail(tail, p.layer, s);
  if (rc != IMBD_OK) return rc;
  return gemm_run(p, ws, ws_bytes, s);
}

int gemm_run(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s) {
  if (p.db_mode != 0 && p.b_kc) {
    set_error("bias sums need the B operand stored [k][n]");
    return IMBD_EINVAL;
  }
  const GemmPlan pl = gemm_plan(p);
  if (p.aux_loss && ((pl.cfg != PLAN_SKINNY && pl.cfg != PLAN_WIDE) || p.M <= 0 || p.N <= 0)) {
    // the skinny-batch launches and the wide-batch product carry the side job; elsewhere
    // it gets its own launch
    GemmProblem q = p;
    q.aux_loss = nullptr;
    const int rc = gemm_run(q, ws, ws_bytes, s);
    if (rc != IMBD_OK) return rc;
    return run_loss_mean(p.aux_n, p.aux_rows, p.aux_scale, p.aux_loss, s);
  }
  if (p.M <= 0 || p.N <= 0) return IMBD_OK;
  {
    const int rc = check_plan_ws(pl, p, ws, ws_bytes);
    if (rc != IMBD_OK) return rc;
  }
  if (pl.cfg == PLAN_SKINNY) return run_skinny(p, ws, s);
  const int esz = p.dtype == IMBD_BF16 ? 2 : 4;
  KArgs g;
  g.A = p.A;
  g.B = p.B;
  g.lda = p.lda;
  g.ldb = p.ldb;
  g.M = p.M;
  g.N = p.N;
  g.K = p.K;
  g.k_split = pl.k_split;
  g.splits = pl.splits;
  g.tiles_m = cdiv(p.M, pl.bm);
  g.tiles_n = cdiv(p.N, pl.bn);
  const int vec_elems = 16 / esz;
  g.a_vec = ((uintptr_t)p.A % 16 == 0) && (p.lda % vec_elems == 0);
  g.b_vec = ((uintptr_t)p.B % 16 == 0) && (p.ldb % vec_elems == 0);
  {
    const Epilogue &e = p.epi;
    const int oes = (e.mode == EPI_SGD || e.out_dtype == IMBD_F32) ? 4 : 2;
    bool ok = ((uintptr_t)e.out % (4 * oes) == 0) && (e.ldo % 4 == 0);
    if (e.mode == EPI_SGD && e.out2) ok = ok && ((uintptr_t)e.out2 % 8 == 0) && (e.ldo2 % 4 == 0);
    g.out_vec = ok;
  }
  {
    const Epilogue &e = p.epi;
    const int mes = e.mask_dtype == IMBD_BF16 ? 2 : 4;
    g.mask_vec = e.mask && ((uintptr_t)e.mask % (4 * mes) == 0) && (e.ldmask % 4 == 0);
    g.bias_vec = e.bias && ((uintptr_t)e.bias % 16 == 0);
  }
  g.fast_ok = 1;
  g.epi = p.epi;
  g.db_mode = p.db_mode;
  g.db_out = p.db_out;
  g.bias = p.bias;
  g.db_alpha = p.db_alpha;
  g.bias_lr = p.bias_lr;
  g.partial = reinterpret_cast<float *>(ws);
  g.ldp = partial_ld(p.M);
  g.sstride = partial_split_stride(p.M, p.N);

  if (pl.cfg == PLAN_WIDE) {
    int rc = run_wide(p, g.partial, g.ldp, g.sstride, s);
    if (rc == IMBD_OK && pl.splits > 1) rc = launch_reduce(p, g, s);
    return rc;
  }
  // A bf16 weight gradient runs on the large-tile kernel when stored as fp32 (any batch) or
  // fused with the update past 256 samples; the fused update of a smaller batch on the
  // persistent one.
  if (dw_wide_fits(p)) return run_dw_wide(p, s);
  if (dw_sgd_fits(p) && opt(IMBD_OPT_DW_GENERIC) == 0) return run_dw_sgd(p, s);
  const TileCfg &c = kCfgs[pl.cfg];
  KernelFn fn = c.fn[p.dtype == IMBD_BF16][p.a_kc][p.b_kc];
  const int grid = g.tiles_m * g.tiles_n * g.splits;
  {
    LaunchTimer t(p.kclass, p.layer, s);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(c.nt), 0, s, g);
  }
  int rc = check_launch("gemm");
  if (rc != IMBD_OK) return rc;
  if (p.db_mode != 0 && pl.splits > 1) {
    // the in-kernel row sums need the whole K range in one workgroup
    rc = run_bias_grad(p.dtype, p.N, p.K, p.B, p.ldb, p.db_alpha, p.db_mode == 1 ? p.db_out : nullptr,
                       p.db_mode == 2 ? p.bias : nullptr, p.bias_lr, s, p.layer);
    if (rc != IMBD_OK) return rc;
  }
  if (pl.splits > 1) rc = launch_reduce(p, g, s);
  return rc;
}

// ------------------------------------------------------------------ 3x3 conv tile
// The three passes of a 3x3, stride-1 conv on a tile whose 1-pixel halo is in place
// (Sec. 2.2 of the paper, domain parallelism), as implicit GEMMs over the positions P of
// the padded (H+2) x (W+2) grid. Positions are numbered up to the last interior pixel, so
// every shifted row stays inside the padded tensors.
//  pass 1  y[P][o]      = sum_{tap,c} w[o][tap][c] x_pad[P + r*(W+2) + s][c]
//  pass 2  dx[P][c]     = sum_{tap,o} w[o][tap][c] dy_pad[P + (2-r)*(W+2) + 2-s][o]
//  pass 3  dw[o][tap][c] = sum_{P inside} dy_pad[P + (W+2) + 1][o] x_pad[P + r*(W+2) + s][c]
namespace {
struct ConvPlan {
  int M, N, K, cfg, bm, bn, splits, k_split;
  size_t ws_bytes;
};

ConvPlan conv_plan(int pass, int N, int H, int W, int Ci, int Co) {
  ConvPlan p{};
  const int64_t Pext = (int64_t)(N - 1) * (H + 2) * (W + 2) + (int64_t)(H - 1) * (W + 2) + W;
  p.M = pass == 1 ? Co : (pass == 2 ? Ci : 9 * Ci);
  p.N = pass == 3 ? Co : (int)Pext;
  p.K = pass == 1 ? 9 * Ci : (pass == 2 ? 9 * Co : (int)Pext);
  // a weight-gradient tile must stay inside one tap (C_in % BM == 0)
  p.cfg = (Ci % 128 == 0 && Co % 128 == 0 && p.M >= 128 && p.N >= 128) ? 1 : 0;
  p.bm = p.bn = p.cfg == 1 ? 128 : 64;
  const int tiles = cdiv(p.M, p.bm) * cdiv(p.N, p.bn);
  const int BK = 64, ktiles = cdiv(p.K, BK);
  int splits = 1;
  if (pass == 3 && tiles < 512 && ktiles >= 16) {
    splits = cdiv(512, tiles);
    if (splits > ktiles / 4) splits = ktiles / 4;
    if (splits < 1) splits = 1;
  }
  p.k_split = cdiv(cdiv(p.K, splits), BK) * BK;
  p.splits = cdiv(p.K, p.k_split);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * (size_t)partial_split_stride(p.M, p.N) * sizeof(float) : 0;
  return p;
}
}  // namespace

size_t conv_wgrad_ws_bytes(int N, int H, int W, int Ci, int Co) {
  if (Ci % 64 || Co % 64) return 0;
  size_t b = conv_plan(3, N, H, W, Ci, Co).ws_bytes;
  if (N >= 1 && conv_wg_fits(N, H, W, Ci, Co, nullptr, nullptr, nullptr)) {
    // the large-tile kernel's split partials (it always goes through them)
    int splits, k_split;
    conv_wg_plan(N, H, W, Ci, &splits, &k_split);
    const size_t w = (size_t)splits * (size_t)partial_split_stride(9 * Ci, Co) * sizeof(float);
    if (w > b) b = w;
  }
  return b;
}

static int conv_launch(int pass, int N, int H, int W, int Ci, int Co, const void *A, const void *B, void *out,
                       int out_dtype, void *ws, size_t ws_bytes, hipStream_t s) {
  if (Ci % 64 || Co % 64) {
    set_error("conv tile needs C_in and C_out multiples of 64 (got %d, %d)", Ci, Co);
    return IMBD_EUNSUPPORTED;
  }
  if (pass != 3 && conv_nt_fits(pass, N, H, W, Ci, Co, B, A, out))
    return run_conv_nt(pass, N, H, W, Ci, Co, B, A, out, out_dtype, s);
  if (pass == 3 && conv_wg_fits(N, H, W, Ci, Co, A, B, out)) {
    int splits, k_split;
    conv_wg_plan(N, H, W, Ci, &splits, &k_split);
    KArgs g{};
    g.M = 9 * Ci;
    g.N = Co;
    g.splits = splits;
    g.partial = reinterpret_cast<float *>(ws);
    g.ldp = partial_ld(g.M);
    g.sstride = partial_split_stride(g.M, g.N);
    g.epi = Epilogue{};
    g.epi.mode = EPI_STORE;
    g.epi.out = out;
    g.epi.out_dtype = IMBD_F32;
    g.epi.ldo = 9 * Ci;
    const size_t need = (size_t)splits * (size_t)g.sstride * sizeof(float);
    if (ws == nullptr || ws_bytes < need || (uintptr_t)ws % 16) {
      set_error("conv weight gradient needs %zu bytes of 16-byte aligned workspace, got %zu", need, ws_bytes);
      return IMBD_EWORKSPACE;
    }
    {
      const int rc = run_conv_wg(N, H, W, Ci, Co, A, B, g.partial, g.ldp, g.sstride, s);
      if (rc != IMBD_OK) return rc;
    }
    {
      LaunchTimer t(IMBD_K_SPLITK, 0, s);
      const dim3 grid((unsigned)((g.M / 8 + 255) / 256), (unsigned)g.N);
      hipLaunchKernelGGL((splitk_reduce_fast<false, false>), grid, dim3(256), 0, s, g);
    }
    return check_launch("conv3x3 reduce");
  }
  const ConvPlan pl = conv_plan(pass, N, H, W, Ci, Co);
  if ((int64_t)N * (H + 2) * (W + 2) * (Ci > Co ? Ci : Co) >= ((int64_t)1 << 31)) {
    set_error("conv tile too large for 32-bit element offsets");
    return IMBD_EUNSUPPORTED;
  }
  if (pl.splits > 1 && (ws == nullptr || ws_bytes < pl.ws_bytes || (uintptr_t)ws % 16)) {
    set_error("conv weight gradient needs %zu bytes of 16-byte aligned workspace, got %zu", pl.ws_bytes, ws_bytes);
    return IMBD_EWORKSPACE;
  }
  for (const void *p : {A, B, (const void *)out})
    if ((uintptr_t)p % 16) {
      set_error("conv tensors must be 16-byte aligned");
      return IMBD_EINVAL;
    }
  KArgs g{};
  g.A = A;
  g.B = pass == 3 ? (const void *)(reinterpret_cast<const uint16_t *>(B) + (int64_t)(W + 3) * Co) : B;
  g.lda = pass == 3 ? Ci : 9 * Ci;
  g.ldb = pass == 1 ? Ci : Co;
  g.M = pl.M;
  g.N = pl.N;
  g.K = pl.K;
  g.k_split = pl.k_split;
  g.splits = pl.splits;
  g.tiles_m = cdiv(pl.M, pl.bm);
  g.tiles_n = cdiv(pl.N, pl.bn);
  g.a_vec = g.b_vec = 1;
  g.out_vec = 1;
  g.fast_ok = 1;
  g.mask_vec = g.bias_vec = 0;
  g.epi = Epilogue{};
  g.epi.mode = EPI_STORE;
  g.epi.out = out;
  g.epi.out_dtype = pass == 3 ? IMBD_F32 : out_dtype;
  g.epi.ldo = pass == 1 ? Co : (pass == 2 ? Ci : 9 * Ci);
  g.partial = reinterpret_cast<float *>(ws);
  g.ldp = partial_ld(pl.M);
  g.sstride = partial_split_stride(pl.M, pl.N);
  g.cH = H;
  g.cW = W;
  g.cCi = Ci;
  g.cCo = Co;
  const int cls = pass == 1 ? IMBD_K_CONV_FWD : (pass == 2 ? IMBD_K_CONV_DGRAD : IMBD_K_CONV_WGRAD);
  {
    LaunchTimer t(cls, 0, s);
    hipLaunchKernelGGL(kConvFns[pl.cfg][pass - 1], dim3(g.tiles_m * g.tiles_n * g.splits), dim3(256), 0, s, g);
  }
  int rc = check_launch("conv3x3");
  if (rc != IMBD_OK || pl.splits == 1) return rc;
  {
    LaunchTimer t(IMBD_K_SPLITK, 0, s);
    const dim3 grid((unsigned)((pl.M / 8 + 255) / 256), (unsigned)pl.N);
    hipLaunchKernelGGL((splitk_reduce_fast<false, false>), grid, dim3(256), 0, s, g);
  }
  return check_launch("conv3x3 reduce");
}

int run_conv_fwd(int N, int H, int W, int Ci, int Co, const void *xp, const void *w, void *y, int y_dtype,
                 hipStream_t s) {
  return conv_launch(1, N, H, W, Ci, Co, w, xp, y, y_dtype, nullptr, 0, s);
}
int run_conv_dgrad(int N, int H, int W, int Ci, int Co, const void *dyp, const void *w, void *dx, int dx_dtype,
                   hipStream_t s) {
  return conv_launch(2, N, H, W, Ci, Co, w, dyp, dx, dx_dtype, nullptr, 0, s);
}
int run_conv_wgrad(int N, int H, int W, int Ci, int Co, const void *xp, const void *dyp, float *dw, void *ws,
                   size_t ws_bytes, hipStream_t s) {
  if (N == 0) {  // an empty tile contributes a zero partial
    if (hipMemsetAsync(dw, 0, (size_t)Co * 9 * Ci * sizeof(float), s) != hipSuccess) return check_launch("memset");
    return IMBD_OK;
  }
  return conv_launch(3, N, H, W, Ci, Co, xp, dyp, dw, IMBD_F32, ws, ws_bytes, s);
}

}  // namespace imbd
