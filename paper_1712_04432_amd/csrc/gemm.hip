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

#include "common.h"

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

// Operand with k contiguous in memory: the tile is R rows x 128 bytes, 8 chunks per row.
template <typename T, int R, int NT>
struct KcLoader {
  static constexpr int VEC = Elem<T>::VEC;
  static constexpr int CH = R * 8;
  static constexpr int PER = (CH + NT - 1) / NT;
  u32x4 v[PER];

  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int rows, int k0,
                                       int kend, bool vec_ok, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (CH % NT == 0 || c < CH) {
        const int r = c >> 3, kc = c & 7;
        const int grow = row0 + r;
        const int kk = k0 + kc * VEC;
        const int valid = (grow < rows) ? (kend - kk) : 0;
        v[i] = load16<T>(base + (int64_t)grow * ld + kk, valid, vec_ok);
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

  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int rows, int k0,
                                       int kend, bool vec_ok, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int blk = tid + i * NT;
      if (NB % NT == 0 || blk < NB) {
        const int kb = blk & 7, rb = blk >> 3;
        const int col = row0 + rb * VEC;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const int k = k0 + kb * VEC + j;
          const int valid = (k < kend) ? (rows - col) : 0;
          v[i][j] = load16<T>(base + (int64_t)k * ld + col, valid, vec_ok);
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

struct KArgs {
  const void *A;
  const void *B;
  int64_t lda, ldb;
  int M, N, K;
  int k_split, splits, tiles_m, tiles_n;
  int a_vec, b_vec, out_vec;
  Epilogue epi;
  float *partial;  // [splits][N][ldp] when splits > 1
  int64_t ldp;
};

// ------------------------------------------------------------------------- epilogue
__device__ __forceinline__ bool mask_keep(const Epilogue &e, int m, int n) {
  if (!e.mask) return true;
  const int64_t off = (int64_t)n * e.ldmask + m;
  const float v = (e.mask_dtype == IMBD_BF16)
                      ? bf16_to_f32(reinterpret_cast<const uint16_t *>(e.mask)[off])
                      : reinterpret_cast<const float *>(e.mask)[off];
  return v > 0.0f;
}

// Finish up to 4 consecutive outputs (m..m+3, n); v holds the accumulated sums.
__device__ __forceinline__ void epilogue4(const Epilogue &e, int M, int m, int n, const float v[4],
                                          bool vec_ok) {
  const int cnt = (M - m) < 4 ? (M - m) : 4;
  if (e.mode == EPI_SGD) {
    float *w = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    float nw[4];
    if (cnt == 4 && vec_ok) {
      f32x4 old = *reinterpret_cast<const f32x4 *>(w);
#pragma unroll
      for (int i = 0; i < 4; ++i) nw[i] = fmaf(-e.lr, e.alpha * v[i], old[i]);
      *reinterpret_cast<f32x4 *>(w) = f32x4{nw[0], nw[1], nw[2], nw[3]};
      if (e.out2) {
        uint16_t *w2 = e.out2 + (int64_t)n * e.ldo2 + m;
        u32x2 pk;
        pk[0] = (uint32_t)f32_to_bf16(nw[0]) | ((uint32_t)f32_to_bf16(nw[1]) << 16);
        pk[1] = (uint32_t)f32_to_bf16(nw[2]) | ((uint32_t)f32_to_bf16(nw[3]) << 16);
        *reinterpret_cast<u32x2 *>(w2) = pk;
      }
    } else {
      for (int i = 0; i < cnt; ++i) {
        nw[i] = fmaf(-e.lr, e.alpha * v[i], w[i]);
        w[i] = nw[i];
        if (e.out2) e.out2[(int64_t)n * e.ldo2 + m + i] = f32_to_bf16(nw[i]);
      }
    }
    return;
  }
  float x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = e.alpha * v[i];
    if (i < cnt) {
      if (e.bias) t += e.bias[m + i];
      if (e.relu) t = t > 0.0f ? t : 0.0f;
      if (!mask_keep(e, m + i, n)) t = 0.0f;
    }
    x[i] = t;
  }
  if (e.out_dtype == IMBD_BF16) {
    uint16_t *o = reinterpret_cast<uint16_t *>(e.out) + (int64_t)n * e.ldo + m;
    if (cnt == 4 && vec_ok) {
      u32x2 pk;
      pk[0] = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
      pk[1] = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
      *reinterpret_cast<u32x2 *>(o) = pk;
    } else {
      for (int i = 0; i < cnt; ++i) o[i] = f32_to_bf16(x[i]);
    }
  } else {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)n * e.ldo + m;
    if (cnt == 4 && vec_ok) {
      *reinterpret_cast<f32x4 *>(o) = f32x4{x[0], x[1], x[2], x[3]};
    } else {
      for (int i = 0; i < cnt; ++i) o[i] = x[i];
    }
  }
}

// --------------------------------------------------------------------------- kernel
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, bool A_KC, bool B_KC>
__global__ void __launch_bounds__(64 * WAVES_M *WAVES_N)
    gemm_kernel(KArgs g) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int BK = KT_BYTES / (int)sizeof(T);
  constexpr int STAGE_A = BM * LDS_PITCH, STAGE = (BM + BN) * LDS_PITCH;
  static_assert(WM % 16 == 0 && WN % 16 == 0, "wave tile must be a multiple of 16");
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const int tid = threadIdx.x;
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
  const int tn = rem / g.tiles_m;
  const int tm = rem - tn * g.tiles_m;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = s * g.k_split;
  const int kend = min(g.K, kbeg + g.k_split);
  const int nk = (kend > kbeg) ? (kend - kbeg + BK - 1) / BK : 0;

  const T *A = reinterpret_cast<const T *>(g.A);
  const T *Bp = reinterpret_cast<const T *>(g.B);
  typename LoaderSel<T, BM, NT, A_KC>::type la;
  typename LoaderSel<T, BN, NT, B_KC>::type lb;

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    la.load(A, g.lda, m0, g.M, kbeg, kend, g.a_vec, tid);
    lb.load(Bp, g.ldb, n0, g.N, kbeg, kend, g.b_vec, tid);
    la.store(smem, tid);
    lb.store(smem + STAGE_A, tid);
  }
  __syncthreads();

  const int fr = lane & 15, fg = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = (kt + 1) < nk;
    if (more) {
      const int k0 = kbeg + (kt + 1) * BK;
      la.load(A, g.lda, m0, g.M, k0, kend, g.a_vec, tid);
      lb.load(Bp, g.ldb, n0, g.N, k0, kend, g.b_vec, tid);
    }
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
    if (more) {
      char *dst = smem + ((kt + 1) & 1) * STAGE;
      la.store(dst, tid);
      lb.store(dst + STAGE_A, tid);
    }
    __syncthreads();
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
        epilogue4(g.epi, g.M, m, n, v, g.out_vec);
      } else {
        float *p = g.partial + ((int64_t)s * g.N + n) * g.ldp + m;
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
    f32x4 a = *reinterpret_cast<const f32x4 *>(g.partial + (int64_t)n * g.ldp + m);
    for (int s = 1; s < g.splits; ++s) {
      const f32x4 b = *reinterpret_cast<const f32x4 *>(g.partial + ((int64_t)s * g.N + n) * g.ldp + m);
      a += b;
    }
    const float v[4] = {a[0], a[1], a[2], a[3]};
    epilogue4(g.epi, g.M, m, n, v, g.out_vec);
  }
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

int env_int(const char *name, int dflt) {
  const char *v = getenv(name);
  return (v && *v) ? atoi(v) : dflt;
}

inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

}  // namespace

GemmPlan gemm_plan(const GemmProblem &p) {
  GemmPlan pl{};
  const int esz = p.dtype == IMBD_BF16 ? 2 : 4;
  const int BK = KT_BYTES / esz;
  // Tile: the largest configuration that still gives a reasonable number of tiles.
  int cfg = 0;
  if (p.M >= 128 && p.N >= 128) cfg = 1;
  else if (p.M >= 128) cfg = 2;
  else if (p.N >= 128) cfg = 3;
  const int forced = env_int("IMBD_GEMM_CFG", -1);
  if (forced >= 0 && forced < kNumCfgs) cfg = forced;
  pl.cfg = cfg;
  pl.bm = kCfgs[cfg].bm;
  pl.bn = kCfgs[cfg].bn;
  const int tiles = cdiv(p.M, pl.bm) * cdiv(p.N, pl.bn);
  // Split K while there are too few tiles to fill 256 CUs twice, keeping >= 4 K tiles
  // per split; short products are left whole (a second launch would cost more).
  int splits = 1;
  const int ktiles = cdiv(p.K, BK);
  if (tiles < 512 && ktiles >= 16) {
    splits = cdiv(512, tiles);
    const int max_s = ktiles / 4;
    if (splits > max_s) splits = max_s;
    if (splits < 1) splits = 1;
  }
  const int forced_s = env_int("IMBD_GEMM_SPLITS", -1);
  if (forced_s >= 1) splits = forced_s < ktiles ? forced_s : (ktiles > 0 ? ktiles : 1);
  int k_split = cdiv(cdiv(p.K > 0 ? p.K : 1, splits), BK) * BK;
  splits = p.K > 0 ? cdiv(p.K, k_split) : 1;
  pl.splits = splits;
  pl.k_split = k_split;
  const int64_t ldp = ((int64_t)p.M + 3) / 4 * 4;
  pl.ws_bytes = splits > 1 ? (size_t)splits * (size_t)p.N * (size_t)ldp * sizeof(float) : 0;
  return pl;
}

int gemm_run(const GemmProblem &p, void *ws, size_t ws_bytes, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return IMBD_OK;
  const GemmPlan pl = gemm_plan(p);
  if (pl.splits > 1 && (ws == nullptr || ws_bytes < pl.ws_bytes)) {
    set_error("product %dx%dx%d needs %zu bytes of workspace for split-K partials, got %zu",
              p.M, p.N, p.K, pl.ws_bytes, ws_bytes);
    return IMBD_EWORKSPACE;
  }
  if (pl.splits > 1 && (uintptr_t)ws % 16 != 0) {
    set_error("workspace must be 16-byte aligned");
    return IMBD_EINVAL;
  }
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
  g.epi = p.epi;
  g.partial = reinterpret_cast<float *>(ws);
  g.ldp = ((int64_t)p.M + 3) / 4 * 4;

  const TileCfg &c = kCfgs[pl.cfg];
  KernelFn fn = c.fn[p.dtype == IMBD_BF16][p.a_kc][p.b_kc];
  const int grid = g.tiles_m * g.tiles_n * g.splits;
  {
    LaunchTimer t(p.kclass, p.layer, s);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(c.nt), 0, s, g);
  }
  int rc = check_launch("gemm");
  if (rc != IMBD_OK) return rc;
  if (pl.splits > 1) {
    const int64_t total = (int64_t)p.N * ((p.M + 3) / 4);
    int blocks = (int)((total + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    {
      LaunchTimer t(IMBD_K_SPLITK, p.layer, s);
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, g);
    }
    rc = check_launch("splitk_reduce");
  }
  return rc;
}

}  // namespace imbd
