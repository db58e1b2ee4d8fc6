// Device side of the large-tile weight-gradient kernel (fused SGD update or fp32 store);
// the kernel itself, its planning and its launch are in dw_wide.hip. Its workgroup body is
// a function of its own so that a launch can also run it beside another product's
// workgroups (the local backward pass's independent Delta_X and Delta_W products).
//   Delta_W[o][i] = sum_b Delta_Y[b][o] X[b][i]      (Sec. 1, K = the batch)
//   w[o][i] -= lr * alpha * Delta_W[o][i];  w16[o][i] = bf16(w[o][i])   (Eq. (1))
#pragma once

#include "cdna4.h"

namespace imbd {

constexpr int DL_NX = 4, DL_ND = 3;  // ring slots
constexpr int DL_PITCH = 128 + 4;    // staging row pitch in floats
constexpr int DL_GM = 8;             // o tiles per launch-order group (twice that on two workgroups per CU)
constexpr int CPOL_MASTER_LD = 2;      // nt
constexpr int CPOL_MASTER_ST = 2 | 16;  // nt, device scope
constexpr int CPOL_COPY_ST = 16;        // device scope

struct DlArgs {
  const uint16_t *X;   // [K][ldx], M columns
  const uint16_t *DY;  // [K][lddy], N columns
  int64_t ldx, lddy;
  uint32_t x_bytes, dy_bytes;
  int M, N, K;
  float *w;            // [N][ldw] fp32 masters
  uint16_t *w16;       // [N][ldw16] bf16 copy
  int64_t ldw, ldw16;
  uint32_t w_bytes, w16_bytes;
  float lr, alpha;
  int tiles_o, tiles_i;
  // bias gradient, db[o] = db_alpha * sum_b Delta_Y[b][o], by the workgroups of the first
  // column tile (db_mode 0: none (a separate launch), 1: store db_out, 2: bias -= bias_lr * db)
  int db_mode;
  float db_alpha, bias_lr;
  float *db_out, *bias;
  // Delta_Y's rows only 4-byte aligned (pitch and base): loaded in 4-byte pieces
  int dy_dw4;
  // a wide-batch product's split-K reduce (mask, bf16 output) carried by the fused-update
  // launch: its tail_items items shared out over the workgroups after their tiles
  LeanReduceArgs tail;
  int64_t tail_items;
};

__device__ __forceinline__ int dl_swz(int r) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1); }

// SGD: update the masters and the bf16 copy; else store alpha * Delta_W to w (fp32).
// OH: output rows o per workgroup, 256 or 128 (half the tile where whole tiles would leave
// most CUs idle in the last round).
// DUAL (OH = 128): two workgroups per CU (80 KB of LDS and at most 128 registers a lane
// each: 32-sample slabs in five-slot rings, fragments read one k-step at a time), so that
// one workgroup's update streams while the other computes its product.
// Bytes of LDS a workgroup of the kernel uses.
template <int OH, bool DUAL>
constexpr int dl_lds_bytes() {
  return (DUAL ? 5 : DL_ND) * (DUAL ? 32 : 64) * 2 * OH + (DUAL ? 5 : DL_NX) * (DUAL ? 32 : 64) * 256;
}

// One workgroup's tile: bid is its index in the launch order of the G (a multiple of 8)
// workgroups that share the work, smem its LDS (dl_lds_bytes<OH, DUAL>() bytes).
template <bool SGD, int OH, bool DUAL>
__device__ __forceinline__ void dw_wide_body(const DlArgs &a, char *smem, int bid, int G) {
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int NQ = OH / 64;                 // 64-column quarters of the Delta_Y slab
  constexpr int SK = DUAL ? 32 : 64;          // samples per slab
  constexpr int QB = SK / 8;                  // 1 KB blocks (8 samples x 128 B) per quarter
  constexpr int QSLOT = SK * 128;             // one 64-column quarter of a slab
  constexpr int DSLOT = SK * 2 * OH;          // SK samples x OH columns
  constexpr int XSLOT = SK * 256;             // SK samples x 128 columns
  constexpr int ND = DUAL ? 5 : DL_ND, NX = DUAL ? 5 : DL_NX;
  constexpr int DRING = ND * DSLOT, XRING = NX * XSLOT;
  static_assert(DRING + XRING == dl_lds_bytes<OH, DUAL>(), "LDS size");
  static_assert(!DUAL || OH == 128, "two workgroups per CU: 128-row tiles");
  static_assert(DRING + XRING <= (DUAL ? 80 : 160) * 1024, "LDS");
  static_assert(OH * DL_PITCH * 4 + 512 * 4 <= DRING + XRING, "staging and bias sums");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // G a multiple of 8; each XCD takes a contiguous range of the launch order,
  // in which tiles come in groups of GM o tiles x all i tiles (shared slabs in L2)
  constexpr int GM = DUAL ? 2 * DL_GM : DL_GM;
  int L = (bid & 7) * (G >> 3) + (bid >> 3);
  if (L >= a.tiles_o * a.tiles_i) return;
  const int og = L / (GM * a.tiles_i);
  const int gsz = min(GM, a.tiles_o - og * GM);
  L -= og * GM * a.tiles_i;
  const int it = L / gsz, ot = og * GM + (L - it * gsz);
  const int o0 = ot * OH, i0 = it * 128;
  const int nsl = (a.K + SK - 1) / SK;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t ldsd = lds0, ldsx = lds0 + DRING;
  // two workgroups per CU (SGD): each wave issues the loads of its masters as soon as its
  // part of the product is done (the loader waves after their last slab landed, the MMA
  // waves after their last MFMAs), so that they are in flight during the staging. (Loads
  // issued by the loader waves right after their last slab's loads, before that slab
  // landed, made the launch 3% slower.)
  constexpr bool EARLY = SGD && DUAL;
  // the update's share of each thread: rows o0 + 16u + sub (u < UR), columns i0 + 4ch .. +3
  constexpr int US = 16, UR = OH / US;
  const int ch = tid & 31, sub = tid >> 5;
  const int i = i0 + 4 * ch;
  const bool colok = i < a.M;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(a.w, 0, (int)a.w_bytes, BUF_DW3);
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(a.w16, 0, (int)a.w16_bytes, BUF_DW3);
  // rows past N and columns past M: an offset past the descriptor (reads zero, no store)
  auto offw = [&](int u) {
    const int o = o0 + US * u + sub;
    return (colok && o < a.N) ? (uint32_t)(((int64_t)o * a.ldw + i) * 4) : OOB;
  };
  f32x4 wold[UR];
  auto load_masters = [&]() {
#pragma unroll
    for (int u = 0; u < UR; ++u)
      wold[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, offw(u), 0, CPOL_MASTER_LD));
  };

  if (wave >= 6) {
    // ---------------------------------------------------- Delta_Y loaders (6, 7)
    // the wave's blocks: quarters (NQ/2) dw .. (NQ/2) dw + NQ/2 - 1, k-rows 8g + lane/8
    constexpr int QN = QB * NQ / 2;  // 1 KB blocks per wave
    const int dw = wave - 6;
    const i32x4 rd = buf_rsrc(a.DY, a.dy_bytes);
    const uint32_t sstep = (uint32_t)(SK * a.lddy * 2);
    // Rows 4-byte aligned only: each 16-byte chunk of the layout below comes as four 4-byte
    // loads. Instruction i of a 1 KB block fills its bytes 256i .. 256i + 255: lane l loads
    // dword l%4 of the chunk that lane 16i + l/4 loads in the 16-byte form. Columns past N
    // feed only outputs that are not stored; the descriptor ends at the last sample's
    // column N (N even).
    constexpr bool DW4_OK = 4 * QN * (ND - 2) <= 63;  // the memory counter's range
    if (DW4_OK && a.dy_dw4) {
      uint32_t b4[QN][4];
#pragma unroll
      for (int q = 0; q < QN; ++q) {
        const int h = (NQ / 2) * dw + q / QB, g = q % QB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int L = 16 * i + (lane >> 2);
          const int r = 8 * g + (L >> 3);
          const int c = (L & 7) ^ dl_swz(r);
          b4[q][i] = (uint32_t)(((int64_t)r * a.lddy + o0 + 64 * h + 8 * c) * 2 + 4 * (lane & 3));
        }
      }
      auto issue4 = [&](int S) {
        const uint32_t slot = ldsd + (uint32_t)((S % ND) * DSLOT);
#pragma unroll
        for (int q = 0; q < QN; ++q) {
          const int h = (NQ / 2) * dw + q / QB, g = q % QB;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            dma4(rd, S < nsl ? b4[q][i] + (uint32_t)S * sstep : OOB,
                 slot + (uint32_t)(h * QSLOT + g * 1024 + 256 * i));
        }
      };
#pragma unroll
      for (int S = 0; S < ND - 1; ++S) issue4(S);
      for (int S = 0; S < nsl; ++S) {
        vm_barrier<(DW4_OK ? 4 : 1) * QN * (ND - 2)>();  // slab S landed: B_S
        issue4(S + ND - 1);                              // into the slot of S-1
      }
    } else {
      uint32_t base[QN], dst[QN];
#pragma unroll
      for (int q = 0; q < QN; ++q) {
        const int h = (NQ / 2) * dw + q / QB, g = q % QB;
        const int r = 8 * g + (lane >> 3);
        const int c = (lane & 7) ^ dl_swz(r);
        base[q] = (uint32_t)(((int64_t)r * a.lddy + o0 + 64 * h + 8 * c) * 2);
        dst[q] = (uint32_t)(h * QSLOT + g * 1024);
      }
      auto issue = [&](int S) {
        const uint32_t slot = ldsd + (uint32_t)((S % ND) * DSLOT);
#pragma unroll
        for (int q = 0; q < QN; ++q) dma16(rd, S < nsl ? base[q] + (uint32_t)S * sstep : OOB, slot + dst[q]);
      };
#pragma unroll
      for (int S = 0; S < ND - 1; ++S) issue(S);
      for (int S = 0; S < nsl; ++S) {
        vm_barrier<QN * (ND - 2)>();  // slab S landed: B_S
        issue(S + ND - 1);            // into the slot of S-1
      }
    }
    vm_barrier<0>();
    if constexpr (EARLY) load_masters();
  } else if (wave >= 4) {
    // --------------------------------------------------------- X loaders (4, 5)
    const int xw = wave - 4;
    const i32x4 rx = buf_rsrc(a.X, a.x_bytes);
    uint32_t base[QB], dst[QB];
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const int r = 8 * q + (lane >> 3);
      const int c = (lane & 7) ^ dl_swz(r);
      base[q] = (uint32_t)(((int64_t)r * a.ldx + i0 + 64 * xw + 8 * c) * 2);
      dst[q] = (uint32_t)(xw * QSLOT + q * 1024);
    }
    const uint32_t sstep = (uint32_t)(SK * a.ldx * 2);
    auto issue = [&](int S) {
      const uint32_t slot = ldsx + (uint32_t)((S % NX) * XSLOT);
#pragma unroll
      for (int q = 0; q < QB; ++q) dma16(rx, S < nsl ? base[q] + (uint32_t)S * sstep : OOB, slot + dst[q]);
    };
#pragma unroll
    for (int S = 0; S < NX - 1; ++S) issue(S);
    for (int S = 0; S < nsl; ++S) {
      vm_barrier<QB * (NX - 2)>();  // slab S landed: B_S
      issue(S + NX - 1);           // into the slot of S-1
    }
    vm_barrier<0>();
    if constexpr (EARLY) load_masters();
  } else {
    // --------------------------------------------------------------- MMA group
    // wave (wm, wn): rows o (OH/2)wm.. (Delta_Y quarters (NQ/2)wm ..), columns i 64wn..
    constexpr int FM = OH / 32;
    const int fi = lane & 15, kg = lane >> 4;
    const int wm = wave & 1, wn = wave >> 1;
    const int r = 8 * kg + (fi >> 2);
    uint32_t fa[FM], fx[4];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int mb = FM * wm + i, h = mb >> 2, ib = mb & 3;
      const int c = (2 * ib + ((fi >> 1) & 1)) ^ dl_swz(r);
      fa[i] = (uint32_t)(h * QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = (2 * j + ((fi >> 1) & 1)) ^ dl_swz(r);
      fx[j] = (uint32_t)(wn * QSLOT + r * 128 + c * 16 + 8 * (fi & 1));
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
    auto mma = [&](const bf16x8 (&df)[FM], const bf16x8 (&xf)[4]) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(df[i], xf[j], acc[i][j], 0, 0, 0);
    };
    uint32_t ds = ldsd, xs = ldsx;
    lds_barrier();  // B_0
    if constexpr (DUAL) {
      // one k-step (the whole 32-sample slab) at a time (register budget of two workgroups
      // per CU); the other workgroup's waves cover the read latency
      for (int S = 0; S < nsl; ++S) {
        read(ds, xs, 0, dv[0], xv[0]);
        mma(dv[0], xv[0]);
        lds_barrier();  // B_{S+1}
        ds = ldsd + (uint32_t)(((S + 1) % ND) * DSLOT);
        xs = ldsx + (uint32_t)(((S + 1) % NX) * XSLOT);
      }
    } else {
      read(ds, xs, 0, dv[0], xv[0]);
      for (int S = 0; S < nsl; ++S) {
        read(ds, xs, 1, dv[1], xv[1]);
        __builtin_amdgcn_sched_barrier(0);
        mma(dv[0], xv[0]);
        __builtin_amdgcn_sched_barrier(0);
        lds_barrier();  // B_{S+1}
        ds = ldsd + (uint32_t)(((S + 1) % ND) * DSLOT);
        xs = ldsx + (uint32_t)(((S + 1) % NX) * XSLOT);
        read(ds, xs, 0, dv[0], xv[0]);  // past the last slab this reads a spent slot, unused
        __builtin_amdgcn_sched_barrier(0);
        mma(dv[1], xv[1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if constexpr (EARLY) load_masters();
    // ---- stage the tile as [o][i] fp32
    float *stg = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          stg[(16 * (FM * wm + i) + 4 * kg + e) * DL_PITCH + 16 * (4 * wn + j) + fi] = acc[i][j][e];
  }
  if (it == 0 && a.db_mode != 0) {
    // ---- bias gradient of the tile's OH rows o: thread t sums column o0 + t%OH over the
    // samples of its part (t/OH of 512/OH parts) in ascending order, the parts are added
    // in order. The staged tile leaves LDS free past it.
    __syncthreads();
    constexpr int NP = 512 / OH;
    float *part = reinterpret_cast<float *>(smem + OH * DL_PITCH * 4);
    const int col = tid % OH, pi = tid / OH, o = o0 + col;
    const int kh = (a.K + NP - 1) / NP, b0 = min(a.K, pi * kh), b1 = min(a.K, b0 + kh);
    float sum = 0.f;
    if (o < a.N) {
      const uint16_t *p = a.DY + o;
      int b = b0;
      for (; b + 8 <= b1; b += 8) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = bf16_to_f32(p[(int64_t)(b + q) * a.lddy]);
#pragma unroll
        for (int q = 0; q < 8; ++q) sum += v[q];
      }
      for (; b < b1; ++b) sum += bf16_to_f32(p[(int64_t)b * a.lddy]);
    }
    part[tid] = sum;
    __syncthreads();
    if (tid < OH && o < a.N) {
      float t = part[tid];
#pragma unroll
      for (int q = 1; q < NP; ++q) t += part[tid + q * OH];
      const float db = a.db_alpha * t;
      if (a.db_mode == 1) a.db_out[o] = db;
      else a.bias[o] -= a.bias_lr * db;
    }
  }
  // ---- the update: thread (sub, ch) takes rows o0 + US*u + sub (u < UR), columns
  // i0 + 4ch .. +3, with all its rows' masters in flight at once. One workgroup per CU: the
  // loads issued after the staging (eight rows in flight instead of sixteen: +1%; issued by
  // the loader waves before the last barrier: +9%). Two per CU: issued before the staging
  // (above; the loader waves alone doing the whole update, their loads issued during the
  // product, was 3% slower).
  const float *stg = reinterpret_cast<const float *>(smem);
  if constexpr (!SGD) {
    lds_barrier();
    if (!colok) return;
#pragma unroll
    for (int u = 0; u < UR; ++u) {
      const f32x4 g = *reinterpret_cast<const f32x4 *>(stg + (US * u + sub) * DL_PITCH + 4 * ch);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, a.alpha * g), rw, offw(u), 0, CPOL_COPY_ST);
    }
    return;
  }
  lds_barrier();
  if constexpr (!EARLY) load_masters();
  if (!colok) return;
#pragma unroll
  for (int u = 0; u < UR; ++u) {
    const int ol = US * u + sub, o = o0 + ol;
    const f32x4 g = *reinterpret_cast<const f32x4 *>(stg + ol * DL_PITCH + 4 * ch);
    f32x4 nw;
#pragma unroll
    for (int e = 0; e < 4; ++e) nw[e] = fmaf(-a.lr, a.alpha * g[e], wold[u][e]);
    u32x2 pk;
    pk[0] = cvt_pk_bf16(nw[0], nw[1]);
    pk[1] = cvt_pk_bf16(nw[2], nw[3]);
    const uint32_t offh = o < a.N ? (uint32_t)(((int64_t)o * a.ldw16 + i) * 2) : OOB;
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, nw), rw, offw(u), 0, CPOL_MASTER_ST);
    __builtin_amdgcn_raw_buffer_store_b64(pk, rh, offh, 0, CPOL_COPY_ST);
  }
}


// Fills the kernel's arguments for a problem dw_wide_fits() accepts; extra_blocks is the
// number of other workgroups launched before these in the same grid (they count in the
// choice of 128- or 256-row tiles). *oh is the tile height, *dual whether two workgroups
// share a CU, *grid the workgroups (a multiple of 8).
void dw_wide_prepare(const GemmProblem &p, int extra_blocks, DlArgs *a, int *oh, bool *dual, int *grid);

}  // namespace imbd
