// MXFP4-weight grouped expert GEMMs for gfx950 (CDNA4) block-scaled MFMA.
//
// Expert weights are MXFP4 (e2m1 codes, one E8M0 scale per 32 elements along
// K), the precision the paper keeps DeepSeek-V4's routed experts in (Section
// 4.1).  Activations are quantised to MXFP8 (e4m3, E8M0 per 32 channels) by
// the pack step and h to MXFP8 in the GEMM1 epilogue, the quantisation step
// between the two expert GEMMs (Appendix C, "Grouped FFN invocations").  With
// both operands in MX form, v_mfma_scale_f32_16x16x128_f8f6f4 applies both
// scales itself: every K step accumulates straight into the float32
// accumulators, with no per-block promotion on the vector ALUs.
//
// Operand layout of that instruction (lane l: row or column l%16, group
// g = l/16): an e4m3 operand lane holds K [16g, 16g+16) in bytes 0-15 and
// K [64+16g, 64+16g+16) in bytes 16-31; an e2m1 operand lane holds
// K [32g, 32g+32) as 32 nibbles (low nibble first) in its first four dwords;
// the scale byte of lane l applies to K block g of its row or column.  The
// LDS reads below follow this so that hardware K equals data K.
#include "gemm_common.h"

#include <algorithm>

namespace cep {
namespace {

// One e2m1 x e4m3 block-scaled MFMA: the weight fragment w is the first
// operand (scale byte OW of the word sw), the activation fragment x the
// second (byte ox of sx), so that output lane l holds activation row l%16
// and four consecutive weight columns.  The instruction takes the byte
// selects as immediates: ox is a constant after the caller's loop is
// unrolled, and the switch folds away.
template <int OW>
__device__ inline f32x4 mx_mfma(const i32x8 &w, const i32x8 &x, const f32x4 &c, int ox, int sx,
                                int sw) {
  switch (ox) {
    case 0: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, c, 4, 0, OW, sw, 0, sx);
    case 1: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, c, 4, 0, OW, sw, 1, sx);
    case 2: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, c, 4, 0, OW, sw, 2, sx);
    default: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, c, 4, 0, OW, sw, 3, sx);
  }
}

// BM x 256 output tile, K step 128 (four scale blocks).  NW waves: four
// column groups of 64 x (NW/4) row groups of 128; each wave owns 128 rows x
// 64 columns = 8 x 4 16x16 fragments.  A stage holds BM x 128 e4m3 codes,
// 256 x 64 bytes of packed e2m1 weights, the BM x 4 row scales and the 256 x
// 4 weight scales, all brought by direct global->LDS loads issued STAGES-1
// steps ahead.  The scale layouts (mx_row_scale_offset,
// mx_weight_scale_offset) give each lane its eight row scales as one 8-byte
// word and its four column scales as one word; the MFMA's byte select picks
// the fragment's byte.
//
// LDS rows: A rows are 128 bytes (8 chunks), chunk c of row r at slot
// c ^ ((r >> 1) & 7); B rows are 64 bytes (4 chunks), chunk c at slot
// c ^ bsw(r), bsw(r) = (r & 1) | ((r >> 1) & 2).  A 16-byte LDS read serves
// per cycle the sixteen lanes of one half-wave whose quad index (lane bits
// 2-4) has one parity, on 64 four-byte banks (mapped lane pair by lane pair
// with SQ_LDS_BANK_CONFLICT); with these swizzles each such group reads
// sixteen distinct 16-byte slots of 256 bytes in both operand reads.
//
// Epilogues: store_h_mx_staged (GEMM1) and store_y_bf16 (GEMM2).  The
// 256-row tiles run as the persistent 8-wave kernel below (same stage, LDS
// layout and MFMA order, so both tile heights give bitwise equal outputs).
__device__ inline int bsw_of(int r) { return (r & 1) | ((r >> 1) & 2); }


template <int NW, int STAGES, bool SWIGLU, int OCC = 1>
__global__ __launch_bounds__(64 * NW, OCC) void k_gemm_mx(GemmArgs g) {
  constexpr int BM = 128 * NW / 4, BN = 256, BK = 128;
  constexpr int A_SEG = BM * BK / 1024, B_SEG = BN * (BK / 2) / 1024;
  constexpr int A_LD = A_SEG / NW, B_LD = B_SEG / NW;  // 1 KB loads per wave per step
  constexpr int PER = A_LD + B_LD;  // waves 0 and 1 add one each (row / weight scales)
  static_assert(A_SEG % NW == 0 && B_SEG % NW == 0, "loads split evenly over the waves");
  static_assert(BM * 4 <= 1024, "one load of the row scales");
  int mt, nt;
  if (!balanced_tile<kGroupM>(*g.n_tiles, g.N / BN, &mt, &nt)) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int K = g.K, nkb = K / BK, KB = K / 2;  // KB: bytes of one packed weight row
  const uint8_t *blob = blob_of(g.bt, t.expert);
  const char *Ag = (const char *)(g.A + (size_t)t.row0 * K);
  const char *Bg = (const char *)(blob + g.b_off);  // mx_block_index layout
  // row scales of K step kb: 512 bytes per 128-row group, groups contiguous
  const char *Asg = (const char *)g.As + (size_t)(t.row0 >> 7) * 512;
  const size_t as_step = (size_t)(g.s_ld >> 7) * 512;
  const char *Bsg = (const char *)(blob + g.bs_off) + (size_t)nt * nkb * 1024;

  __shared__ u32x4 sA[STAGES][BM * 8];
  __shared__ u32x4 sB[STAGES][BN * 4];
  __shared__ u32x4 sAs[STAGES][BM / 4];
  __shared__ u32x4 sBs[STAGES][64];

  const int a_row = lane >> 3, b_row = lane >> 2;
#define CEP_MX_STAGE(kb)                                                            \
  {                                                                                 \
    const int buf_ = (kb) % STAGES;                                                 \
    _Pragma("unroll") for (int i = 0; i < A_LD; ++i) {                              \
      const int seg = wid * A_LD + i, r = seg * 8 + a_row;                          \
      dma16(Ag + (size_t)(kb) * BK + (size_t)r * K + (((lane & 7) ^ ((r >> 1) & 7)) * 16), \
            __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf_][seg * 64])));       \
    }                                                                               \
    _Pragma("unroll") for (int i = 0; i < B_LD; ++i) {                              \
      const int seg = wid * B_LD + i, r = seg * 16 + b_row;                         \
      dma16(Bg + mx_block_index(nt * BN + r, (kb) * (BK / 2) + ((lane & 3) ^ bsw_of(r)) * 16, KB), \
            __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf_][seg * 64])));       \
    }                                                                               \
    if (wid == 0 && lane < BM / 4)                                                  \
      dma16(Asg + (size_t)(kb) * as_step + lane * 16,                               \
            __builtin_amdgcn_readfirstlane(lds_offset(&sAs[buf_][0])));             \
    if (wid == 1)                                                                   \
      dma16(Bsg + (size_t)(kb) * 1024 + lane * 16,                                  \
            __builtin_amdgcn_readfirstlane(lds_offset(&sBs[buf_][0])));             \
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{};

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nkb) CEP_MX_STAGE(s);

  float wr[8];
  int yd[8];  // GEMM2: output rows of the lane's rows (GemmArgs::ydst)
  if constexpr (!SWIGLU) {
    load_row_coef(g, t, wm, lane, wr);
    load_row_dst(g, t, wm, lane, yd);
  }
  const int r16 = lane & 15, grp = lane >> 4;
  const int asw = (r16 >> 1) & 7;  // A swizzle of every row this lane reads
  const int bsw = bsw_of(r16);     // B swizzle of every row this lane reads
  for (int kb = 0; kb < nkb; ++kb) {
    const int later = min(nkb - 1, kb + STAGES - 2) - kb;
    if (wid < 2)
      wait_stages<PER + 1, STAGES - 2>(later);
    else
      wait_stages<PER, STAGES - 2>(later);
    // every wave's loads of step kb landed; step kb-1 fully consumed
    __builtin_amdgcn_s_barrier();
    if (kb + STAGES - 1 < nkb) CEP_MX_STAGE(kb + STAGES - 1);
    const int cur = kb % STAGES;
    const uint32_t sb = ((const uint32_t *)&sBs[cur][0])[(wn * 4 + grp) * 16 + r16];
    const uint2 sa = ((const uint2 *)&sAs[cur][0])[wm * 64 + grp * 16 + r16];

    i32x8 b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = wn * 64 + j * 16 + r16;
      const u32x4 v = sB[cur][row * 4 + (grp ^ bsw)];
      b[j] = __builtin_bit_cast(i32x8, __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1));
    }
    // A fragments one row group ahead: the reads of group i+1 are issued
    // before the MFMAs of group i, so LDS latency hides behind them
    auto read_a = [&](int i) {
      const int row = wm * 128 + i * 16 + r16;
      const u32x4 lo = sA[cur][row * 8 + (grp ^ asw)];
      const u32x4 hi = sA[cur][row * 8 + ((grp + 4) ^ asw)];
      return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    i32x8 a_next = read_a(0);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const i32x8 a = a_next;
      if (i + 1 < 8) a_next = read_a(i + 1);
      __builtin_amdgcn_sched_barrier(0);
      const int sai = (int)(i < 4 ? sa.x : sa.y);
      acc[i][0] = mx_mfma<0>(b[0], a, acc[i][0], i & 3, sai, (int)sb);
      acc[i][1] = mx_mfma<1>(b[1], a, acc[i][1], i & 3, sai, (int)sb);
      acc[i][2] = mx_mfma<2>(b[2], a, acc[i][2], i & 3, sai, (int)sb);
      acc[i][3] = mx_mfma<3>(b[3], a, acc[i][3], i & 3, sai, (int)sb);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#undef CEP_MX_STAGE

  // GEMM1 stages BM x 128 code bytes through the A ring
  static_assert(sizeof(sA) >= BM * 128, "the h tile fits the A ring");
  if constexpr (SWIGLU) {
    store_h_mx_staged<NW>(acc, g, t, nt, wm, wn, lane, tid, &sA[0][0]);
  } else {
    store_y_bf16(acc, wr, yd, g, t, nt, wm, wn, lane);
  }
}


// Persistent 8-wave tiles, as the e4m3 GEMMs': one workgroup per CU walks
// its XCD's share of the tile order (work_item_xg).  After a tile's K loop
// it issues the next tile's first stage into ring buffer 0 (and, for
// GEMM2, the next tile's routing coefficients and output rows into LDS),
// then runs the epilogue through buffer 1 (GEMM2's y rows 64-127 of a pass
// through sY), storing every row so that each wave issues a fixed number of
// stores, and waits until at most those stores are outstanding: the next
// tile's loads have landed, the stores may still drain.
struct MxTile {
  Tile t;
  int nt;
  const char *Ag, *Bt, *Asg, *Bsg;
};

template <bool SWIGLU>
__global__ __launch_bounds__(512, 1) void k_gemm_mx_persist(GemmArgs g) {
  constexpr int NW = 8, BM = 256, BN = 256, BK = 128;
  constexpr int A_LD = BM * BK / 1024 / NW, B_LD = BN * (BK / 2) / 1024 / NW;
  const int n_live = __builtin_amdgcn_readfirstlane(*g.n_tiles), ntn = g.N / BN;
  int mt, nt;
  if (!work_item_xg<kGroupXcd>(0, n_live, ntn, &mt, &nt)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int K = g.K, nkb = K / BK, KB = K / 2;  // KB: bytes of one packed weight row
  const size_t as_step = (size_t)(g.s_ld >> 7) * 512;

  __shared__ u32x4 sA[2][BM * 8];
  __shared__ u32x4 sB[2][BN * 4];
  __shared__ u32x4 sAs[2][BM / 4];
  __shared__ u32x4 sBs[2][64];
  // GEMM2: the second 32 KB of a staged pass of y rows, the tile's routing
  // coefficients and (two buffers: the next tile's beside the current
  // epilogue) its rows' output rows
  __shared__ u32x4 sY[SWIGLU ? 1 : 64 * 32];
  __shared__ float sW[SWIGLU ? 1 : BM];
  __shared__ int sD[SWIGLU ? 1 : 2][SWIGLU ? 1 : BM];

  auto tile_at = [&](int mt_, int nt_) {
    MxTile f;
    mt_ = __builtin_amdgcn_readfirstlane(mt_);
    nt_ = __builtin_amdgcn_readfirstlane(nt_);
    f.t = g.tiles[mt_];
    f.nt = nt_;
    const uint8_t *blob = blob_of(g.bt, f.t.expert);
    f.Ag = (const char *)(g.A + (size_t)f.t.row0 * K);
    // the tile's 16 blocks of 16 weight rows (mx_block_index): K step kb
    // 1 KB further into each
    f.Bt = (const char *)(blob + g.b_off) + (size_t)nt_ * (BN / 16) * (KB >> 6) * 1024;
    f.Asg = (const char *)g.As + (size_t)(f.t.row0 >> 7) * 512;
    f.Bsg = (const char *)(blob + g.bs_off) + (size_t)nt_ * nkb * 1024;
    return f;
  };
  const int a_row = lane >> 3, b_row = lane >> 2;
  auto stage = [&](const MxTile &f, int kb, int buf) {
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int seg = wid * A_LD + i, r = seg * 8 + a_row;
      dma16(f.Ag + (size_t)kb * BK + (size_t)r * K + (((lane & 7) ^ ((r >> 1) & 7)) * 16),
            __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf][seg * 64])));
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int seg = wid * B_LD + i, r = seg * 16 + b_row;
      dma16(f.Bt + (size_t)kb * 1024 + mx_block_index(r, ((lane & 3) ^ bsw_of(r)) * 16, KB),
            __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf][seg * 64])));
    }
    if (wid == 0)
      dma16(f.Asg + (size_t)kb * as_step + lane * 16,
            __builtin_amdgcn_readfirstlane(lds_offset(&sAs[buf][0])));
    if (wid == 1)
      dma16(f.Bsg + (size_t)kb * 1024 + lane * 16,
            __builtin_amdgcn_readfirstlane(lds_offset(&sBs[buf][0])));
  };
  // GEMM2: the coefficients and output rows of the tile's BM rows, one 1 KB
  // load each by waves 2 and 3 (the rows of a tile lie inside the layout's
  // padded rows)
  auto stage_coef = [&](const MxTile &f, int db) {
    if constexpr (!SWIGLU) {
      if (wid == 2)
        dma16_s(g.wrow + f.t.row0, lane * 16, __builtin_amdgcn_readfirstlane(lds_offset(&sW[0])));
      if (g.ydst) {
        if (wid == 3)
          dma16_s(g.ydst + f.t.row0, lane * 16,
                  __builtin_amdgcn_readfirstlane(lds_offset(&sD[db][0])));
      } else if (tid < BM) {
        sD[db][tid] = -1;
      }
    }
  };

  MxTile cur = tile_at(mt, nt);
  stage(cur, 0, 0);
  int db = 0;
  stage_coef(cur, db);
  // the direct loads are invisible to the compiler: __syncthreads() alone
  // would not wait for them
  wait_vmcnt<0>();
  __syncthreads();

  const int r16 = lane & 15, grp = lane >> 4;
  const int asw = (r16 >> 1) & 7;  // A swizzle of every row this lane reads
  const int bsw = bsw_of(r16);     // B swizzle of every row this lane reads
  // stores each wave issues at least in a GEMM1 epilogue: BM x 128 code
  // bytes in 16-byte pieces by 512 threads (4), and one scale word
  constexpr int S_EPI = 4;
  for (int it = 0;; ++it) {
    f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{};
    for (int kb = 0; kb < nkb; ++kb) {
      // this wave's loads of step kb are its only ones outstanding (a
      // tile's first stage was waited for before its K loop)
      if (kb > 0) wait_vmcnt<0>();
      // every wave's loads of step kb landed; step kb-1 fully consumed
      __builtin_amdgcn_s_barrier();
      if (kb + 1 < nkb) stage(cur, kb + 1, (kb + 1) & 1);
      const int buf = kb & 1;
      const uint32_t sb = ((const uint32_t *)&sBs[buf][0])[(wn * 4 + grp) * 16 + r16];
      const uint2 sa = ((const uint2 *)&sAs[buf][0])[wm * 64 + grp * 16 + r16];
      i32x8 b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wn * 64 + j * 16 + r16;
        const u32x4 v = sB[buf][row * 4 + (grp ^ bsw)];
        b[j] = __builtin_bit_cast(i32x8, __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1));
      }
      auto read_a = [&](int i) {
        const int row = wm * 128 + i * 16 + r16;
        const u32x4 lo = sA[buf][row * 8 + (grp ^ asw)];
        const u32x4 hi = sA[buf][row * 8 + ((grp + 4) ^ asw)];
        return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      i32x8 a_next = read_a(0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const i32x8 a = a_next;
        if (i + 1 < 8) a_next = read_a(i + 1);
        __builtin_amdgcn_sched_barrier(0);
        const int sai = (int)(i < 4 ? sa.x : sa.y);
        acc[i][0] = mx_mfma<0>(b[0], a, acc[i][0], i & 3, sai, (int)sb);
        acc[i][1] = mx_mfma<1>(b[1], a, acc[i][1], i & 3, sai, (int)sb);
        acc[i][2] = mx_mfma<2>(b[2], a, acc[i][2], i & 3, sai, (int)sb);
        acc[i][3] = mx_mfma<3>(b[3], a, acc[i][3], i & 3, sai, (int)sb);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // GEMM2: outputs scaled by the coefficients and packed to bf16 before
    // the next tile's coefficients overwrite them
    uint32_t yb[SWIGLU ? 1 : 8][4][2];
    if constexpr (!SWIGLU) {
      float wr[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) wr[i] = sW[wm * 128 + i * 16 + r16];
      pack_y_bf16(acc, wr, yb);
    }
    int mt2, nt2;
    const bool more = work_item_xg<kGroupXcd>(it + 1, n_live, ntn, &mt2, &nt2);
    MxTile nxt;
    if (more) {
      // every wave's reads of the last step (and of sW) completed: buffer
      // 0 and sW may be refilled
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      nxt = tile_at(mt2, nt2);
      stage(nxt, 0, 0);
      stage_coef(nxt, db ^ 1);
    }
    static_assert(sizeof(sA[1]) >= BM * 128 && sizeof(sA[1]) >= 64 * 512 &&
                      sizeof(sY) >= (SWIGLU ? 16 : 64 * 512),
                  "staging fits buffer 1 and sY");
    int n_st = S_EPI;
    if constexpr (SWIGLU)
      store_h_mx_staged<NW, true>(acc, g, cur.t, cur.nt, wm, wn, lane, tid, &sA[1][0]);
    else
      n_st = store_y_bf16_staged<NW, true>(yb, g, cur.t, cur.nt, wm, wn, lane, tid, &sA[1][0],
                                           &sY[0], &sD[db][0]);
    if (!more) return;
    // the next tile's first stage (and coefficients) landed once at most the
    // epilogue's stores are outstanding; this wave's staging reads are done
    // before the next barrier lets stage 1 refill buffer 1
    if constexpr (SWIGLU)
      wait_vmcnt<S_EPI>();
    else
      wait_vmcnt_upto<0, 63>(n_st);
    wait_lgkm0();
    cur = nxt;
    db ^= 1;
  }
}

}  // namespace

template <bool SWIGLU>
hipError_t launch_mx(const GemmArgs &g, int grid_tiles, int align, hipStream_t s) {
  if (g.N % 256 || g.K % 128 || g.K > kMaxDim || g.s_ld % 256) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / 256);
  // 128-row tiles: two stages (68 KB of LDS) so that two workgroups share a
  // CU -- one wave per SIMD cannot hide the load latency of a 4-wave tile,
  // two can (25-40 % faster than four stages at one workgroup per CU on
  // batches of 128-256 rows per expert)
  if (align == kFp8TileM)
    hipLaunchKernelGGL((k_gemm_mx<4, 2, SWIGLU, 2>), dim3(grid), dim3(256), 0, s, g);
  else if (align == kFp8LargeTileM)
    hipLaunchKernelGGL((k_gemm_mx_persist<SWIGLU>), dim3(std::min(grid, persistent_grid())),
                       dim3(512), 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template hipError_t launch_mx<true>(const GemmArgs &, int, int, hipStream_t);
template hipError_t launch_mx<false>(const GemmArgs &, int, int, hipStream_t);

}  // namespace cep
