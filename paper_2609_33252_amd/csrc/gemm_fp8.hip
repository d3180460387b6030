// e4m3 (OCP fp8) grouped expert GEMMs for gfx950 (CDNA4) block-scaled MFMA.
//
// Expert weights arrive as e4m3 codes with one float32 scale per 128x128
// block.  Activations are quantised to MXFP8 (e4m3 codes, one E8M0
// power-of-two scale per 32 channels) by the pack step and h to MXFP8 in the
// GEMM1 epilogue (Appendix C, "Grouped FFN invocations": the layout
// transform packs activations with their quantisation metadata, and the
// activation and quantisation run between the two expert GEMMs).
// v_mfma_scale_f32_16x16x128_f8f6f4 applies the activation scales itself
// (E8M0 operands); the weight block scales are arbitrary float32, so each
// 128-wide K block -- exactly one instruction -- is promoted into the float32
// accumulator with one fused multiply-add by its block's scale, a value
// shared by every element of the wave's 16-column fragment.  With float32
// activation scales the promotion would need the product of a per-row and a
// per-column scale for every element: a multiply on top of each FMA and a
// row-scale read per row fragment.
//
// Operand layout of the instruction (lane l: row or column l%16, group
// g = l/16): an e4m3 operand lane holds K [16g, 16g+16) in bytes 0-15 and
// K [64+16g, 64+16g+16) in bytes 16-31; an operand's scale byte of lane l
// applies to K block g of its row or column.
#include "gemm_common.h"

#include <algorithm>

namespace cep {
namespace {

// One e4m3 x e4m3 MFMA of a K block: the weight fragment w is the
// instruction's first operand (unit scales), the activation fragment x its
// second, with E8M0 scales (byte ox of the word sx).  Output lane l then
// holds activation row l%16 and the four consecutive weight columns
// 4*(l/16) .. 4*(l/16)+3, so an epilogue stores 4 consecutive outputs of a
// row per lane.  ox is a constant after the caller's loop is unrolled, and
// the switch folds away.
__device__ inline f32x4 f8_mfma(const i32x8 &w, const i32x8 &x, int ox, int sx) {
  switch (ox) {
    case 0: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, f32x4{}, 0, 0, 0, 127, 0, sx);
    case 1: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, f32x4{}, 0, 0, 0, 127, 1, sx);
    case 2: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, f32x4{}, 0, 0, 0, 127, 2, sx);
    default: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(w, x, f32x4{}, 0, 0, 0, 127, 3, sx);
  }
}

// BM x 256 output tile, K step 128 (one weight scale block).  NW waves: four
// column groups of 64 x (NW/4) row groups of 128, each wave owning 128 rows x
// 64 columns = 8 x 4 16x16 fragments.  With 8 waves (two per SIMD) one wave's
// promotion overlaps the other's MFMAs.
//
// Operands stream through a ring of STAGES LDS stages filled by direct
// global->LDS loads issued STAGES-1 steps ahead ((BM + 256) x 128 codes plus
// the BM x 4 row scales per stage).  The row-scale layout
// (mx_row_scale_offset) gives each lane its eight row fragments' scales of
// its K block as one 8-byte word.  The weight block scales of the tile's
// columns go to LDS once per tile.  An LDS row is 128 codes = eight 16-byte
// chunks; chunk c of row r lives at slot c ^ ((r >> 1) & 7).  A lane reads
// chunks g and g + 4 of its row (g = lane / 16): a 16-byte LDS read serves
// per cycle the sixteen lanes of one half-wave whose quad index (lane bits
// 2-4) has one parity, and those lanes then touch sixteen distinct slots of
// 256 bytes.
//
// PERSIST (8 waves, two stages): one workgroup per CU takes work items j,
// j + grid/8, ... of its XCD's share.  After a tile's K loop it issues the
// next tile's first stage into buffer 0 and loads the next tile's block
// scales into registers, then runs the epilogue through buffer 1 (staged
// stores of every row, so each wave issues a fixed number S of stores), so
// that the next tile's first loads and its memory latency overlap the
// epilogue; it then waits until at most those S stores are outstanding (the
// loads issued before them have landed) and moves on.
//
// Epilogues: store_h_mx_staged (GEMM1) and store_y_bf16_staged (GEMM2).
struct F8Tile {
  Tile t;
  int nt;
  const char *Ag, *Bg, *Asg;
  const float *bs;
};

template <int NW, int STAGES, bool SWIGLU, bool PERSIST, int OCC = 1>
__global__ __launch_bounds__(64 * NW, OCC) void k_gemm_fp8(GemmArgs g) {
  constexpr int BM = 128 * NW / 4, BN = 256, BK = 128, WN = BN / 4;
  constexpr int A_LD = BM * BK / 1024 / NW, B_LD = BN * BK / 1024 / NW;  // loads per wave
  constexpr int PER = A_LD + B_LD;  // per thread per step; wave 0 adds one (row scales)
  static_assert(BM * 4 <= 1024, "one load of the row scales");
  static_assert(PERSIST == (NW == 8) && (!PERSIST || STAGES == 2),
                "the 8-wave tiles are the persistent two-stage ones");
  // uniform over the workgroup: kept in scalar registers
  const int n_live = __builtin_amdgcn_readfirstlane(*g.n_tiles), ntn = g.N / BN;
  int mt, nt;
  if (!(PERSIST ? work_item_xg<kGroupXcd>(0, n_live, ntn, &mt, &nt)
                : work_item<kGroupM, false>(0, n_live, ntn, &mt, &nt)))
    return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int K = g.K, nkb = K / BK;
  const size_t as_step = (size_t)(g.s_ld >> 7) * 512;  // row scales: 512 bytes per 128-row group
  // weight block scales of a tile's columns: 8 consecutive rows of
  // [N/32][nkb] for GEMM1, 2 of [N/128][nkb] for GEMM2
  const int nbs = (SWIGLU ? BN / kInterleave : BN / 128) * nkb;

  __shared__ u32x4 sA[STAGES][BM * 8];
  __shared__ u32x4 sB[STAGES][BN * 8];
  __shared__ u32x4 sAs[STAGES][BM / 4];
  __shared__ float sBs[8 * (kMaxDim / BK)];
  // PERSIST GEMM2: the tile's routing coefficients, brought with its first
  // stage (they are only needed after the K loop)
  __shared__ float sW[PERSIST && !SWIGLU ? BM : 1];
  // GEMM2: the tile rows' output rows for direct writes (GemmArgs::ydst);
  // PERSIST: two buffers, the next tile's loads beside the current epilogue
  __shared__ int sD[SWIGLU ? 1 : (PERSIST ? 2 : 1)][SWIGLU ? 1 : BM];

  auto tile_at = [&](int mt_, int nt_) {
    F8Tile f;
    mt_ = __builtin_amdgcn_readfirstlane(mt_);
    nt_ = __builtin_amdgcn_readfirstlane(nt_);
    f.t = g.tiles[mt_];
    f.nt = nt_;
    const uint8_t *blob = blob_of(g.bt, f.t.expert);
    f.Ag = (const char *)(g.A + (size_t)f.t.row0 * K);
    f.Bg = (const char *)(blob + g.b_off + (size_t)nt_ * BN * K);
    f.Asg = (const char *)g.As + (size_t)(f.t.row0 >> 7) * 512;
    f.bs = (const float *)(blob + g.bs_off) + (size_t)nt_ * nbs;
    return f;
  };
  // lane l of a load fills slot l of a 1 KB segment (8 rows x 8 chunks)
  const int seg_row = lane >> 3;
  auto lane_off = [&](int seg) {
    const int r = seg * 8 + seg_row;
    return (uint32_t)r * K + (uint32_t)(((lane & 7) ^ ((r >> 1) & 7)) * 16);
  };
  auto stage = [&](const F8Tile &f, int kb, int buf) {
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int seg = wid * A_LD + i;
      dma16_s(f.Ag + (size_t)kb * BK, lane_off(seg),
              __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf][seg * 64])));
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int seg = wid * B_LD + i;
      dma16_s(f.Bg + (size_t)kb * BK, lane_off(seg),
              __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf][seg * 64])));
    }
    if (wid == 0 && lane < BM / 4)
      dma16(f.Asg + (size_t)kb * as_step + lane * 16,
            __builtin_amdgcn_readfirstlane(lds_offset(&sAs[buf][0])));
  };
  // the coefficients and output rows of the tile's BM rows: one 1 KB load
  // each, by waves 1 and 2 (the rows of a tile lie inside the layout's
  // padded rows)
  auto stage_coef = [&](const F8Tile &f, int db) {
    if constexpr (PERSIST && !SWIGLU) {
      static_assert(BM * 4 == 1024, "one 1 KB load");
      if (wid == 1)
        dma16_s(g.wrow + f.t.row0, lane * 16, __builtin_amdgcn_readfirstlane(lds_offset(&sW[0])));
      if (g.ydst) {
        if (wid == 2)
          dma16_s(g.ydst + f.t.row0, lane * 16,
                  __builtin_amdgcn_readfirstlane(lds_offset(&sD[db][0])));
      } else if (tid < BM) {
        sD[db][tid] = -1;
      }
    }
  };

  F8Tile cur = tile_at(mt, nt);
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nkb) stage(cur, s, s % STAGES);
  int db = 0;  // PERSIST GEMM2: sD buffer of the current tile
  stage_coef(cur, db);
  for (int i = tid; i < nbs; i += 64 * NW) sBs[i] = cur.bs[i];
  // a PERSIST tile's K loop starts without a wait: its first stage (and the
  // coefficients) must have landed for every wave here.  The direct loads
  // are invisible to the compiler, so __syncthreads() alone would not wait
  // for them in the waves that load no block scale.
  if constexpr (PERSIST) wait_vmcnt<0>();
  __syncthreads();

  const int r16 = lane & 15, grp = lane >> 4;
  const int rsw = (r16 >> 1) & 7;  // swizzle of every operand row this lane reads
  // scale rows of this wave's column blocks: GEMM1 fragments j = 0,1 (gate)
  // use row 2*wn, j = 2,3 (up) row 2*wn + 1; GEMM2's 64 columns lie in row
  // wn/2
  const float *sb_row0 = &sBs[(SWIGLU ? 2 * wn : wn / 2) * nkb];
  const float *sb_row1 = &sBs[(SWIGLU ? 2 * wn + 1 : wn / 2) * nkb];
  auto read_op = [&](const u32x4 *s, int row) {
    const u32x4 lo = s[row * 8 + (grp ^ rsw)];
    const u32x4 hi = s[row * 8 + ((grp + 4) ^ rsw)];
    return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // stores each wave issues at least in a PERSIST epilogue (FULL staging,
  // 512 threads): GEMM1 256 x 128 code bytes in 16-byte pieces (4) and one
  // scale word; GEMM2 two passes of 128 x 512 bytes (8 each; the staging
  // counts its direct float32 rows' extra stores)
  constexpr int S_EPI = SWIGLU ? 4 : 16;
  // block scales per thread (at most 8 or 2 rows of kMaxDim/BK per tile)
  constexpr int NBSV = PERSIST ? (SWIGLU ? 8 : 2) * (kMaxDim / BK) / (64 * NW) : 1;

  for (int it = 0;; ++it) {
    float wr[8];
    int ydv = -1;  // non-PERSIST GEMM2: row tid's output row, to sD after the K loop
    if (!SWIGLU && !PERSIST) {
      load_row_coef(g, cur.t, wm, lane, wr);
      if (g.ydst && tid < BM) ydv = g.ydst[(size_t)cur.t.row0 + tid];
    }
    f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{};

    for (int kb = 0; kb < nkb; ++kb) {
      // this wave's loads of step kb are done when at most the loads of the
      // steps issued after it are outstanding (a PERSIST tile's first stage
      // was waited for before its block scales went to LDS)
      const int later = min(nkb - 1, kb + STAGES - 2) - kb;
      if (!PERSIST || kb > 0) {
        if (wid == 0)
          wait_stages<PER + 1, STAGES - 2>(later);
        else
          wait_stages<PER, STAGES - 2>(later);
      }
      // every wave's loads of step kb landed; step kb-1 fully consumed
      __builtin_amdgcn_s_barrier();
      if (kb + STAGES - 1 < nkb) stage(cur, kb + STAGES - 1, (kb + STAGES - 1) % STAGES);
      const int buf = kb % STAGES;
      const float sb0 = sb_row0[kb], sb1 = sb_row1[kb];
      const uint2 sa = ((const uint2 *)&sAs[buf][0])[wm * 64 + grp * 16 + r16];

      i32x8 b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = read_op(sB[buf], wn * WN + j * 16 + r16);
      // A fragments one row group ahead: the reads of group i+1 are issued
      // before the MFMAs of group i, so LDS latency hides behind them
      i32x8 a_next = read_op(sA[buf], wm * 128 + r16);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const i32x8 a = a_next;
        if (i + 1 < 8) a_next = read_op(sA[buf], wm * 128 + (i + 1) * 16 + r16);
        const int sai = (int)(i < 4 ? sa.x : sa.y);
        f32x4 p[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = f8_mfma(b[j], a, i & 3, sai);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += p[j] * (j < 2 ? sb0 : sb1);
      }
    }

    if constexpr (!PERSIST) {
      // staging: BM x 128 code bytes; y rows of 512 bytes, 64 per 32 KB piece
      static_assert(sizeof(sA) >= BM * 128, "the h tile fits the A ring");
      static_assert(sizeof(sB[0]) >= 64 * 512, "y rows fit the ring");
      if constexpr (!SWIGLU) {
        // read after the epilogue's first barrier
        if (tid < BM) sD[0][tid] = ydv;
      }
      if constexpr (SWIGLU) {
        store_h_mx_staged<NW>(acc, g, cur.t, cur.nt, wm, wn, lane, tid, &sA[0][0]);
      } else {
        uint32_t yb[8][4][2];
        pack_y_bf16(acc, wr, yb);
        store_y_bf16_staged<NW>(yb, g, cur.t, cur.nt, wm, wn, lane, tid, &sB[0][0], &sB[1][0],
                                &sD[0][0]);
      }
      return;
    } else {
      // GEMM2: the outputs are scaled by the coefficients (in LDS since the
      // tile's first step) and packed to bf16 before the next tile's
      // coefficients overwrite them
      uint32_t yb[SWIGLU ? 1 : 8][4][2];
      if constexpr (!SWIGLU) {
#pragma unroll
        for (int i = 0; i < 8; ++i) wr[i] = sW[wm * 128 + i * 16 + r16];
        pack_y_bf16(acc, wr, yb);
      }
      int mt2, nt2;
      const bool more = work_item_xg<kGroupXcd>(it + 1, n_live, ntn, &mt2, &nt2);
      F8Tile nxt;
      float sbv[NBSV];
      if (more) {
        // every wave's operand reads of the last step completed (it may
        // have used buffer 0): the next tile's first stage may fill it
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
        nxt = tile_at(mt2, nt2);
        stage(nxt, 0, 0);
        stage_coef(nxt, db ^ 1);
#pragma unroll
        for (int v = 0; v < NBSV; ++v) {
          const int i = tid + v * 64 * NW;
          sbv[v] = i < nbs ? nxt.bs[i] : 0.0f;
        }
      }
      // epilogue through buffer 1 (sA[1], sB[1]: 32 KB each)
      static_assert(sizeof(sA[1]) >= BM * 128 && sizeof(sA[1]) >= 64 * 512 &&
                        sizeof(sB[1]) >= 64 * 512, "staging fits buffer 1");
      int n_st = S_EPI;
      if constexpr (SWIGLU)
        store_h_mx_staged<NW, true>(acc, g, cur.t, cur.nt, wm, wn, lane, tid, &sA[1][0]);
      else
        n_st = store_y_bf16_staged<NW, true>(yb, g, cur.t, cur.nt, wm, wn, lane, tid, &sA[1][0],
                                             &sB[1][0], &sD[db][0]);
      if (!more) return;
      // the next tile's first stage and block scales landed once at most the
      // epilogue's stores are outstanding
      if constexpr (SWIGLU)
        wait_vmcnt<S_EPI>();
      else
        wait_vmcnt_upto<0, 63>(n_st);
#pragma unroll
      for (int v = 0; v < NBSV; ++v) {
        const int i = tid + v * 64 * NW;
        if (i < nbs) sBs[i] = sbv[v];
      }
      wait_lgkm0();  // the block scales are in LDS before the K loop's barrier
      cur = nxt;
      db ^= 1;
    }
  }
}

}  // namespace

template <bool SWIGLU>
hipError_t launch_fp8(const GemmArgs &g, int grid_tiles, int align, hipStream_t s) {
  if (g.N % 256 || g.K % 128 || g.K > kMaxDim || g.s_ld % 256) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / 256);
  if (align == kFp8TileM)
    hipLaunchKernelGGL((k_gemm_fp8<4, 3, SWIGLU, false>), dim3(grid), dim3(256), 0, s, g);
  else if (align == kFp8LargeTileM)
    hipLaunchKernelGGL((k_gemm_fp8<8, 2, SWIGLU, true>), dim3(std::min(grid, persistent_grid())),
                       dim3(512), 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template hipError_t launch_fp8<true>(const GemmArgs &, int, int, hipStream_t);
template hipError_t launch_fp8<false>(const GemmArgs &, int, int, hipStream_t);

}  // namespace cep
