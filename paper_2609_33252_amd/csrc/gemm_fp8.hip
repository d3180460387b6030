// e4m3 (OCP fp8) grouped expert GEMMs for gfx950 (CDNA4) MFMA.
//
// Expert weights arrive as e4m3 codes with one float32 scale per 128x128
// block; activations are quantised per (row, 128 channels) by the pack step
// and h per (row, 128 columns) in the GEMM1 epilogue (Appendix C, "Grouped
// FFN invocations": the layout transform packs activations with their
// quantisation metadata, and the activation and quantisation run between
// the two expert GEMMs).  The hardware-scaled MFMA takes power-of-two
// (E8M0) scales per 32 elements; these block scales are arbitrary float32,
// so each 128-wide K block runs unscaled and is promoted in float32.
#include "gemm_common.h"

namespace cep {
namespace {

// BM x 256 output tile, K step 128 (one scale block).  NW waves: four
// column groups of 64 x (NW/4) row groups of 128, each wave owning 128 rows x
// 64 columns built from 8x4 v_mfma_scale_f32_16x16x128_f8f6f4 with unit
// hardware scales.  Every instruction covers one whole K block, so its
// result is promoted into the float32 accumulator with the product of the
// row's activation scale and the weight block's scale: two VALU operations
// per output element and K block, which is why each wave holds few column
// scale blocks (GEMM1: the gate and the up block of its 32 h columns; GEMM2:
// one) and few rows per lane.  With 8 waves (two per SIMD) one wave's
// promotion overlaps the other's MFMAs.
//
// Operands stream through a ring of STAGES LDS stages filled by direct
// global->LDS loads issued STAGES-1 steps ahead ((BM + 256) x 128 codes + BM
// row scales per stage).  An LDS row is 128 codes = eight 16-byte chunks;
// chunk c of row r lives at slot c ^ ((r >> 1) & 7).  A lane reads chunks
// g and g + 4 of its row (g = lane / 16): a 16-byte LDS read serves per
// cycle the sixteen lanes of one half-wave whose quad index (lane bits 2-4)
// has one parity, and those lanes then touch sixteen distinct slots of 256
// bytes (reading chunks 2g, 2g + 1 instead measured two-way bank conflicts).
//
// GEMM1 epilogue: h = silu(gate) * up over the tile's 128 h columns, one
// amax per row (lanes, then the four column waves via LDS), scale =
// amax / 448, e4m3 codes of h / scale.
template <int NW, int STAGES, bool SWIGLU>
__global__ __launch_bounds__(64 * NW, 1) void k_gemm_fp8(GemmArgs g) {
  constexpr int BM = 128 * NW / 4, BN = 256, BK = 128, WN = BN / 4;
  constexpr int A_LD = BM * BK / 1024 / NW, B_LD = BN * BK / 1024 / NW;  // loads per wave
  constexpr int PER = A_LD + B_LD;  // per thread per step; wave 0 adds one (row scales)
  static_assert(BM / 4 <= 64, "one load of BM row scales");
  int mt, nt;
  if (!balanced_tile<kGroupM>(*g.n_tiles, g.N / BN, &mt, &nt)) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int K = g.K, nkb = K / BK;
  const uint8_t *blob = blob_of(g.bt, t.expert);
  const char *Ag = (const char *)(g.A + (size_t)t.row0 * K);
  const char *Bg = (const char *)(blob + g.b_off + (size_t)nt * BN * K);
  const char *Asg = (const char *)(g.As + t.row0);  // k-block kb at + kb * s_ld floats
  const float *Bs = (const float *)(blob + g.bs_off);

  __shared__ u32x4 sA[STAGES][BM * 8];
  __shared__ u32x4 sB[STAGES][BN * 8];
  __shared__ float sAs[STAGES][BM];
  __shared__ float red[4][BM];
  __shared__ float sBs[8 * (kMaxDim / BK)];

  // lane l of a load fills slot l of a 1 KB segment (8 rows x 8 chunks)
  const int seg_row = lane >> 3;
#define CEP_F8_OFF(seg)                                                            \
  ((uint32_t)((seg) * 8 + seg_row) * K +                                           \
   (uint32_t)(((lane & 7) ^ ((((seg) * 8 + seg_row) >> 1) & 7)) * 16))
#define CEP_F8_STAGE(kb)                                                           \
  {                                                                                \
    const int buf_ = (kb) % STAGES;                                                \
    _Pragma("unroll") for (int i = 0; i < A_LD; ++i) {                             \
      const int seg = wid * A_LD + i;                                              \
      dma16(Ag + (size_t)(kb) * BK + CEP_F8_OFF(seg),                              \
            __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf_][seg * 64])));      \
    }                                                                              \
    _Pragma("unroll") for (int i = 0; i < B_LD; ++i) {                             \
      const int seg = wid * B_LD + i;                                              \
      dma16(Bg + (size_t)(kb) * BK + CEP_F8_OFF(seg),                              \
            __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf_][seg * 64])));      \
    }                                                                              \
    if (wid == 0 && lane < BM / 4)                                                 \
      dma16(Asg + (size_t)(kb) * g.s_ld * 4 + lane * 16,                           \
            __builtin_amdgcn_readfirstlane(lds_offset(&sAs[buf_][0])));            \
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{};

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nkb) CEP_F8_STAGE(s);

  // The weight block scales of the tile's columns (8 consecutive rows of
  // [N/32][nkb] for GEMM1, 2 of [N/128][nkb] for GEMM2) go to LDS once, so
  // the main loop issues no vector loads besides the ring's.
  {
    const int nbs = (SWIGLU ? BN / kInterleave : BN / 128) * nkb;
    const float *src = Bs + (size_t)nt * nbs;
    for (int i = tid; i < nbs; i += 64 * NW) sBs[i] = src[i];
  }
  __syncthreads();

  const int rsw = ((lane & 15) >> 1) & 7;  // swizzle of every operand row this lane reads
  // this lane's two chunks: K bytes [16g, 16g+16) and [64+16g, 64+16g+16),
  // g = lane / 16, the instruction's own K order (A and B alike); reading the
  // chunk pair (g, g + 4) keeps every 16-lane LDS cycle on distinct banks
  const int c0 = lane >> 4, c1 = c0 + 4;
  // scale rows of this wave's column blocks: GEMM1 blocks j = 0,1 (gate) use
  // row 2*wn, j = 2,3 (up) row 2*wn + 1; GEMM2's 64 columns lie in row wn/2
  const float *sb_row0 = &sBs[(SWIGLU ? 2 * wn : wn / 2) * nkb];
  const float *sb_row1 = &sBs[(SWIGLU ? 2 * wn + 1 : wn / 2) * nkb];
  for (int kb = 0; kb < nkb; ++kb) {
    // this wave's loads of step kb are done when at most the loads of the
    // steps issued after it are outstanding
    const int later = min(nkb - 1, kb + STAGES - 2) - kb;
    if (wid == 0)
      wait_stages<PER + 1, STAGES - 2>(later);
    else
      wait_stages<PER, STAGES - 2>(later);
    // every wave's loads of step kb landed; step kb-1 fully consumed
    __builtin_amdgcn_s_barrier();
    if (kb + STAGES - 1 < nkb) CEP_F8_STAGE(kb + STAGES - 1);
    const int cur = kb % STAGES;
    const float sb0 = sb_row0[kb], sb1 = sb_row1[kb];

    i32x8 b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = wn * WN + j * 16 + (lane & 15);
      const u32x4 lo = sB[cur][row * 8 + (c0 ^ rsw)];
      const u32x4 hi = sB[cur][row * 8 + (c1 ^ rsw)];
      b[j] = __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = wm * 128 + i * 16 + (lane & 15);
      const u32x4 lo = sA[cur][row * 8 + (c0 ^ rsw)];
      const u32x4 hi = sA[cur][row * 8 + (c1 ^ rsw)];
      const i32x8 a =
          __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      f32x4 p[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        p[j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b[j], f32x4{}, 0, 0, 0, 127,
                                                               0, 127);
      const f32x4 sa = *(const f32x4 *)&sAs[cur][wm * 128 + i * 16 + 4 * (lane >> 4)];
      const f32x4 s0 = sa * sb0, s1 = sa * sb1;
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] += p[j] * (j < 2 ? s0 : s1);
    }
  }
#undef CEP_F8_STAGE
#undef CEP_F8_OFF

  // 16x16 accumulator layout: lane l, element r -> column l%16,
  // row 4*(l/16) + r.
  if (SWIGLU) {
    // h column nt*128 + wn*32 + jj*16 + l%16 = silu(gate block jj) * up block jj+2
    float h[8][2][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[i][jj][r] = silu_mul(acc[i][jj][r], acc[i][jj + 2][r]);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float m = fmaxf(fabsf(h[i][0][r]), fabsf(h[i][1][r]));
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) m = fmaxf(m, __shfl_xor(m, sh, 16));
        if ((lane & 15) == 0) red[wn][wm * 128 + i * 16 + 4 * (lane >> 4) + r] = m;
      }
    __syncthreads();
    uint8_t *H = (uint8_t *)g.out;
    const int I = g.N / 2;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rt = wm * 128 + i * 16 + 4 * (lane >> 4) + r;
        if (rt >= t.rows) continue;
        const float amax = fmaxf(fmaxf(red[0][rt], red[1][rt]), fmaxf(red[2][rt], red[3][rt]));
        const float scale = amax > 0.f ? amax / 448.0f : 1.0f;
        const size_t row = (size_t)t.row0 + rt;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int col = nt * 128 + wn * 32 + jj * 16 + (lane & 15);
          const int q = __builtin_amdgcn_cvt_pk_fp8_f32(h[i][jj][r] / scale, 0.f, 0, false);
          H[row * I + col] = (uint8_t)(q & 0xff);
        }
        if (wn == 0 && (lane & 15) == 0) g.out_s[(size_t)nt * g.s_ld + row] = scale;
      }
  } else {
    __bf16 *Y = (__bf16 *)g.out;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rt = wm * 128 + i * 16 + 4 * (lane >> 4) + r;
        if (rt >= t.rows) continue;
        const size_t row = (size_t)t.row0 + rt;
        const float w = g.wrow[row];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          Y[row * g.N + nt * BN + wn * WN + j * 16 + (lane & 15)] = (__bf16)(acc[i][j][r] * w);
      }
  }
}

}  // namespace

template <bool SWIGLU>
hipError_t launch_fp8(const GemmArgs &g, int grid_tiles, int align, hipStream_t s) {
  if (g.N % 256 || g.K % 128 || g.K > kMaxDim || g.s_ld % 4) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / 256);
  if (align == kFp8TileM)
    hipLaunchKernelGGL((k_gemm_fp8<4, 3, SWIGLU>), dim3(grid), dim3(256), 0, s, g);
  else if (align == kFp8LargeTileM)
    hipLaunchKernelGGL((k_gemm_fp8<8, 2, SWIGLU>), dim3(grid), dim3(512), 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template hipError_t launch_fp8<true>(const GemmArgs &, int, int, hipStream_t);
template hipError_t launch_fp8<false>(const GemmArgs &, int, int, hipStream_t);

}  // namespace cep
