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

namespace cep {
namespace {

// One e4m3 x e2m1 block-scaled MFMA; OB and oa pick the byte of the B and A
// scale words (the instruction takes them as immediates: oa is a constant
// after the caller's loop is unrolled, and the switch folds away).
template <int OB>
__device__ inline f32x4 mx_mfma(const i32x8 &a, const i32x8 &b, const f32x4 &c, int oa, int sa,
                                int sb) {
  switch (oa) {
    case 0: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 0, sa, OB, sb);
    case 1: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 1, sa, OB, sb);
    case 2: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 2, sa, OB, sb);
    default: return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 3, sa, OB, sb);
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
// GEMM1 epilogue: h = silu(gate) * up; each wave's 32 h columns of a row
// are one MX block, so the block amax needs only a 16-lane reduction; the
// E8M0 scale is 2^(floor(log2 amax) - 8), the codes e4m3(h / scale)
// saturated at 448.
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
      acc[i][0] = mx_mfma<0>(a, b[0], acc[i][0], i & 3, sai, (int)sb);
      acc[i][1] = mx_mfma<1>(a, b[1], acc[i][1], i & 3, sai, (int)sb);
      acc[i][2] = mx_mfma<2>(a, b[2], acc[i][2], i & 3, sai, (int)sb);
      acc[i][3] = mx_mfma<3>(a, b[3], acc[i][3], i & 3, sai, (int)sb);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#undef CEP_MX_STAGE

  // 16x16 accumulator layout: lane l, element r -> column l%16,
  // row 4*(l/16) + r.
  if (SWIGLU) {
    uint8_t *H = (uint8_t *)g.out;
    uint8_t *Hs = (uint8_t *)g.out_s;
    const int I = g.N / 2, hblk = nt * 4 + wn;  // this wave's MX block of h columns
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // h column nt*128 + wn*32 + jj*16 + l%16 = silu(gate block jj) * up block jj+2
        const float h0 = silu_mul(acc[i][0][r], acc[i][2][r]);
        const float h1 = silu_mul(acc[i][1][r], acc[i][3][r]);
        float m = fmaxf(fabsf(h0), fabsf(h1));
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) m = fmaxf(m, __shfl_xor(m, sh, 16));
        const int rt = wm * 128 + i * 16 + 4 * grp + r;
        if (rt >= t.rows) continue;
        const int code = max((int)((__float_as_uint(m) >> 23) & 0xff) - 8, 0);
        const int e = 127 - code;  // h / 2^(code - 127), exact
        const float q0 = fminf(fmaxf(ldexpf(h0, e), -448.0f), 448.0f);
        const float q1 = fminf(fmaxf(ldexpf(h1, e), -448.0f), 448.0f);
        const int q = __builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false);
        const size_t row = (size_t)t.row0 + rt;
        uint8_t *hrow = H + row * I + nt * 128 + wn * 32 + r16;
        hrow[0] = (uint8_t)(q & 0xff);
        hrow[16] = (uint8_t)((q >> 8) & 0xff);
        if (r16 == 0) Hs[mx_row_scale_offset((int)row, hblk, g.s_ld)] = (uint8_t)code;
      }
  } else {
    __bf16 *Y = (__bf16 *)g.out;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rt = wm * 128 + i * 16 + 4 * grp + r;
        if (rt >= t.rows) continue;
        const size_t row = (size_t)t.row0 + rt;
        const float w = g.wrow[row];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          Y[row * g.N + nt * BN + wn * 64 + j * 16 + r16] = (__bf16)(acc[i][j][r] * w);
      }
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
    hipLaunchKernelGGL((k_gemm_mx<8, 2, SWIGLU>), dim3(grid), dim3(512), 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template hipError_t launch_mx<true>(const GemmArgs &, int, int, hipStream_t);
template hipError_t launch_mx<false>(const GemmArgs &, int, int, hipStream_t);

}  // namespace cep
