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

// 128x256 output tile, K step 128 (one scale block), 4 waves as 2x2, each
// wave 64x128 built from 4x8 v_mfma_scale_f32_16x16x128_f8f6f4 with unit
// hardware scales.  Each instruction covers one whole 128-wide K block, so
// its result is promoted into the float32 accumulator with the product of
// the row's activation scale and the weight block's scale.
//
// GEMM1 epilogue: h = silu(gate) * up over the tile's 128 h columns, one
// amax per row (lanes, then the two column waves via LDS), scale =
// amax / 448, e4m3 codes of h / scale.
template <bool SWIGLU>
__global__ __launch_bounds__(256) void k_gemm_fp8(GemmArgs g) {
  int mt, nt;
  if (!balanced_tile<kGroupM>(*g.n_tiles, g.N / 256, &mt, &nt)) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int K = g.K, kv = K / 16, nkb = K / 128;
  const uint8_t *blob = blob_of(g.bt, t.expert);
  const u32x4 *Ag = (const u32x4 *)(g.A + (size_t)t.row0 * K);
  const u32x4 *Bg = (const u32x4 *)(blob + g.b_off + (size_t)nt * 256 * K);
  const float *Asg = g.As + (size_t)t.row0 * nkb;
  const float *Bs = (const float *)(blob + g.bs_off);

  __shared__ u32x4 sA[128 * 8];
  __shared__ u32x4 sB[256 * 8];
  __shared__ float sAs[128];
  __shared__ float red[2][128];
  u32x4 ra[4], rb[8];
  float ras = 0.f;
#define CEP_FP8_GLOAD(kb)                                    \
  _Pragma("unroll") for (int i = 0; i < 4; ++i) {            \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;   \
    ra[i] = Ag[(size_t)row * kv + (kb) * 8 + ch];            \
  }                                                          \
  _Pragma("unroll") for (int i = 0; i < 8; ++i) {            \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;   \
    rb[i] = Bg[(size_t)row * kv + (kb) * 8 + ch];            \
  }                                                          \
  if (tid < 128) ras = Asg[(size_t)tid * nkb + (kb)];
  f32x4 acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{};

  CEP_FP8_GLOAD(0);
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = tid + 256 * i, row = v >> 3, ch = v & 7;
      sA[row * 8 + (ch ^ (row & 7))] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int v = tid + 256 * i, row = v >> 3, ch = v & 7;
      sB[row * 8 + (ch ^ (row & 7))] = rb[i];
    }
    if (tid < 128) sAs[tid] = ras;
    __syncthreads();
    if (kb + 1 < nkb) {
      CEP_FP8_GLOAD(kb + 1);
    }

    // weight block scales of this wave's columns at k-block kb
    float sb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = nt * 256 + wn * 128 + j * 16;
      sb[j] = SWIGLU ? Bs[(size_t)(col / kInterleave) * nkb + kb]
                     : Bs[(size_t)(col / 128) * nkb + kb];
    }
    i32x8 b[8];
    const int c0 = (lane >> 4) * 2;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = wn * 128 + j * 16 + (lane & 15);
      const u32x4 lo = sB[row * 8 + (c0 ^ (row & 7))];
      const u32x4 hi = sB[row * 8 + ((c0 + 1) ^ (row & 7))];
      b[j] = __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = wm * 64 + i * 16 + (lane & 15);
      const u32x4 lo = sA[row * 8 + (c0 ^ (row & 7))];
      const u32x4 hi = sA[row * 8 + ((c0 + 1) ^ (row & 7))];
      const i32x8 a =
          __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      const f32x4 sa = *(const f32x4 *)&sAs[wm * 64 + i * 16 + 4 * (lane >> 4)];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const f32x4 p = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
            a, b[j], f32x4{}, 0, 0, 0, 127, 0, 127);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] += p[r] * (sa[r] * sb[j]);
      }
    }
  }

  // 16x16 accumulator layout: lane l, element r -> column l%16,
  // row 4*(l/16) + r.
  if (SWIGLU) {
    // h for jj in 0..3: gate block j = (jj/2)*4 + jj%2, up block j + 2;
    // h column nt*128 + wn*64 + (jj/2)*32 + (jj%2)*16 + l%16
    float h[4][4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int j = (jj >> 1) * 4 + (jj & 1);
#pragma unroll
        for (int r = 0; r < 4; ++r) h[i][jj][r] = silu_mul(acc[i][j][r], acc[i][j + 2][r]);
      }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float m = 0.f;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) m = fmaxf(m, fabsf(h[i][jj][r]));
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) m = fmaxf(m, __shfl_xor(m, sh, 16));
        if ((lane & 15) == 0) red[wn][wm * 64 + i * 16 + 4 * (lane >> 4) + r] = m;
      }
    __syncthreads();
    uint8_t *H = (uint8_t *)g.out;
    const int I = g.N / 2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rt = wm * 64 + i * 16 + 4 * (lane >> 4) + r;
        if (rt >= t.rows) continue;
        const float amax = fmaxf(red[0][rt], red[1][rt]);
        const float scale = amax > 0.f ? amax / 448.0f : 1.0f;
        const size_t row = (size_t)t.row0 + rt;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int col = nt * 128 + wn * 64 + (jj >> 1) * 32 + (jj & 1) * 16 + (lane & 15);
          const int q = __builtin_amdgcn_cvt_pk_fp8_f32(h[i][jj][r] / scale, 0.f, 0, false);
          H[row * I + col] = (uint8_t)(q & 0xff);
        }
        if (wn == 0 && (lane & 15) == 0) g.out_s[row * (I / 128) + nt] = scale;
      }
  } else {
    float *Y = (float *)g.out;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rt = wm * 64 + i * 16 + 4 * (lane >> 4) + r;
        if (rt >= t.rows) continue;
        const size_t row = (size_t)t.row0 + rt;
        const float w = g.wrow[row];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          Y[row * g.N + nt * 256 + wn * 128 + j * 16 + (lane & 15)] = acc[i][j][r] * w;
      }
  }
}


}  // namespace

template <bool SWIGLU>
hipError_t launch_fp8(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  if (g.N % 256 || g.K % 128) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / 256);
  hipLaunchKernelGGL(k_gemm_fp8<SWIGLU>, dim3(grid), dim3(256), 0, s, g);
  return hipGetLastError();
}

template hipError_t launch_fp8<true>(const GemmArgs &, int, hipStream_t);
template hipError_t launch_fp8<false>(const GemmArgs &, int, hipStream_t);

}  // namespace cep
