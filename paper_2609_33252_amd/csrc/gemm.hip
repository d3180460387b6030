// Grouped expert GEMMs of the streamFFN path for gfx950 (CDNA4) MFMA.
//
// Appendix C, "Grouped FFN invocations": within an invocation the two expert
// GEMMs and the intervening activation and quantisation run in stream order.
// GEMM1 computes the gate and up projections of every grouped row against its
// expert's weights and applies SwiGLU in the epilogue; GEMM2 computes the
// down projection and scales each row by its routing coefficient (the one
// place the coefficient is applied).
//
// Both are "NT" products: A = grouped rows [M][K], B = packed weights [N][K],
// K contiguous in both, so every MFMA operand is a 16-byte (bf16) or 32-byte
// (fp8) contiguous run of K.  Work is a device tile list (expert, first row,
// valid rows) built by the routing scan: no host round trip for the counts.
// The grid is an upper bound on tiles x N tiles; surplus workgroups exit.
//
// Workgroup ids are dispatched round-robin over the 8 XCDs; they are remapped
// so that each XCD walks a contiguous range of (N tile, M tile) pairs, M
// fastest, keeping one weight tile hot in that XCD's L2 while its M tiles run.
#include "common.h"

#include <hip/hip_bf16.h>

namespace cep {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct GemmArgs {
  const uint8_t *A;       // grouped rows [mpad][K] (bf16 or e4m3)
  const float *As;        // fp8: [mpad][K/128] row scales
  const Tile *tiles;      // tile list
  const int32_t *n_tiles; // live tiles in the list
  int max_tiles;          // grid extent in M tiles
  int K, N;               // contraction length, packed output columns
  size_t b_off, bs_off;   // offsets of B and its scales in each blob
  BlobTable bt;
  void *out;              // H [mpad][N/2] (GEMM1) or Y [mpad][N] f32 (GEMM2)
  float *out_s;           // fp8 GEMM1: h scales [mpad][N/256]
  const float *wrow;      // GEMM2: routing coefficient per grouped row
};

__device__ inline int xcd_remap(int bid, int G) {
  const int x = bid & 7, j = bid >> 3;
  const int q = G >> 3, r = G & 7;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// ---------------------------------------------------------------- bf16
// 128x128 output tile, K step 64, 4 waves as 2x2, each wave 64x64 built from
// 2x2 v_mfma_f32_32x32x16_bf16.  LDS rows are 64 bf16 (eight 16-byte chunks),
// chunk c of row r stored at c ^ (r & 7) so both the global->LDS stores and
// the MFMA operand reads (32 rows, one chunk each) are conflict-free.
template <bool SWIGLU>
__global__ __launch_bounds__(256) void k_gemm_bf16(GemmArgs g) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = L % g.max_tiles, nt = L / g.max_tiles;
  if (mt >= *g.n_tiles) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int K = g.K, kv = K / 8;
  const u32x4 *Ag = (const u32x4 *)(g.A + (size_t)t.row0 * K * 2);
  const u32x4 *Bg = (const u32x4 *)(blob_of(g.bt, t.expert) + g.b_off + (size_t)nt * 128 * K * 2);

  __shared__ u32x4 sA[128 * 8];
  __shared__ u32x4 sB[128 * 8];
  u32x4 ra[4], rb[4];
#define CEP_BF16_GLOAD(k0)                                   \
  _Pragma("unroll") for (int i = 0; i < 4; ++i) {            \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;   \
    ra[i] = Ag[(size_t)row * kv + ((k0) >> 3) + ch];         \
    rb[i] = Bg[(size_t)row * kv + ((k0) >> 3) + ch];         \
  }
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  CEP_BF16_GLOAD(0);
  for (int k0 = 0; k0 < K; k0 += 64) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = tid + 256 * i, row = v >> 3, ch = v & 7;
      sA[row * 8 + (ch ^ (row & 7))] = ra[i];
      sB[row * 8 + (ch ^ (row & 7))] = rb[i];
    }
    __syncthreads();
    if (k0 + 64 < K) {
      CEP_BF16_GLOAD(k0 + 64);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 a[2], b[2];
      const int ch = kk * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wm * 64 + i * 32 + (lane & 31);
        a[i] = __builtin_bit_cast(bf16x8, sA[row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wn * 64 + j * 32 + (lane & 31);
        b[j] = __builtin_bit_cast(bf16x8, sB[row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  // 32x32 accumulator layout: lane l, element r -> column l%32,
  // row 8*(r/4) + 4*(l/32) + r%4.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rt = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (rt >= t.rows) continue;
      const size_t row = (size_t)t.row0 + rt;
      if (SWIGLU) {
        // wave columns: [gate 32 | up 32] of h columns nt*64 + wn*32 + [0, 32)
        const float h = silu_mul(acc[i][0][r], acc[i][1][r]);
        __bf16 *H = (__bf16 *)g.out;
        H[row * (g.N / 2) + nt * 64 + wn * 32 + (lane & 31)] = (__bf16)h;
      } else {
        const float w = g.wrow[row];
        float *Y = (float *)g.out;
#pragma unroll
        for (int j = 0; j < 2; ++j)
          Y[row * g.N + nt * 128 + wn * 64 + j * 32 + (lane & 31)] = acc[i][j][r] * w;
      }
    }
  }
}

// ----------------------------------------------------------------- fp8
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
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = L % g.max_tiles, nt = L / g.max_tiles;
  if (mt >= *g.n_tiles) return;
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

GemmArgs base_args(const Scratch &sc, int which, int list_cap, int grid_tiles,
                   const BlobTable &bt) {
  GemmArgs g{};
  g.tiles = sc.tiles + (size_t)which * list_cap;
  g.n_tiles = sc.n_tiles + which;
  g.max_tiles = grid_tiles;
  g.bt = bt;
  return g;
}

}  // namespace

hipError_t launch_gemm1(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        const BlobTable &bt, const BlobLayout &L, bool fp8, int d, int I,
                        hipStream_t s) {
  if (grid_tiles <= 0) return hipSuccess;
  GemmArgs g = base_args(sc, which, list_cap, grid_tiles, bt);
  g.A = (const uint8_t *)sc.xg;
  g.As = sc.xs;
  g.K = d;
  g.N = 2 * I;
  g.b_off = L.w1_off;
  g.bs_off = L.s1_off;
  g.out = sc.h;
  g.out_s = sc.hs;
  if (fp8) {
    const int grid = grid_tiles * (g.N / 256);
    hipLaunchKernelGGL(k_gemm_fp8<true>, dim3(grid), dim3(256), 0, s, g);
  } else {
    const int grid = grid_tiles * (g.N / 128);
    hipLaunchKernelGGL(k_gemm_bf16<true>, dim3(grid), dim3(256), 0, s, g);
  }
  return hipGetLastError();
}

hipError_t launch_gemm2(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        const BlobTable &bt, const BlobLayout &L, bool fp8, int d, int I,
                        hipStream_t s) {
  if (grid_tiles <= 0) return hipSuccess;
  GemmArgs g = base_args(sc, which, list_cap, grid_tiles, bt);
  g.A = (const uint8_t *)sc.h;
  g.As = sc.hs;
  g.K = I;
  g.N = d;
  g.b_off = L.w2_off;
  g.bs_off = L.s2_off;
  g.out = sc.y;
  g.wrow = sc.wrow;
  if (fp8) {
    const int grid = grid_tiles * (g.N / 256);
    hipLaunchKernelGGL(k_gemm_fp8<false>, dim3(grid), dim3(256), 0, s, g);
  } else {
    const int grid = grid_tiles * (g.N / 128);
    hipLaunchKernelGGL(k_gemm_bf16<false>, dim3(grid), dim3(256), 0, s, g);
  }
  return hipGetLastError();
}

}  // namespace cep
