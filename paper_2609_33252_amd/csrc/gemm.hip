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

// Grouped tile order: GM consecutive M tiles x all N tiles form a group, M
// fastest inside it, so the blocks an XCD runs together share GM row panels
// of A and the weight panels of their N tiles in that XCD's L2.
template <int GM>
__device__ inline void tile_of(int L, int n_tiles_n, int *mt, int *nt) {
  const int grp = L / (GM * n_tiles_n), idx = L % (GM * n_tiles_n);
  *mt = grp * GM + idx % GM;
  *nt = idx / GM;
}

// Work item of this workgroup, balanced over the XCDs.  The grid covers the
// host's upper bound on M tiles; the live count is on the device.  The live
// work W (whole groups) is cut into 8 contiguous shares, one per XCD
// (workgroup ids are dispatched round-robin over the XCDs), so the surplus
// workgroups of the bound never leave an XCD idle while another holds the
// tail.  Returns false for a surplus workgroup.
template <int GM>
__device__ inline bool balanced_tile(int n_live, int n_tiles_n, int *mt, int *nt) {
  const int W = (n_live + GM - 1) / GM * GM * n_tiles_n;
  const int C = (W + 7) / 8;
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int L = x * C + j;
  if (j >= C || L >= W) return false;
  tile_of<GM>(L, n_tiles_n, mt, nt);
  return *mt < n_live;
}

// Grid for balanced_tile: at least the bound's work, a multiple of 8.
inline int balanced_grid(int grid_tiles, int gm, int n_tiles_n) {
  return ((grid_tiles + gm - 1) / gm * gm * n_tiles_n + 7) / 8 * 8;
}
constexpr int kGroupM = 8;

typedef __attribute__((address_space(3))) void lds_void;

// One direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// LDS byte offset lds_seg + 16*l.  Issued as inline assembly so that the
// compiler does not order later LDS reads behind it; the caller synchronises
// with wait_vmcnt and a barrier.  m0 holds the LDS base; it is reserved to
// the compiler, so its value is saved and restored around the load (one wait
// state after writing m0 before the load reads it).
__device__ inline void dma16(const void *gptr, uint32_t lds_seg) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gptr), "s"(lds_seg)
      : "memory");
}

__device__ inline uint32_t lds_offset(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// s_waitcnt immediate that waits until at most N vector-memory operations of
// this wave are outstanding (gfx9 encoding: vmcnt in bits [3:0] and [15:14];
// expcnt 7 and lgkmcnt 15 mean "do not wait" on those counters).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// ------------------------------------------------------- bf16, LDS DMA
// BM x BN output tile (256 x 256), 4 waves as 2x2, each wave (BM/2) x (BN/2)
// built from v_mfma_f32_32x32x16_bf16 fragments.  K advances in steps of 32
// through a ring of STAGES LDS buffers filled by direct global->LDS loads
// (global_load_lds_dwordx4, no staging registers) issued STAGES-1 steps
// ahead, one barrier per step.  An LDS row is 32 bf16 = four 16-byte chunks;
// chunk c of row r lives at slot c ^ ((r >> 2) & 3): sixteen consecutive
// rows read at one chunk (what one LDS cycle serves of an MFMA operand read)
// then cover all sixteen 16-byte slots of a 256-byte bank window, so the
// reads are conflict-free (a (r >> 1) swizzle measured 50% bank-conflict
// cycles).  A load instruction fills 64 consecutive slots, so each lane
// fetches the global chunk that belongs in its slot.
template <int BM, int BN, bool SWIGLU>
__global__ __launch_bounds__(256, 1) void k_gemm_bf16_dma(GemmArgs g) {
  constexpr int BK = 32, STAGES = 4;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int A_SEG = BM * BK * 2 / 1024, B_SEG = BN * BK * 2 / 1024;  // 1 KB segments
  constexpr int A_LD = A_SEG / 4, B_LD = B_SEG / 4;                      // per wave
  int mt, nt;
  if (!balanced_tile<kGroupM>(*g.n_tiles, g.N / BN, &mt, &nt)) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int K = g.K, nk = K / BK;
  const char *Ag = (const char *)(g.A + (size_t)t.row0 * K * 2);
  const char *Bg = (const char *)(blob_of(g.bt, t.expert) + g.b_off + (size_t)nt * BN * K * 2);

  __shared__ u32x4 sA[STAGES][BM * 4];
  __shared__ u32x4 sB[STAGES][BN * 4];

  // this lane's source chunk inside a 1 KB segment (16 rows x 4 chunks)
  const int seg_row = lane >> 2;
  const int src_chunk = (lane & 3) ^ ((seg_row >> 2) & 3);
  const uint32_t lane_off = (uint32_t)seg_row * K * 2 + src_chunk * 16;

#define CEP_DMA_STAGE(kt)                                                              \
  {                                                                                    \
    const int buf_ = (kt) % STAGES;                                                    \
    _Pragma("unroll") for (int i = 0; i < A_LD; ++i) {                                 \
      const int seg = wid * A_LD + i;                                                  \
      dma16(Ag + (size_t)seg * 16 * K * 2 + (size_t)(kt) * BK * 2 + lane_off,          \
            __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf_][seg * 64])));          \
    }                                                                                  \
    _Pragma("unroll") for (int i = 0; i < B_LD; ++i) {                                 \
      const int seg = wid * B_LD + i;                                                  \
      dma16(Bg + (size_t)seg * 16 * K * 2 + (size_t)(kt) * BK * 2 + lane_off,          \
            __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf_][seg * 64])));          \
    }                                                                                  \
  }

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) CEP_DMA_STAGE(s);

  // operand slot offsets: row r = (wave base) + i*32 + lane%32 has
  // (r >> 2) & 3 == ((lane & 31) >> 2) & 3 for every fragment
  const int rsw = ((lane & 31) >> 2) & 3;
  for (int kt = 0; kt < nk; ++kt) {
    // this thread's loads of step kt are done when at most the loads of the
    // steps issued after it are still outstanding
    static_assert(STAGES == 4, "the waits below assume two later steps in flight");
    if (kt + 2 < nk)
      wait_vmcnt<2 * (A_LD + B_LD)>();
    else if (kt + 1 < nk)
      wait_vmcnt<A_LD + B_LD>();
    else
      wait_vmcnt<0>();
    // every wave's loads of step kt landed; step kt-1 fully consumed.  A bare
    // barrier: __syncthreads() would also drain the later steps' loads.
    __builtin_amdgcn_s_barrier();
    if (kt + STAGES - 1 < nk) CEP_DMA_STAGE(kt + STAGES - 1);
    const int cur = kt % STAGES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int slot = (kk * 2 + (lane >> 5)) ^ rsw;
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = __builtin_bit_cast(bf16x8, sA[cur][(wm * WM + i * 32 + (lane & 31)) * 4 + slot]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, sB[cur][(wn * WN + j * 32 + (lane & 31)) * 4 + slot]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
#undef CEP_DMA_STAGE

  // 32x32 accumulator layout: lane l, element r -> column l%32,
  // row 8*(r/4) + 4*(l/32) + r%4.
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rt = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (rt >= t.rows) continue;
      const size_t row = (size_t)t.row0 + rt;
      if (SWIGLU) {
        __bf16 *H = (__bf16 *)g.out;
        const size_t hbase = row * (g.N / 2) + (nt * BN + wn * WN) / 2 + (lane & 31);
#pragma unroll
        for (int j2 = 0; j2 < FN / 2; ++j2)
          H[hbase + j2 * 32] = (__bf16)silu_mul(acc[i][2 * j2][r], acc[i][2 * j2 + 1][r]);
      } else {
        const float w = g.wrow[row];
        float *Y = (float *)g.out;
        const size_t ybase = row * g.N + nt * BN + wn * WN + (lane & 31);
#pragma unroll
        for (int j = 0; j < FN; ++j) Y[ybase + j * 32] = acc[i][j][r] * w;
      }
    }
  }
}

// ---------------------------------------------------------------- bf16
// BM x BN output tile (256 x 256), K step 64, 4 waves as 2x2, each wave
// (BM/2) x (BN/2) built from v_mfma_f32_32x32x16_bf16 fragments, so each
// 16-byte LDS read feeds BM/64 (or BN/64) MFMAs.  LDS holds two K steps of
// A and B (double buffer, one barrier per step); the next step's tiles are
// fetched into registers while the current step computes, then written to
// the other buffer.  LDS rows are 64 bf16 (eight 16-byte chunks), chunk c of
// row r stored at c ^ (r & 7): the global->LDS stores and the MFMA operand
// reads (32 rows, one chunk each) are conflict-free.
template <int BM, int BN, bool SWIGLU>
__global__ __launch_bounds__(256, 1) void k_gemm_bf16(GemmArgs g) {
  constexpr int BK = 64;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int AV = BM * BK / 8 / 256, BV = BN * BK / 8 / 256;  // 16-byte loads per thread
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = L % g.max_tiles, nt = L / g.max_tiles;
  if (mt >= *g.n_tiles) return;
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int K = g.K, kv = K / 8, nk = K / BK;
  const u32x4 *Ag = (const u32x4 *)(g.A + (size_t)t.row0 * K * 2);
  const u32x4 *Bg = (const u32x4 *)(blob_of(g.bt, t.expert) + g.b_off + (size_t)nt * BN * K * 2);

  __shared__ u32x4 sA[2][BM * 8];
  __shared__ u32x4 sB[2][BN * 8];
  u32x4 ra[AV], rb[BV];
#define CEP_BF16_GLOAD(kt)                                              \
  _Pragma("unroll") for (int i = 0; i < AV; ++i) {                      \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;              \
    ra[i] = Ag[(size_t)row * kv + (kt) * 8 + ch];                       \
  }                                                                     \
  _Pragma("unroll") for (int i = 0; i < BV; ++i) {                      \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;              \
    rb[i] = Bg[(size_t)row * kv + (kt) * 8 + ch];                       \
  }
#define CEP_BF16_LSTORE(buf)                                            \
  _Pragma("unroll") for (int i = 0; i < AV; ++i) {                      \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;              \
    sA[buf][row * 8 + (ch ^ (row & 7))] = ra[i];                        \
  }                                                                     \
  _Pragma("unroll") for (int i = 0; i < BV; ++i) {                      \
    const int v = tid + 256 * i, row = v >> 3, ch = v & 7;              \
    sB[buf][row * 8 + (ch ^ (row & 7))] = rb[i];                        \
  }

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

  CEP_BF16_GLOAD(0);
  CEP_BF16_LSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      CEP_BF16_GLOAD(kt + 1);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 a[FM], b[FN];
      const int ch = kk * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * WM + i * 32 + (lane & 31);
        a[i] = __builtin_bit_cast(bf16x8, sA[cur][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * WN + j * 32 + (lane & 31);
        b[j] = __builtin_bit_cast(bf16x8, sB[cur][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      CEP_BF16_LSTORE(cur ^ 1);
    }
    __syncthreads();
  }
#undef CEP_BF16_GLOAD
#undef CEP_BF16_LSTORE

  // 32x32 accumulator layout: lane l, element r -> column l%32,
  // row 8*(r/4) + 4*(l/32) + r%4.
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rt = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (rt >= t.rows) continue;
      const size_t row = (size_t)t.row0 + rt;
      if (SWIGLU) {
        // fragment pairs (2*j2, 2*j2+1) are the gate and up columns of h
        // columns (nt*BN + wn*WN)/2 + j2*32 + [0, 32)
        __bf16 *H = (__bf16 *)g.out;
        const size_t hbase = row * (g.N / 2) + (nt * BN + wn * WN) / 2 + (lane & 31);
#pragma unroll
        for (int j2 = 0; j2 < FN / 2; ++j2)
          H[hbase + j2 * 32] = (__bf16)silu_mul(acc[i][2 * j2][r], acc[i][2 * j2 + 1][r]);
      } else {
        const float w = g.wrow[row];
        float *Y = (float *)g.out;
        const size_t ybase = row * g.N + nt * BN + wn * WN + (lane & 31);
#pragma unroll
        for (int j = 0; j < FN; ++j) Y[ybase + j * 32] = acc[i][j][r] * w;
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

template <bool SWIGLU>
hipError_t launch_any(const GemmArgs &g, int grid_tiles, int align, bool fp8, hipStream_t s) {
  if (fp8) {
    if (align != kFp8TileM) return hipErrorInvalidValue;
    const int grid = grid_tiles * (g.N / 256);
    hipLaunchKernelGGL(k_gemm_fp8<SWIGLU>, dim3(grid), dim3(256), 0, s, g);
  } else if (align == kBf16TileM) {
    const int grid = balanced_grid(grid_tiles, kGroupM, g.N / kBf16TileN);
    hipLaunchKernelGGL((k_gemm_bf16_dma<kBf16TileM, kBf16TileN, SWIGLU>), dim3(grid), dim3(256),
                       0, s, g);
  } else if (align == kBf16SmallTileM) {
    const int grid = balanced_grid(grid_tiles, kGroupM, g.N / kBf16TileN);
    hipLaunchKernelGGL((k_gemm_bf16_dma<kBf16SmallTileM, kBf16TileN, SWIGLU>), dim3(grid),
                       dim3(256), 0, s, g);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm1(const Scratch &sc, int which, int list_cap, int grid_tiles, int align,
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
  return launch_any<true>(g, grid_tiles, align, fp8, s);
}

hipError_t launch_gemm2(const Scratch &sc, int which, int list_cap, int grid_tiles, int align,
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
  return launch_any<false>(g, grid_tiles, align, fp8, s);
}

}  // namespace cep
