// Device helpers shared by the grouped GEMM kernels (bf16, e4m3, MXFP4).
// Internal to libcep.
#pragma once

#include "common.h"

#include <hip/hip_bf16.h>

namespace cep {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Arguments of one grouped GEMM launch.  Both GEMMs are "NT" products:
// A = grouped rows [M][K], B = packed weights [N][K], K contiguous in both,
// so every MFMA operand is a contiguous run of K.  Work is a device tile
// list (expert, first row, valid rows) built by the routing scan.
struct GemmArgs {
  const uint8_t *A;       // grouped rows [mpad][K] (bf16 or e4m3)
  const float *As;        // e4m3: [K/128][s_ld] row scales, k-block major;
                          // mx: E8M0 bytes at mx_row_scale_offset
  int s_ld;               // quantised A: row stride of the scale matrices
  const Tile *tiles;      // tile list
  const int32_t *n_tiles; // live tiles in the list
  int max_tiles;          // grid extent in M tiles (host upper bound)
  int K, N;               // contraction length, packed output columns
  size_t b_off, bs_off;   // offsets of B and its scales in each blob
  BlobTable bt;
  void *out;              // H [mpad][N/2] (GEMM1) or Y [mpad][N] (GEMM2: float32
                          // with bf16 weights, bf16 with e4m3 / MXFP4 weights)
  float *out_s;           // quantised GEMM1: h scales (layout of As, K = N/2)
  const float *wrow;      // GEMM2: routing coefficient per grouped row
  // GEMM2 (e4m3, MXFP4): ydst[r] >= 0 sends grouped row r to row ydst[r] of
  // yout ([.][N] float32), the output row of its token's only local pair;
  // null: every row goes to out
  float *yout;
  const int32_t *ydst;
  // bf16 GEMM1 with A == nullptr: grouped row r is the batch's input row
  // xrow[arow0 + perm[r] / k] (padding rows, perm -1, read row arow0)
  const void *const *xrow;
  const int32_t *perm;
  int arow0, k;
};

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Grouped tile order over the n_live M tiles: GM consecutive M tiles x all
// N tiles form a group, M fastest inside it, so the workgroups an XCD runs
// together share GM row panels of A and the weight panels of their N tiles
// in that XCD's L2.  The last group holds the n_live % GM remaining M tiles,
// so the order covers live tiles only.
template <int GM>
__device__ inline void tile_of(int L, int n_live, int n_tiles_n, int *mt, int *nt) {
  const int full = n_live / GM, full_work = full * GM * n_tiles_n;
  if (L < full_work) {
    const int grp = L / (GM * n_tiles_n), idx = L % (GM * n_tiles_n);
    *mt = grp * GM + idx % GM;
    *nt = idx / GM;
  } else {
    const int gl = n_live - full * GM, idx = L - full_work;
    *mt = full * GM + idx % gl;
    *nt = idx / gl;
  }
}

// Work item of this workgroup, balanced over the XCDs.  The grid covers the
// host's upper bound on M tiles; the live count is on the device.  The live
// work W = n_live x N tiles is cut into 8 contiguous shares, one per XCD
// (workgroup ids are dispatched round-robin over the XCDs), so the surplus
// workgroups of the bound never leave an XCD idle while another holds the
// tail.  Returns false for a surplus workgroup.
template <int GM>
__device__ inline bool balanced_tile(int n_live, int n_tiles_n, int *mt, int *nt) {
  const int W = n_live * n_tiles_n;
  const int C = (W + 7) / 8;
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int L = x * C + j;
  if (j >= C || L >= W) return false;
  tile_of<GM>(L, n_live, n_tiles_n, mt, nt);
  return true;
}

// Work item it of this workgroup, balanced over the XCDs as balanced_tile:
// the live work W = n_live x N tiles is cut into 8 contiguous shares, one per
// XCD.  A persistent grid (one workgroup per CU, gridDim.x a multiple of 8)
// takes items j, j + gridDim.x/8, ... of its XCD's share; otherwise a
// workgroup takes item blockIdx.x/8 only.
template <int GM, bool PERSIST>
__device__ inline bool work_item(int it, int n_live, int n_tiles_n, int *mt, int *nt) {
  if (!PERSIST && it > 0) return false;
  const int W = n_live * n_tiles_n;
  const int C = (W + 7) / 8;
  const int x = blockIdx.x & 7, j = (blockIdx.x >> 3) + it * (int)(gridDim.x >> 3);
  const int L = x * C + j;
  if (j >= C || L >= W) return false;
  tile_of<GM>(L, n_live, n_tiles_n, mt, nt);
  return true;
}

// One workgroup per CU of the current device, a multiple of 8 (the XCDs).
inline int persistent_grid() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8)
      n = 256;
    cached[dev] = n / 8 * 8;
  }
  return cached[dev];
}

// Grid for balanced_tile: at least the bound's work, a multiple of 8.
inline int balanced_grid(int grid_tiles, int gm, int n_tiles_n) {
  return ((grid_tiles + gm - 1) / gm * gm * n_tiles_n + 7) / 8 * 8;
}
// M tiles per tile group.  With four, the workgroups an XCD runs together
// re-read each 256-row A panel about a third less often from HBM than with
// eight, at equal or better speed (measured on the bf16 and MXFP4 GEMM1 of
// the DeepSeek-V4-Flash-shaped and 4096-wide workloads).
constexpr int kGroupM = 4;
// M tiles per group when whole groups go to one XCD (work_item_xg): eight,
// so that 32 workgroups run an 8 x 4 block (as few distinct panels as 4 x 8)
// and groups of 20 or 24 column tiles are a whole number of rounds.
constexpr int kGroupXcd = 8;

// Persistent work item it of this workgroup, whole tile groups per XCD when
// that costs no round: group g (GM consecutive M tiles x all N tiles, M
// fastest) belongs to XCD g % 8, whose gridDim.x/8 workgroups take items j,
// j + gridDim.x/8, ... of its groups in order.  When a group's items are a
// whole number of rounds, every round of an XCD's workgroups is then one
// GM x (32/GM) block of a single group (work_item's contiguous shares start
// mid-group, so some of its rounds span two groups and share less in L2:
// e4m3 GEMM1 L2 hit rate 73 -> 78 %).  Otherwise, or when whole groups would
// leave the busiest XCD more rounds than contiguous shares, work_item.
template <int GM>
__device__ inline bool work_item_xg(int it, int n_live, int n_tiles_n, int *mt, int *nt) {
  const int wpx = (int)(gridDim.x >> 3);  // workgroups per XCD
  const int per = GM * n_tiles_n;         // items of a full group
  const int ngroups = (n_live + GM - 1) / GM;
  const int r_xg = ((ngroups + 7) / 8 * per + wpx - 1) / wpx;
  const int r_bal = ((n_live * n_tiles_n + 7) / 8 + wpx - 1) / wpx;
  if (per % wpx != 0 || r_xg > r_bal) return work_item<kGroupM, true>(it, n_live, n_tiles_n, mt, nt);
  const int x = blockIdx.x & 7, j = (blockIdx.x >> 3) + it * wpx;
  const int g = x + 8 * (j / per), w = j % per;
  if (g >= ngroups) return false;
  const int gm = min(GM, n_live - g * GM);  // M tiles of this group
  if (w >= gm * n_tiles_n) return false;    // past the last (partial) group
  *mt = g * GM + w % gm;
  *nt = w / gm;
  return true;
}

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

// dma16 from a wave-uniform base address (scalar registers) plus a per-lane
// 32-bit byte offset: only the offset occupies a vector register.
__device__ inline void dma16_s(const void *sbase, uint32_t voff, uint32_t lds_seg) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "s"(lds_seg)
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

// Waits until at most n (wave-uniform, LO <= n) vector-memory operations of
// this wave are outstanding; n above HI waits for HI.  A binary search over
// the immediate of s_waitcnt.
template <int LO, int HI>
__device__ inline void wait_vmcnt_upto(int n) {
  if constexpr (LO >= HI) {
    wait_vmcnt<HI>();
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (n <= MID)
      wait_vmcnt_upto<LO, MID>(n);
    else
      wait_vmcnt_upto<MID + 1, HI>(n);
  }
}

// Waits for this wave's LDS (and scalar-memory) operations only; a barrier
// after it synchronises LDS use without waiting for outstanding global
// stores (__syncthreads() would also wait for those).
__device__ inline void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (3 << 14)); }

// Waits until at most r (0 <= r <= R) groups of PER vector-memory operations
// of this wave are outstanding.
template <int PER, int R>
__device__ inline void wait_stages(int r) {
  static_assert(R <= 6, "deeper rings need more cases");
  if constexpr (R >= 6) {
    if (r >= 6) return wait_vmcnt<6 * PER>();
  }
  if constexpr (R >= 5) {
    if (r >= 5) return wait_vmcnt<5 * PER>();
  }
  if constexpr (R >= 4) {
    if (r >= 4) return wait_vmcnt<4 * PER>();
  }
  if constexpr (R >= 3) {
    if (r >= 3) return wait_vmcnt<3 * PER>();
  }
  if constexpr (R >= 2) {
    if (r >= 2) return wait_vmcnt<2 * PER>();
  }
  if constexpr (R >= 1) {
    if (r >= 1) return wait_vmcnt<PER>();
  }
  wait_vmcnt<0>();
}

// Epilogues of the block-scaled 8 x 4-fragment wave tiles (e4m3 and MXFP4
// weights).  With the weight fragment as the MFMA's first operand,
// acc[i][j][r] is row wm*128 + i*16 + l%16 and column wn*64 + j*16 +
// 4*(l/16) + r of the 256-column tile nt (lane l), so each lane holds four
// consecutive outputs of a row.
//
// GEMM2: the routing coefficients of the lane's eight rows, loaded before
// the K loop so that their latency hides behind it (loaded in the epilogue,
// each load's wait would also wait for the stores before it).
__device__ inline void load_row_coef(const GemmArgs &g, const Tile &t, int wm, int lane,
                                     float (&wr)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int rt = wm * 128 + i * 16 + (lane & 15);
    wr[i] = rt < t.rows ? g.wrow[(size_t)t.row0 + rt] : 0.0f;
  }
}

// GEMM2: the output rows of the lane's eight rows for a direct write
// (GemmArgs::ydst), -1 for a grouped output row; loaded with the
// coefficients.
__device__ inline void load_row_dst(const GemmArgs &g, const Tile &t, int wm, int lane,
                                    int (&yd)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int rt = wm * 128 + i * 16 + (lane & 15);
    yd[i] = g.ydst && rt < t.rows ? g.ydst[(size_t)t.row0 + rt] : -1;
  }
}

// The bits of +0.0f + x for the float with bits x: -0 becomes +0.  A token's
// only grouped output, written as its output row, gets the bits the combine's
// float32 sum from +0 would give it.
__device__ inline uint32_t plus_zero(uint32_t x) { return x == 0x80000000u ? 0u : x; }

// Eight bf16 (a 16-byte piece of a y row) widened to float32, +0 for -0.
__device__ inline void widen_bf16x8(const u32x4 &v, u32x4 &lo, u32x4 &hi) {
  lo = u32x4{plus_zero(v.x << 16), plus_zero(v.x & 0xffff0000u), plus_zero(v.y << 16),
             plus_zero(v.y & 0xffff0000u)};
  hi = u32x4{plus_zero(v.z << 16), plus_zero(v.z & 0xffff0000u), plus_zero(v.w << 16),
             plus_zero(v.w & 0xffff0000u)};
}

// GEMM2: y = coefficient * acc in bf16, four consecutive columns (8 bytes)
// per lane and row; a row with yd[i] >= 0 goes to that output row as float32
// (16 bytes).
__device__ inline void store_y_bf16(const f32x4 (&acc)[8][4], const float (&wrow)[8],
                                    const int (&yd)[8], const GemmArgs &g, const Tile &t, int nt,
                                    int wm, int wn, int lane) {
  __bf16 *Y = (__bf16 *)g.out;
  const int r16 = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int rt = wm * 128 + i * 16 + r16;
    if (rt >= t.rows) continue;
    const size_t row = (size_t)t.row0 + rt;
    const float wr = wrow[i];
    const size_t col = (size_t)nt * 256 + wn * 64 + 4 * grp;
    __bf16 *yrow = Y + row * g.N + col;
    uint32_t *orow = yd[i] >= 0 ? (uint32_t *)g.yout + (size_t)yd[i] * g.N + col : nullptr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t v[2];
#pragma unroll
      for (int r = 0; r < 2; ++r)
        v[r] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[i][j][2 * r] * wr)) |
               ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[i][j][2 * r + 1] * wr)) << 16);
      if (orow)
        *(u32x4 *)(orow + j * 16) = u32x4{plus_zero(v[0] << 16), plus_zero(v[0] & 0xffff0000u),
                                          plus_zero(v[1] << 16), plus_zero(v[1] & 0xffff0000u)};
      else
        *(uint2 *)(yrow + j * 16) = make_uint2(v[0], v[1]);
    }
  }
}

// GEMM2 outputs y = coefficient * acc of a wave's 8 x 4 fragments, rounded
// to bf16: two consecutive columns per word.  Packed as soon as the
// accumulators are final, they take half the registers.
__device__ inline void pack_y_bf16(const f32x4 (&acc)[8][4], const float (&wrow)[8],
                                   uint32_t (&yb)[8][4][2]) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        yb[i][j][h] =
            (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[i][j][2 * h] * wrow[i])) |
            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[i][j][2 * h + 1] * wrow[i]))
             << 16);
}

// GEMM2 through LDS: the waves write their packed bf16 outputs (pack_y_bf16)
// into idle operand-ring buffers (512 bytes a row, 16-byte chunk c of row r
// at slot c ^ (r & 15), so that the sixteen rows of one write instruction
// hit distinct banks), then the workgroup stores whole rows with 16-byte
// stores: one store instruction covers two full rows, where the accumulator
// layout gives 64 pieces of 8 bytes.  One pass per wave row of 128 rows,
// staged as rows 0-63 in lo and 64-127 in hi (32 KB each).  The barriers
// wait for LDS operations only: loads and stores in flight (the previous
// pass's stores, a persistent workgroup's prefetch of its next tile) are not
// waited for.  FULL stores the padding rows of the tile too (never read), so
// that every wave issues at least a fixed number of stores.  sD (LDS) holds
// the tile rows' GemmArgs::ydst: a row with sD[row] >= 0 goes to that output
// row as float32 (two 16-byte stores per piece), padding rows have -1.
// Returns a lower bound of the store instructions the wave issued (FULL): a
// piece's store instructions run only for lanes that take their branch.
template <int NW, bool FULL = false>
__device__ inline int store_y_bf16_staged(const uint32_t (&yb)[8][4][2], const GemmArgs &g,
                                          const Tile &t, int nt, int wm, int wn, int lane,
                                          int tid, u32x4 *lo, u32x4 *hi, const int *sD) {
  const int r16 = lane & 15, grp = lane >> 4;
  int n_st = 0;
  __bf16 *Y = (__bf16 *)g.out + (size_t)t.row0 * g.N + (size_t)nt * 256;
#pragma unroll
  for (int pass = 0; pass < NW / 4; ++pass) {
    // no wave still reads the buffers (ring or the previous pass's rows)
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    if (wm == pass) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        u32x4 *st = i < 4 ? lo : hi;
        const int r = (i & 3) * 16 + r16;  // row within the 64-row piece
#pragma unroll
        for (int j = 0; j < 4; ++j) {
      const int c = wn * 8 + j * 2 + (grp >> 1);  // 16-byte chunk of the row
          uint2 *dst = (uint2 *)&st[r * 32 + (c ^ r16)] + (grp & 1);
          *dst = make_uint2(yb[i][j][0], yb[i][j][1]);
        }
      }
    }
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
#pragma unroll 4
    for (int q = tid; q < 128 * 32; q += 64 * NW) {
      const int lr = q >> 5, c = q & 31, row = pass * 128 + lr;
      if (!FULL && row >= t.rows) break;  // q grows with the row
      const u32x4 *src = lr < 64 ? lo : hi;
      const int pr = lr & 63;
      const u32x4 v = src[pr * 32 + (c ^ (pr & 15))];
      const int od = sD[row];
      n_st += (__ballot(od >= 0) ? 2 : 0) + (__ballot(od < 0) ? 1 : 0);
      if (od >= 0) {
        u32x4 f0, f1;
        widen_bf16x8(v, f0, f1);
        u32x4 *o = (u32x4 *)(g.yout + (size_t)od * g.N + (size_t)nt * 256 + c * 8);
        o[0] = f0;
        o[1] = f1;
      } else {
        *(u32x4 *)(Y + (size_t)row * g.N + c * 8) = v;
      }
    }
  }
  return __builtin_amdgcn_readfirstlane(n_st);
}

// GEMM1: h = silu(gate) * up, quantised to MXFP8.  The wave's 64 columns are
// 32 gate and 32 up columns (interleaved in groups of 32), so its 32 h
// columns of a row -- one MX block -- lie in the four lanes of the row: the
// block amax takes two cross-lane steps.  The E8M0 scale is
// 2^(floor(log2 amax) - 8) (emax of e4m3), the codes e4m3(h / scale)
// saturated at 448.
//
// The codes go through the idle operand ring (128 bytes a row, 16-byte chunk
// c of row r at slot c ^ ((r >> 1) & 7): a write instruction's sixteen rows x
// four dwords hit distinct banks), then the workgroup stores whole 128-byte
// row segments with 16-byte stores.  st holds BM x 128 bytes.  Barriers and
// FULL as in store_y_bf16_staged.
template <int NW, bool FULL = false>
__device__ inline void store_h_mx_staged(const f32x4 (&acc)[8][4], const GemmArgs &g,
                                         const Tile &t, int nt, int wm, int wn, int lane,
                                         int tid, u32x4 *st) {
  uint8_t *Hs = (uint8_t *)g.out_s;
  const int I = g.N / 2, hblk = nt * 4 + wn;  // this wave's MX block of h columns
  const int r16 = lane & 15, grp = lane >> 4;
  wait_lgkm0();  // every wave's last operand reads completed: the buffer is idle
  __builtin_amdgcn_s_barrier();
  uint32_t *st32 = (uint32_t *)st;
  int codes[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float h[2][4];
    float m = 0.0f;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        h[jj][r] = silu_mul(acc[i][jj][r], acc[i][jj + 2][r]);
        m = fmaxf(m, fabsf(h[jj][r]));
      }
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    const int code = max((int)((__float_as_uint(m) >> 23) & 0xff) - 8, 0);
    const int e = 127 - code;  // h / 2^(code - 127), exact
    const int rt = wm * 128 + i * 16 + r16;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      float q[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) q[r] = fminf(fmaxf(ldexpf(h[jj][r], e), -448.0f), 448.0f);
      int v = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], 0, false);
      v = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], v, true);
      // bytes wn*32 + jj*16 + 4*grp of the row: chunk 2*wn + jj, dword grp
      const int c = 2 * wn + jj;
      st32[(rt * 8 + (c ^ ((rt >> 1) & 7))) * 4 + grp] = (uint32_t)v;
    }
    codes[i] = code;
  }
  wait_lgkm0();
  __builtin_amdgcn_s_barrier();
  uint8_t *H = (uint8_t *)g.out + (size_t)t.row0 * I + (size_t)nt * 128;
  constexpr int BM = 128 * NW / 4;
#pragma unroll 2
  for (int q = tid; q < BM * 8; q += 64 * NW) {
    const int row = q >> 3, c = q & 7;
    if (!FULL && row >= t.rows) break;  // q grows with the row
    *(u32x4 *)(H + (size_t)row * I + c * 16) = st[row * 8 + (c ^ ((row >> 1) & 7))];
  }
  // the scales last (a store before the barrier would make it wait for
  // them): lane r16 of the wave's first sixteen holds rows r16 + 16i of a
  // 128-row group (the tile's rows start at a multiple of 128), whose scales
  // are one 8-byte word of the layout; padding rows' words are never read
  if (grp == 0) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lo |= (uint32_t)codes[i] << (8 * i);
      hi |= (uint32_t)codes[i + 4] << (8 * i);
    }
    *(uint2 *)(Hs + mx_row_scale_offset(t.row0 + wm * 128 + r16, hblk, g.s_ld)) =
        make_uint2(lo, hi);
  }
}

// Launchers of the two kernel families (grid from the tile bound).
template <bool SWIGLU>
hipError_t launch_bf16(const GemmArgs &g, int grid_tiles, int align, hipStream_t s);
// bf16 GEMM over the scan's 64-row remainder tiles
template <bool SWIGLU>
hipError_t launch_bf16_rem(const GemmArgs &g, int grid_tiles, hipStream_t s);
// bf16 GEMM over a list of 128-row and 64-row (half) tiles
template <bool SWIGLU>
hipError_t launch_bf16_var(const GemmArgs &g, int grid_tiles, hipStream_t s);
// bf16 GEMM1 (SwiGLU) of a weight-streaming batch over its 64-row tiles
// ordered by rows, one 64-column work item per workgroup in list order
hipError_t launch_bf16_stream(const GemmArgs &g, int grid_tiles, hipStream_t s);
// bf16 GEMM2 of a weight-streaming batch over the same list, 128-column items
hipError_t launch_bf16_stream2(const GemmArgs &g, int grid_tiles, hipStream_t s);
template <bool SWIGLU>
hipError_t launch_fp8(const GemmArgs &g, int grid_tiles, int align, hipStream_t s);
template <bool SWIGLU>
hipError_t launch_mx(const GemmArgs &g, int grid_tiles, int align, hipStream_t s);

}  // namespace cep
