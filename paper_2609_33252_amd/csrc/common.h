// Internal declarations shared by libcep's kernels and its runtime.
// Not part of the public ABI (include/cep.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#define CEP_API extern "C" __attribute__((visibility("default")))

namespace cep {

constexpr int kMaxExperts = 64;
constexpr int kMaxTopK = 16;
constexpr int kMaxDim = 32768;  // largest d_model and d_ff (fp8 GEMM keeps K/128 weight scales per row in LDS)
constexpr int kBf16TileM = 256;      // bf16 grouped GEMM tile
constexpr int kBf16TileN = 256;
constexpr int kFp8TileM = 128;       // e4m3 / MXFP4 grouped GEMM tile (4 waves)
constexpr int kFp8LargeTileM = 256;  // e4m3 / MXFP4 tile for large batches (8 waves)
constexpr int kRouteThreads = 256;   // threads per routing block
constexpr int kRoutePairs = 1024;    // flat pairs per routing block (4 rounds of 256)
constexpr int kInterleave = 32;           // gate/up column interleave of the packed W1
// Packed bf16 weights ([N][K], K contiguous per output column n) are stored
// in 16 KB blocks of 128 columns x 64 K, block (n/128, k/64) at element
// ((n/128)*(K/64) + k/64)*8192; inside a block the 32-wide K half
// (k/32)%2 takes 8 KB, each 16-column group (n/16)%8 of it 1 KB, column
// n%16 32 elements, k%32 within it.  A weight-streaming workgroup (128
// columns, 64 K per step) then reads one contiguous 16 KB run per step and
// a 256-column tile two 8 KB runs (32 K per step); each 1 KB direct-to-LDS
// load is one contiguous piece.  Requires N % 128 == 0 and K % 64 == 0.
__host__ __device__ inline size_t bf16_block_index(int n, int k, int K) {
  return ((size_t)(n >> 7) * (K >> 6) + (k >> 6)) * 8192 + ((k >> 5) & 1) * 4096 +
         ((n >> 4) & 7) * 512 + (n & 15) * 32 + (k & 31);
}
// K-step stride of bf16_block_index: K advancing by 32 moves 8 KB
constexpr int kBf16BlockStepBytes = 8192;
// batches up to this many flat (row, slot) entries route in one block (ids
// in LDS); beyond it the two-kernel path (count, then scan + scatter) is
// faster: one block's scatter grows with the entries, the other path's cost
// is mostly its two launches (staging and routing per batch, straggler
// workload: batches of ~2 K pairs 31 -> 22 us, of ~1 K pairs 19.3 -> 18.4 us
// against a 16 K crossover)
constexpr int kFusedRoutePairs = 1 << 12;
constexpr int kMxBlock = 32;               // MX scale block along K

// Expert weight format of a context (from cep_config.w_dtype).
enum WKind : int { kWBf16 = 0, kWFp8 = 1, kWMx = 2 };

// One M tile of a grouped GEMM: expert, first grouped row, valid rows in it.
struct Tile {
  int expert;
  int row0;
  int rows;
  int pad;
};

// Where each expert's packed weight blob lives for one grouped invocation:
// resident experts in the context's region, fetched experts in the fetch
// buffer (or, after a failed or skipped copy, in the donor region itself),
// experts without weights null (the host never launches tiles for them).
struct BlobTable {
  const uint8_t *blob[kMaxExperts];
};

__host__ __device__ inline const uint8_t *blob_of(const BlobTable &t, int e) { return t.blob[e]; }

// Packed blob layout of one expert (byte offsets from the blob start).
//   bf16: W1p [2I][d] bf16, W2p [d][I] bf16, in bf16_block_index order
//   fp8 : W1p [2I][d] u8, W2p [d][I] u8, S1 [2I/32][d/128] f32, S2 [d/128][I/128] f32
//   mx  : W1p [2I][d/2], W2p [d][I/2] packed e2m1 (even K in the low nibble)
//         in mx_block_index order,
//         S1, S2: E8M0 bytes in mx_weight_scale_offset order (N = 2I or d)
// Row n' of W1p holds column j = (n'/64)*32 + n'%32 of the gate weights when
// (n'/32) is even and of the up weights when it is odd, so that one 64-row
// group carries matching gate and up columns for the fused SwiGLU.
struct BlobLayout {
  size_t w1_off, w2_off, s1_off, s2_off, bytes;
};

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

constexpr int kBf16SmallTileM = 64;  // bf16 tile for batches with few rows per expert
// Such batches with at least kBf16VarMinRows pairs per local expert on
// average run both GEMMs in 128-row tiles over the same 64-aligned layout:
// an expert's rows in tiles of 128, the last of them a 64-row half tile when
// at most 64 rows remain (a hot expert then reads its weights once per 128
// rows instead of once per 64)
constexpr int kBf16VarTileM = 128;
constexpr int kBf16VarMinRows = 64;
inline bool batch_var_tiles(int wk, int align, int pairs, int n_experts) {
  return wk == kWBf16 && align == kBf16SmallTileM && pairs >= kBf16VarMinRows * n_experts;
}
// Smaller bf16 batches stream the weights: GEMM1 runs the 64-row tiles
// ordered by rows (most first) in 64-column work items handed to free CUs
// in that order (launch_bf16_stream), GEMM2 the 64-row tiles as listed.
inline bool batch_stream_tiles(int wk, int align, int pairs, int n_experts) {
  return wk == kWBf16 && align == kBf16SmallTileM && pairs < kBf16VarMinRows * n_experts;
}

// Per-expert row alignment A of one batch's grouped layout = M tile of the
// GEMMs that run it.  bf16 batches with fewer than one large tile of rows
// per local expert on average use the small tile: the GEMMs then stream the
// weights with four times as many workgroups.  Both bf16 tiles accumulate K
// in the same order with the same MFMA, so results do not depend on it.
inline int batch_align(int wk, int pairs, int n_experts) {
  if (wk != kWBf16) return pairs >= kFp8LargeTileM * n_experts ? kFp8LargeTileM : kFp8TileM;
  return pairs >= kBf16TileM * n_experts ? kBf16TileM : kBf16SmallTileM;
}
constexpr int kMinAlign = 64;
constexpr int kMaxAlign = 256;

inline BlobLayout blob_layout(int d, int I, int wk) {
  BlobLayout L{};
  if (wk == kWMx) {
    L.w1_off = 0;
    L.w2_off = align_up((size_t)I * d, 256);
    L.s1_off = align_up(L.w2_off + (size_t)d * I / 2, 256);
    L.s2_off = align_up(L.s1_off + (size_t)2 * I * d / kMxBlock, 256);
    L.bytes = align_up(L.s2_off + (size_t)d * I / kMxBlock, 256);
    return L;
  }
  const bool fp8 = wk == kWFp8;
  size_t es = fp8 ? 1 : 2;
  L.w1_off = 0;
  L.w2_off = align_up(L.w1_off + (size_t)2 * I * d * es, 256);
  size_t end = L.w2_off + (size_t)d * I * es;
  if (fp8) {
    L.s1_off = align_up(end, 256);
    L.s2_off = align_up(L.s1_off + (size_t)(2 * I / kInterleave) * (d / 128) * 4, 256);
    end = L.s2_off + (size_t)(d / 128) * (I / 128) * 4;
  }
  L.bytes = align_up(end, 256);
  return L;
}

// MXFP8 scales of grouped rows (activations and h; s_ld a multiple of 256,
// row groups of 128).  The E8M0 scale of row R, K block b (32 channels) sits
// where one K step of 128 (4 blocks) of a 128-row group is 512 contiguous
// bytes and the scales of rows R%16 + 16i, i = 0..7, of one block are one
// 8-byte word: the four-byte halves feed the MFMA's byte-selected scale
// operand of row fragments i = 0..3 and 4..7.
__host__ __device__ inline size_t mx_row_scale_offset(int R, int b, int s_ld) {
  return ((size_t)(b >> 2) * (s_ld >> 7) + (R >> 7)) * 512 + (b & 3) * 128 + (R & 15) * 8 +
         ((R & 127) >> 4);
}

// E8M0 weight scales in a blob (B = [N][K] packed weights, N a multiple of
// 256): for each 256-column tile and K step of 128 one 1 KB record holding,
// for the wave of column group wn (64 columns), the lane of K block g and
// column n16, the scales of its four 16-column fragments j as one word.
// Packed e2m1 weights ([N][K/2] bytes, row_bytes = K/2 per output column n)
// are stored in 1 KB blocks of 16 columns x 64 bytes (128 K), so that one
// 1 KB direct-to-LDS load of a 128-wide K step reads one contiguous block:
// byte k of column n at ((n/16)*(row_bytes/64) + k/64)*1024 + (n%16)*64 + k%64.
__host__ __device__ inline size_t mx_block_index(int n, int k, int row_bytes) {
  return ((size_t)(n >> 4) * (row_bytes >> 6) + (k >> 6)) * 1024 + (n & 15) * 64 + (k & 63);
}

__host__ __device__ inline size_t mx_weight_scale_offset(int n, int b, int K) {
  const int nt = n >> 8, wn = (n >> 6) & 3, j = (n >> 4) & 3, n16 = n & 15;
  return ((size_t)nt * (K >> 7) + (b >> 2)) * 1024 + ((wn * 4 + (b & 3)) * 16 + n16) * 4 + j;
}

// Chunk arena of one layer: one entry per submitted row, in submission order.
struct Arena {
  int32_t *ids;        // [cap][k] local expert id or -1
  float *w;            // [cap][k] routing coefficient
  int32_t *dst;        // [cap] output row (replica * T_max + token) or -1
  int32_t *solo;       // [cap] the output row of a row with exactly one local
                       // pair, else -1
  const void **xrow;   // [cap] pointer to the row's input
};

// Per-stream-slot scratch of one grouped invocation.
struct Scratch {
  int32_t *blk_cnt;    // [max_blocks][E] pairs per (routing block, expert)
  int32_t *cnt;        // [E]
  int32_t *off;        // [E+1]
  int32_t *off_pad;    // [E+1]
  Tile *tiles;         // [4][max_tiles]: list 2*f + r for resident (f = 0) or
                       // fetched (f = 1) experts; r = 1: 64-row remainder tiles
                       // (256-row batches) or 128-row tiles (batch_var_tiles)
  int32_t *n_tiles;    // [4]
  int32_t *pos_of;     // [max_rows * k] grouped row of each flat pair or -1
  int32_t *perm;       // [max_mpad] flat pair of each grouped row or -1
  float *wrow;         // [max_mpad] routing coefficient of each grouped row
  int32_t *ydst;       // [max_mpad] output row of a grouped row that is its
                       // token's only local pair (GEMM2 writes that token's
                       // output row itself), else -1
  void *xg;            // [max_mpad][d] bf16 or e4m3
  float *xs;           // e4m3 and MXFP4 weights: the rows' E8M0 scales (MXFP8,
                       // one byte per 32 channels) at mx_row_scale_offset
  uint8_t *xs_rows;    // [max_mpad][xs_pitch] the same bytes row-major, as the
                       // pack writes them (k_scale_layout moves them to xs)
  int xs_pitch;        // d/32 rounded up to 16 bytes
  void *h;             // [max_mpad][I] bf16 or e4m3
  float *hs;           // scales of h, laid out like xs (K = I)
  int s_ld;            // row stride of xs / hs (= max_mpad, a multiple of 256)
  void *y;             // [max_mpad][d] expert outputs already scaled by the
                       // coefficient: float32 with bf16 weights (the combine
                       // then sums exactly the float32 products), bf16 with
                       // e4m3 / MXFP4 weights (their h quantisation error is
                       // ~2^-4, a bf16 rounding ~2^-9 adds nothing measurable)
};

// Device error word bits.
enum : uint32_t { kErrBadId = 1u, kErrPairCount = 2u, kErrBadToken = 4u, kErrOverflow = 8u };

// ---- launchers (implemented in the .hip files) ----
// weight packing
hipError_t launch_pack_w1(const void *wg, const void *wu, int w_dtype, int d, int I,
                          uint8_t *dst_w1, hipStream_t s);
hipError_t launch_pack_w2(const void *wd, int w_dtype, int d, int I, uint8_t *dst_w2,
                          hipStream_t s);
hipError_t launch_pack_scales(const float *sg, const float *su, const float *sd, int d, int I,
                              float *dst_s1, float *dst_s2, hipStream_t s);
// MXFP4 experts: caller layout gate/up [I][d/2] + [I][d/32], down [d][I/2] +
// [d][I/32] (output-major, K packed) into the blob of layout L
hipError_t launch_pack_mx(const uint8_t *wg, const uint8_t *wu, const uint8_t *wd,
                          const uint8_t *sg, const uint8_t *su, const uint8_t *sd, int d, int I,
                          uint8_t *blob, const BlobLayout &L, hipStream_t s);

// routing
// One staging launch covers up to kIngestGroup chunks (passed by value).
struct IngestChunk {
  const int32_t *token_idx;
  const void *x;
  const int32_t *topk_id;
  const float *topk_w;
  int row0, n_rows, replica;
};
constexpr int kIngestGroup = 64;  // 3 KB of kernel arguments per staging launch
struct IngestGroup {
  IngestChunk c[kIngestGroup];
  int n;
};
hipError_t launch_ingest(const Arena &a, const IngestGroup &grp, int k, int E, int t_max,
                         size_t x_row_bytes, uint32_t *err, hipStream_t s);
// split_cu > 0 (bf16 batches with 256-row tiles): the scan may move each
// expert's last partial tile of at most 128 rows to 64-row remainder tiles
// when its makespan estimate for split_cu compute units and GEMM1's
// n_tiles_n 256-wide column tiles improves.  list2: the scan also lists,
// in the second list of each kind, the 128-row tiles (kListVar,
// batch_var_tiles) or the same tiles ordered by rows, most first
// (kListSorted, batch_stream_tiles).
enum : int { kListNone = 0, kListVar = 1, kListSorted = 2 };
hipError_t launch_route(const Arena &a, const Scratch &sc, int row0, int n_rows, int k, int E,
                        int align, int expected_pairs, int max_mpad, int max_tiles,
                        uint64_t fetched_mask, int x_dtype, int wk, int d, int split_cu,
                        int n_tiles_n, int list2, uint32_t *err, hipStream_t s);
// y_f32: the grouped outputs are float32 (bf16 weights), else bf16.
// skip_solo: the batch's GEMM2 wrote the output rows of tokens with one
// local pair (gemm2_writes_solo); the combine leaves them alone.
hipError_t launch_combine(const Arena &a, const Scratch &sc, int row0, int n_rows, int k, int d,
                          bool y_f32, bool skip_solo, float *out, hipStream_t s);

// grouped GEMMs over the tile lists of `which` (0 resident, 1 fetched) of a
// scratch whose lists hold list_cap tiles each; the grid covers grid_tiles
// M tiles with M tile `align` (the batch's row alignment), then, if
// split_tiles > 0, up to split_tiles 64-row remainder tiles
// gather (bf16 weights and rows only): GEMM1 reads the batch's input rows
// (arena rows from row0) in place through the permutation instead of a
// packed copy.  var: both GEMMs run the 128-row tile list instead.
// stream (batch_stream_tiles, the scan run with kListSorted): both GEMMs
// run the sorted tile list (launch_bf16_stream, launch_bf16_stream2).
hipError_t launch_gemm1(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        int split_tiles, int align, bool var, bool stream, const BlobTable &bt,
                        const BlobLayout &L, int wk, int d, int I, const Arena *gather, int row0,
                        int k, hipStream_t s);
// out (may be null): with gemm2_writes_solo, a grouped row whose token
// has no other local pair (Scratch::ydst) is written to that token's output
// row [d] float32 as the combine would write it, instead of to y.
hipError_t launch_gemm2(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        int split_tiles, int align, bool var, bool stream, const BlobTable &bt,
                        const BlobLayout &L, int wk, int d, int I, float *out, hipStream_t s);
// GEMM2 writes single-pair tokens' output rows itself, except in the 256-row
// bf16 tiles (batches of row alignment kBf16TileM, and their remainders).
inline bool gemm2_writes_solo(int wk, int align) { return wk != kWBf16 || align != kBf16TileM; }

}  // namespace cep
