// Routing, packing and combine kernels of the streamFFN path for gfx950.
//
// Appendix C, "Grouped FFN invocations": the rows selected from ready source
// lanes are grouped contiguously by expert, with per-expert offsets aligned
// to the GEMM tile and an inverse map back to (source replica, token, slot).
// Appendix C, "Output return and combine": each routed contribution is
// weighted by its routing coefficient exactly once and summed at the source
// token.
//
// All of these are HBM-bound scans; none of them is a contraction.
#include "common.h"

#include <type_traits>

#include <hip/hip_bf16.h>

#include <algorithm>

namespace cep {
namespace {

__device__ inline uint64_t lanemask_lt_popc(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// The lanes of this wave whose id equals this lane's (ids in [-1, 64); -1
// is key 127): one ballot per key bit, intersected.  Called with every lane
// of the wave active.
__device__ inline uint64_t same_id_lanes(int id) {
  const int key = id & 127;
  uint64_t m = __ballot(1);
#pragma unroll
  for (int b = 0; b < 7; ++b) {
    const uint64_t v = __ballot((key >> b) & 1);
    m &= ((key >> b) & 1) ? v : ~v;
  }
  return m;
}

// ---------------------------------------------------------------- ingest
// Stages the routing metadata of a group of ready chunks into the layer's
// arena (one entry per row, in submission order), so that a batch of whole
// chunks is a contiguous arena range; blockIdx.y names the chunk.  Ids
// outside [-1, E) are flagged and treated as remote; token slots outside
// [0, T_max) are flagged and their row dropped.
__global__ __launch_bounds__(256) void k_ingest(Arena a, IngestGroup grp, int k, int E, int t_max,
                                                size_t x_row_bytes, uint32_t *err) {
  const IngestChunk &c = grp.c[blockIdx.y];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= c.n_rows) return;
  const int row = c.row0 + i;
  // every load of the row first (one memory latency), the checks after; the
  // error flags are raised once per row
  const int t = c.token_idx[i];
  int idv[kMaxTopK];
  float wv[kMaxTopK];
#pragma unroll
  for (int s = 0; s < kMaxTopK; ++s) {
    if (s < k) {
      idv[s] = c.topk_id[(size_t)i * k + s];
      wv[s] = c.topk_w[(size_t)i * k + s];
    }
  }
  uint32_t bad = 0;
  int dst = -1;
  if (t >= 0 && t < t_max) dst = c.replica * t_max + t;
  else bad |= kErrBadToken;
  a.dst[row] = dst;
  a.xrow[row] = (const char *)c.x + (size_t)i * x_row_bytes;
  int n_local = 0;
#pragma unroll
  for (int s = 0; s < kMaxTopK; ++s) {
    if (s < k) {
      int id = idv[s];
      if (id < -1 || id >= E) {
        bad |= kErrBadId;
        id = -1;
      }
      if (dst < 0) id = -1;
      n_local += id >= 0;
      a.ids[(size_t)row * k + s] = id;
      a.w[(size_t)row * k + s] = wv[s];
    }
  }
  a.solo[row] = n_local == 1 ? dst : -1;
  if (bad) atomicOr(err, bad);
}

// ------------------------------------------------------------ histogram
// Block b counts the valid pairs of flat pairs [b*1024, (b+1)*1024) per
// expert.  Each wave resolves its 64 ids with seven ballots (the lanes
// sharing each lane's id); the lowest lane of each id adds the group's size.
__global__ __launch_bounds__(kRouteThreads) void k_route_count(const int32_t *__restrict__ ids,
                                                               int n_flat, int E,
                                                               int32_t *__restrict__ blk_cnt) {
  __shared__ int hist[kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63;
  if (tid < E) hist[tid] = 0;
  __syncthreads();
  const int base = blockIdx.x * kRoutePairs;
  constexpr int R = kRoutePairs / kRouteThreads;
  int idv[R];  // all loads first: one memory latency per block, not one per round
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int p = base + r * kRouteThreads + tid;
    idv[r] = p < n_flat ? ids[p] : -1;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int id = idv[r];
    const uint64_t m = same_id_lanes(id);
    if (id >= 0 && lane == __builtin_ctzll(m)) atomicAdd(&hist[id], (int)__popcll(m));
  }
  __syncthreads();
  if (tid < E) blk_cnt[blockIdx.x * E + tid] = hist[tid];
}

// ------------------------------------------------------------ tile plan
// Batch-wide quantities shared by both routing variants.
struct PlanArgs {
  int E, align, expected_pairs, max_mpad, max_tiles;
  uint64_t fetched_mask;
  int split_cu, n_tiles_n;
  // second list of each kind: kListVar each expert's 128-row tiles,
  // kListSorted the 64-row tiles ordered by rows, most first; kListNone none
  int list2;
  uint32_t *err;
};

struct PlanLds {
  int cnt[kMaxExperts], off[kMaxExperts + 1], pad[kMaxExperts + 1];
  int tile0[kMaxExperts], rtile0[kMaxExperts];
  int nfull[2];  // full tiles of resident / fetched experts (sorted list)
  int split;
};

// Given the per-expert totals in L.cnt (visible to the block), computes the
// unpadded and tile-aligned exclusive scans, the tile plan and the M-tile
// lists of the resident and the fetched experts, marks the padding rows of
// each expert's last tile (no pair), and publishes cnt / off / off_pad /
// n_tiles.  Called by all nthr threads of the block; ends with L.pad visible.
__device__ void plan_batch(const Scratch &sc, PlanLds &L, const PlanArgs &a, int tid, int nthr) {
  const int E = a.E, align = a.align;
  if (tid == 0) {
    // Remainder split: an expert's last partial tile of at most align/2 rows
    // can run as 64-row tiles (64 x 128 outputs, two workgroups per CU, about
    // a quarter of a full tile's time each) instead of a full tile.  Split
    // when that shortens the estimated makespan in full-tile rounds of
    // split_cu CUs; results are the same either way.
    int split = 0;
    if (a.split_cu > 0) {
      long long full = 0, kept = 0, rem = 0;
      for (int x = 0; x < E; ++x) {
        const int c = L.cnt[x], r = c % align;
        full += (c + align - 1) / align;
        kept += c / align + (r > align / 2 ? 1 : 0);
        rem += (r > 0 && r <= align / 2) ? (r + kBf16SmallTileM - 1) / kBf16SmallTileM : 0;
      }
      const long long wn = a.n_tiles_n, cu = a.split_cu;
      const long long rounds_full = (full * wn + cu - 1) / cu;
      const long long rounds_kept = (kept * wn + cu - 1) / cu;
      const long long rounds_rem = (rem * 2 * wn + 2 * cu - 1) / (2 * cu);  // quarter rounds
      split = rem > 0 && 4 * rounds_kept + rounds_rem < 4 * rounds_full;
    }
    L.split = split;
    int o = 0, op = 0;
    int t0[4] = {0, 0, 0, 0};
    int nfull[2] = {0, 0};
    for (int x = 0; x < E; ++x) {
      L.off[x] = o;
      L.pad[x] = op;
      const int which = (int)((a.fetched_mask >> x) & 1);
      const int c = L.cnt[x], r = c % align;
      const bool rem = split && r > 0 && r <= align / 2;
      L.tile0[x] = t0[2 * which];
      L.rtile0[x] = t0[2 * which + 1];
      t0[2 * which] += rem ? c / align : (c + align - 1) / align;
      t0[2 * which + 1] += rem                     ? (r + kBf16SmallTileM - 1) / kBf16SmallTileM
                           : a.list2 == kListVar    ? (c + kBf16VarTileM - 1) / kBf16VarTileM
                           : a.list2 == kListSorted ? (c + align - 1) / align
                                                    : 0;
      // sorted list: the kind's full tiles first, in expert order (rtile0 =
      // full tiles of the kind's earlier experts), then its partial tiles
      if (a.list2 == kListSorted) {
        L.rtile0[x] = nfull[which];
        nfull[which] += c / align;
      }
      o += c;
      op += (c + align - 1) / align * align;
    }
    L.off[E] = o;
    L.pad[E] = op;
    L.nfull[0] = nfull[0];
    L.nfull[1] = nfull[1];
    if (o != a.expected_pairs) atomicOr(a.err, kErrPairCount);
    bool over = op > a.max_mpad;
    for (int l = 0; l < 4; ++l) {
      over = over || t0[l] > a.max_tiles;
      sc.n_tiles[l] = min(t0[l], a.max_tiles);
    }
    if (over) atomicOr(a.err, kErrOverflow);
  }
  __syncthreads();
  if (tid <= E) {
    sc.off[tid] = L.off[tid];
    sc.off_pad[tid] = L.pad[tid];
  }
  if (tid < E) sc.cnt[tid] = L.cnt[tid];
  // padding rows of each expert's last tile carry no pair
  for (int i = tid; i < E * align; i += nthr) {
    const int x = i / align, r = L.pad[x] + L.cnt[x] + i % align;
    if (r < L.pad[x + 1] && r < a.max_mpad) {
      sc.perm[r] = -1;
      sc.ydst[r] = -1;
    }
  }
  if (tid < E) {
    const int which = (int)((a.fetched_mask >> tid) & 1);
    const int c = L.cnt[tid], r = c % align;
    const bool rem = L.split && r > 0 && r <= align / 2;
    Tile *list = sc.tiles + (size_t)(2 * which) * a.max_tiles;
    const int nt = rem ? c / align : (c + align - 1) / align;
    for (int q = 0; q < nt; ++q) {
      const int ti = L.tile0[tid] + q;
      const int row0 = L.pad[tid] + q * align;
      if (ti >= a.max_tiles || row0 + align > a.max_mpad) break;
      list[ti] = Tile{tid, row0, min(align, c - q * align), 0};
    }
    if (a.list2 == kListSorted) {
      // the second list holds the same tiles ordered by rows, most first:
      // the kind's full tiles in expert order, then its partial tiles by
      // rows, ties by expert
      Tile *slist = sc.tiles + (size_t)(2 * which + 1) * a.max_tiles;
      for (int q = 0; q < c / align; ++q) {
        const int ti = L.rtile0[tid] + q;
        const int row0 = L.pad[tid] + q * align;
        if (ti >= a.max_tiles || row0 + align > a.max_mpad) break;
        slist[ti] = Tile{tid, row0, align, 0};
      }
      if (r > 0) {
        int rank = 0;
        for (int x = 0; x < E; ++x) {
          const int rx = L.cnt[x] % align;
          rank += (int)((a.fetched_mask >> x) & 1) == which && rx > 0 &&
                  (rx > r || (rx == r && x < tid));
        }
        const int ti = L.nfull[which] + rank;
        const int row0 = L.pad[tid] + (c / align) * align;
        if (ti < a.max_tiles && row0 + align <= a.max_mpad) slist[ti] = Tile{tid, row0, r, 0};
      }
    }
    if (a.list2 == kListVar) {
      // the second list holds the 128-row tiles; a tile of more than 64
      // rows spans 128 rows of the expert's 64-aligned region
      Tile *vlist = sc.tiles + (size_t)(2 * which + 1) * a.max_tiles;
      for (int q = 0; q * kBf16VarTileM < c; ++q) {
        const int ti = L.rtile0[tid] + q;
        const int rows = min(kBf16VarTileM, c - q * kBf16VarTileM);
        const int row0 = L.pad[tid] + q * kBf16VarTileM;
        const int span = rows > kBf16VarTileM / 2 ? kBf16VarTileM : kBf16VarTileM / 2;
        if (ti >= a.max_tiles || row0 + span > a.max_mpad) break;
        vlist[ti] = Tile{tid, row0, rows, 0};
      }
    }
    if (rem) {
      Tile *rlist = sc.tiles + (size_t)(2 * which + 1) * a.max_tiles;
      const int base = L.pad[tid] + nt * align;
      for (int q = 0; q * kBf16SmallTileM < r; ++q) {
        const int ti = L.rtile0[tid] + q;
        const int row0 = base + q * kBf16SmallTileM;
        if (ti >= a.max_tiles || row0 + kBf16SmallTileM > a.max_mpad) break;
        rlist[ti] = Tile{tid, row0, min(kBf16SmallTileM, r - q * kBf16SmallTileM), 0};
      }
    }
  }
}

// ---------------------------------------------------- fused (one block)
// Histogram, scan, tile plan and stable scatter of a batch in one block of
// 16 waves, for batches whose ids fit in LDS: one coalesced pass stages the
// ids, then everything runs from LDS.  Wave w owns the contiguous flat pairs
// [w*span, (w+1)*span) and walks them in order, so a pair's grouped row is
// its expert's first row + the pairs of that expert in lower waves + those
// earlier in its own wave: the same stable order as the multi-block path.
constexpr int kFusedWaves = 16;

__global__ __launch_bounds__(64 * kFusedWaves) void k_route_fused(Arena a, Scratch sc, int row0,
                                                                  int n_flat, int k,
                                                                  PlanArgs pa) {
  __shared__ int s_ids[kFusedRoutePairs];
  __shared__ int wcnt[kFusedWaves][kMaxExperts];  // counts, then running rows
  __shared__ PlanLds L;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, E = pa.E;
  constexpr int NT = 64 * kFusedWaves;
  const int32_t *ids = a.ids + (size_t)row0 * k;
  for (int i = tid; i < kFusedWaves * kMaxExperts; i += NT) (&wcnt[0][0])[i] = 0;
#pragma unroll 8
  for (int i = tid; i < n_flat; i += NT) s_ids[i] = ids[i];
  __syncthreads();
  const int span = (n_flat + 64 * kFusedWaves - 1) / (64 * kFusedWaves) * 64;
  const int p0 = min(wid * span, n_flat), p1 = min(p0 + span, n_flat);
  for (int base = p0; base < p1; base += 64) {
    const int p = base + lane;
    const int id = p < p1 ? s_ids[p] : -1;
    const uint64_t m = same_id_lanes(id);
    if (id >= 0 && lane == __builtin_ctzll(m)) wcnt[wid][id] += (int)__popcll(m);
  }
  __syncthreads();
  if (tid < E) {
    int run = 0;
    for (int w = 0; w < kFusedWaves; ++w) {
      const int v = wcnt[w][tid];
      wcnt[w][tid] = run;
      run += v;
    }
    L.cnt[tid] = run;
  }
  __syncthreads();
  plan_batch(sc, L, pa, tid, NT);
  for (int base = p0; base < p1; base += 64) {
    const int p = base + lane;
    const int id = p < p1 ? s_ids[p] : -1;
    int pos = -1;
    // each id's lowest lane reads and advances the wave's running row; the
    // other lanes of that id take the old value from it
    const uint64_t m = same_id_lanes(id);
    const int leader = __builtin_ctzll(m);
    int run = 0;
    if (id >= 0 && lane == leader) {
      run = wcnt[wid][id];
      wcnt[wid][id] = run + (int)__popcll(m);
    }
    run = __shfl(run, leader);
    if (id >= 0) pos = L.pad[id] + run + (int)lanemask_lt_popc(m);
    if (pos >= pa.max_mpad) pos = -1;
    if (p < p1) {
      sc.pos_of[p] = pos;
      if (pos >= 0) {
        sc.perm[pos] = p;
        sc.wrow[pos] = a.w[(size_t)row0 * k + p];  // the row's routing coefficient
        sc.ydst[pos] = a.solo[row0 + p / k];
      }
    }
  }
}

// ------------------------------------------------------- scan + permute
// Same block decomposition as k_route_count.  Every block first reads all
// blocks' counts (thread t serves expert t % E over a contiguous range of
// blocks, group t / E) and scans them in LDS: the per-expert totals give the
// tile-aligned expert offsets, and the counts of the blocks before it give
// this block's first grouped row per expert.  One extra block (the last)
// publishes the tile plan (plan_batch) instead.  Then each pair's grouped row is that first row
// for its expert, plus pairs of that expert in earlier rounds of this block,
// in earlier waves of this round, and in lower lanes of this wave (stable in
// canonical order).  Writes the inverse map (grouped row of each pair), the
// permutation (pair of each grouped row) and each grouped row's routing
// coefficient.
__global__ __launch_bounds__(kRouteThreads) void k_route_scan_scatter(Arena a, Scratch sc, int row0,
                                                                      int n_flat, int k,
                                                                      int n_blocks, PlanArgs pa) {
  static_assert(kRouteThreads == 256, "one thread per (group, expert) of the count scan");
  __shared__ int s_part[kRouteThreads];  // [group][expert]: range sum, then exclusive prefix
  __shared__ PlanLds L;
  __shared__ int running[kMaxExperts];
  __shared__ int wave_cnt[kRouteThreads / 64][kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, E = pa.E;
  const int b = blockIdx.x;
  const int G = kRouteThreads / E, e = tid % E, grp = tid / E;
  const bool mine = grp < G;
  const int span = (n_blocks + G - 1) / G;
  {
    const int b0 = min(grp * span, n_blocks), b1 = min(b0 + span, n_blocks);
    if (mine) {
      int part = 0;
      for (int q = b0; q < b1; ++q) part += sc.blk_cnt[q * E + e];
      s_part[grp * E + e] = part;
    }
  }
  for (int i = tid; i < (kRouteThreads / 64) * kMaxExperts; i += kRouteThreads)
    (&wave_cnt[0][0])[i] = 0;
  __syncthreads();
  if (tid < E) {
    int run = 0;
    for (int q = 0; q < G; ++q) {
      const int v = s_part[q * E + tid];
      s_part[q * E + tid] = run;
      run += v;
    }
    L.cnt[tid] = run;
  }
  __syncthreads();
  if (b == n_blocks) {
    // the extra block publishes the tile plan while the others scatter
    plan_batch(sc, L, pa, tid, kRouteThreads);
    return;
  }
  {
    if (tid == 0) {
      int op = 0;
      for (int x = 0; x < E; ++x) {
        L.pad[x] = op;
        op += (L.cnt[x] + pa.align - 1) / pa.align * pa.align;
      }
    }
    __syncthreads();
  }
  if (tid < E) {
    // blocks before b: whole groups, then the blocks of b's group before it
    const int gb = b / span;
    int run = L.pad[tid] + s_part[gb * E + tid];
    for (int q = gb * span; q < b; ++q) run += sc.blk_cnt[q * E + tid];
    running[tid] = run;
  }
  __syncthreads();
  const int max_mpad = pa.max_mpad;
  const int32_t *ids = a.ids + (size_t)row0 * k;
  const int base = b * kRoutePairs;
  constexpr int R = kRoutePairs / kRouteThreads;
  int idv[R];  // all loads first: one memory latency per block, not one per round
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int p = base + r * kRouteThreads + tid;
    idv[r] = p < n_flat ? ids[p] : -1;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int p = base + r * kRouteThreads + tid;
    const int id = idv[r];
    const uint64_t m = same_id_lanes(id);
    const int rank = (int)lanemask_lt_popc(m);
    if (id >= 0 && lane == __builtin_ctzll(m)) wave_cnt[wid][id] = (int)__popcll(m);
    __syncthreads();
    int pos = -1;
    if (id >= 0) {
      pos = running[id] + rank;
      for (int w = 0; w < wid; ++w) pos += wave_cnt[w][id];
      if (pos >= max_mpad) pos = -1;
    }
    __syncthreads();
    if (tid < E) {
      int add = 0;
      for (int w = 0; w < kRouteThreads / 64; ++w) {
        add += wave_cnt[w][tid];
        wave_cnt[w][tid] = 0;
      }
      running[tid] += add;
    }
    __syncthreads();  // wave_cnt cleared before the next round writes it
    if (p < n_flat) sc.pos_of[p] = pos;
    if (pos >= 0) {
      sc.perm[pos] = p;
      sc.wrow[pos] = a.w[(size_t)row0 * k + p];  // the row's routing coefficient
      sc.ydst[pos] = a.solo[row0 + p / k];
    }
  }
}

// ----------------------------------------------------------------- pack
// Input rows reach their grouped rows converted (f32 -> bf16, k_pack_rows)
// or quantised to MXFP8 (e4m3 codes, one E8M0 scale per 32 channels, for
// e4m3 and MXFP4 weights, k_pack_tokens).  Padding rows (no pair) are left
// as they are: their outputs are never stored.  bf16 rows are not packed:
// the bf16 GEMM1 gathers them through the permutation.
constexpr int kPackRows = 8;

constexpr int kQuantPass = 8;  // 512-channel groups loaded per pass of a quantised row

__device__ inline void bf16x8_to_f32(const uint4 &u, float v[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
  }
}

__device__ inline uint2 e4m3x8(const float q[8]) {
  int lo = 0, hi = 0;
  lo = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], lo, false);
  lo = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], lo, true);
  hi = __builtin_amdgcn_cvt_pk_fp8_f32(q[4], q[5], hi, false);
  hi = __builtin_amdgcn_cvt_pk_fp8_f32(q[6], q[7], hi, true);
  return make_uint2((uint32_t)lo, (uint32_t)hi);
}

// 4 lanes x 8 channels = one 32-channel MX block: E8M0 scale
// 2^(floor(log2 amax) - 8), codes e4m3(x / scale) saturated at 448.  Returns
// the lane's eight codes; *code gets the block's scale code.
__device__ inline uint2 quant_mx8(const uint4 &in, int *code) {
  float v[8];
  bf16x8_to_f32(in, v);
  float amax = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[j]));
  amax = fmaxf(amax, __shfl_xor(amax, 1, 4));
  amax = fmaxf(amax, __shfl_xor(amax, 2, 4));
  *code = max((int)((__float_as_uint(amax) >> 23) & 0xff) - 8, 0);
  const int e = 127 - *code;
  float q[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) q[j] = fminf(fmaxf(ldexpf(v[j], e), -448.0f), 448.0f);
  return e4m3x8(q);
}

// f32 -> bf16 rows (one wave per grouped row).
__global__ __launch_bounds__(256) void k_pack_rows(Arena a, Scratch sc, int row0, int k, int E,
                                                   int d, int n_rows_pad) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int end = min(n_rows_pad, sc.off_pad[E]);
  for (int q = 0; q < kPackRows / 4; ++q) {
    const int pos = blockIdx.x * kPackRows + q * 4 + wid;
    if (pos >= end) return;
    const int p = sc.perm[pos];
    if (p < 0) continue;
    const float4 *s4 = (const float4 *)a.xrow[row0 + p / k];
    uint4 *d4 = (uint4 *)((char *)sc.xg + (size_t)pos * d * 2);
    for (int c = lane; c < d / 8; c += 64) {
      const float4 lo = s4[2 * c], hi = s4[2 * c + 1];
      union { __bf16 h[8]; uint4 u; } o;
      o.h[0] = (__bf16)lo.x; o.h[1] = (__bf16)lo.y; o.h[2] = (__bf16)lo.z; o.h[3] = (__bf16)lo.w;
      o.h[4] = (__bf16)hi.x; o.h[5] = (__bf16)hi.y; o.h[6] = (__bf16)hi.z; o.h[7] = (__bf16)hi.w;
      d4[c] = o.u;
    }
  }
}

// bf16 -> MXFP8 rows (e4m3 and MXFP4 weights), one wave per batch row: the
// row is read and quantised once and its codes and scales written to the
// grouped row of each of its local slots (a token averages 1.3 local slots
// on the skewed workloads, so reading per token rather than per pair saves a
// quarter of the reads).  A pass first loads up to kQuantPass 512-channel
// groups (eight channels per lane), then quantises them, so that many loads
// are in flight per wave.
__global__ __launch_bounds__(256) void k_pack_tokens(Arena a, Scratch sc, int row0, int n_rows,
                                                     int k, int d) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n_rows) return;  // uniform over the wave
  static_assert(kMaxTopK <= 64, "a row's slots fit one wave");
  const int ps = lane < k ? sc.pos_of[(size_t)i * k + lane] : -1;
  const uint64_t valid = __ballot(ps >= 0);
  if (valid == 0) return;
  const uint4 *s4 = (const uint4 *)a.xrow[row0 + i];
  uint8_t *xs_rows = sc.xs_rows;
  for (int p0 = 0; p0 < d; p0 += 512 * kQuantPass) {
    uint4 in[kQuantPass];
#pragma unroll
    for (int u = 0; u < kQuantPass; ++u) {
      const int c = p0 + u * 512 + lane * 8;
      in[u] = c < d ? s4[c / 8] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kQuantPass; ++u) {
      if (p0 + u * 512 >= d) break;  // uniform over the wave
      const int c = p0 + u * 512 + lane * 8;
      int code;
      const uint2 q = quant_mx8(in[u], &code);
      if (c >= d) continue;
      for (uint64_t m = valid; m; m &= m - 1) {
        const int pos = __shfl(ps, __builtin_ctzll(m));
        *(uint2 *)((uint8_t *)sc.xg + (size_t)pos * d + c) = q;
        // the wave's 16 scale bytes of this pass are contiguous here
        if ((lane & 3) == 0) xs_rows[(size_t)pos * sc.xs_pitch + c / kMxBlock] = (uint8_t)code;
      }
    }
  }
}

// The packed rows' scale bytes, row-major in xs_rows, moved to the GEMM's
// layout (mx_row_scale_offset): for a 128-row group and a 32-channel block
// the 128 bytes are one contiguous run, byte (r % 16) * 8 + r / 16 for row r
// of the group.  One block per (128-row group, 256 blocks): the rows come
// into LDS with 16-byte loads and leave as 4-byte words of the runs.  (The
// pack writing them there directly scatters single bytes: a position's
// scales are 192 bytes in 192 different runs at d = 6144.)
constexpr int kScaleCols = 256;                 // 32-channel blocks per LDS tile
constexpr int kScaleLdsPitch = kScaleCols + 4;  // rows 16 apart fall in distinct banks

__global__ __launch_bounds__(256) void k_scale_layout(Scratch sc, int nb) {
  __shared__ uint8_t tile[128 * kScaleLdsPitch];
  const int g = blockIdx.x, b0 = blockIdx.y * kScaleCols;
  const int nbt = min(kScaleCols, nb - b0);            // blocks of this tile
  const int nq = (min(b0 + kScaleCols, sc.xs_pitch) - b0) / 16;  // 16-byte chunks a row
  const uint8_t *src = sc.xs_rows + (size_t)g * 128 * sc.xs_pitch + b0;
  for (int q = threadIdx.x; q < 128 * nq; q += blockDim.x) {
    const int r = q / nq, ch = q % nq;
    const uint4 v = *(const uint4 *)(src + (size_t)r * sc.xs_pitch + ch * 16);
    uint32_t *t = (uint32_t *)&tile[r * kScaleLdsPitch + ch * 16];
    t[0] = v.x; t[1] = v.y; t[2] = v.z; t[3] = v.w;
  }
  __syncthreads();
  uint8_t *xs = (uint8_t *)sc.xs;
  for (int q = threadIdx.x; q < nbt * 32; q += blockDim.x) {
    const int bl = q >> 5, w = q & 31, b = b0 + bl;
    uint32_t word = 0;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int p = 4 * w + t, r = (p & 7) * 16 + (p >> 3);
      word |= (uint32_t)tile[r * kScaleLdsPitch + bl] << (8 * t);
    }
    *(uint32_t *)(xs + mx_row_scale_offset(g * 128, b, sc.s_ld) + 4 * w) = word;
  }
}

// --------------------------------------------------------------- combine
// One block per batch row: out[dst] = sum over its valid slots, in slot
// order, of the grouped output rows (already scaled by their coefficient;
// float32, or bf16 with YF32 false), accumulated in float32 from +0.
// The row's valid slot positions are gathered once into LDS; each thread
// then issues the loads of all its columns before summing, slot by slot.
// skip_solo: GEMM2 has written the rows with exactly one local pair itself
// (the same value: +0 plus the one grouped output); they are skipped.
constexpr int kCombineCols = 4;  // float4 columns per thread per pass

template <bool YF32>
__global__ __launch_bounds__(256) void k_combine(Arena a, Scratch sc, int row0, int k, int d,
                                                 bool skip_solo, float *__restrict__ out) {
  __shared__ int s_pos[kMaxTopK];
  __shared__ int s_n;
  const int i = blockIdx.x;
  // the row's slot positions load beside its destination (one memory
  // latency, not two); lane s of wave 0 holds slot s, and a ballot keeps the
  // valid ones in slot order
  static_assert(kMaxTopK <= 64, "a row's slots fit one wave");
  int ps = -1;
  if (threadIdx.x < k) ps = sc.pos_of[(size_t)i * k + threadIdx.x];
  const int dst = a.dst[row0 + i];
  const int solo = skip_solo ? a.solo[row0 + i] : -1;
  if (dst < 0) return;  // the same for the whole block
  if (threadIdx.x < 64) {
    const uint64_t m = __ballot(ps >= 0);
    if (ps >= 0) s_pos[lanemask_lt_popc(m)] = ps;
    if (threadIdx.x == 0) s_n = (int)__popcll(m);
  }
  __syncthreads();
  const int n = s_n, d4 = d / 4;
  // a row whose one local pair has a grouped row: GEMM2 wrote it
  if (solo >= 0 && n == 1) return;
  float4 *o = (float4 *)(out + (size_t)dst * d);
  for (int c0 = threadIdx.x; c0 < d4; c0 += blockDim.x * kCombineCols) {
    float4 acc[kCombineCols];
#pragma unroll
    for (int u = 0; u < kCombineCols; ++u) acc[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (YF32) {
      const float4 *y = (const float4 *)sc.y;
      for (int j = 0; j < n; ++j) {
        const float4 *yr = y + (size_t)s_pos[j] * d4;
        float4 v[kCombineCols];
#pragma unroll
        for (int u = 0; u < kCombineCols; ++u) {
          const int c = c0 + u * blockDim.x;
          v[u] = c < d4 ? yr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < kCombineCols; ++u) {
          acc[u].x += v[u].x;
          acc[u].y += v[u].y;
          acc[u].z += v[u].z;
          acc[u].w += v[u].w;
        }
      }
    }
    const uint2 *y = (const uint2 *)sc.y;  // four bf16 per column group
    for (int j = 0; !YF32 && j < n; ++j) {
      const uint2 *yr = y + (size_t)s_pos[j] * d4;
      uint2 v[kCombineCols];
#pragma unroll
      for (int u = 0; u < kCombineCols; ++u) {
        const int c = c0 + u * blockDim.x;
        v[u] = c < d4 ? yr[c] : make_uint2(0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < kCombineCols; ++u) {  // bf16 -> f32: the upper half of the word
        acc[u].x += __uint_as_float(v[u].x << 16);
        acc[u].y += __uint_as_float(v[u].x & 0xffff0000u);
        acc[u].z += __uint_as_float(v[u].y << 16);
        acc[u].w += __uint_as_float(v[u].y & 0xffff0000u);
      }
    }
#pragma unroll
    for (int u = 0; u < kCombineCols; ++u) {
      const int c = c0 + u * blockDim.x;
      if (c < d4) o[c] = acc[u];
    }
  }
}

// ------------------------------------------------------- weight packing
// out[map(c)][r] = in[r][c] for a [rows][cols] matrix, 64x64 tiles via LDS.
// MAP 0: identity; MAP 1: gate half of the W1 interleave; MAP 2: up half.
// e4m3 outputs are row-major [cols][rows]; bf16 outputs are stored in the
// blocked layout of bf16_block_index (16 KB blocks of 128 rows x 64 K).
template <typename TI, typename TO, int MAP>
__global__ __launch_bounds__(256) void k_transpose(const TI *__restrict__ in, TO *__restrict__ out,
                                                   int rows, int cols) {
  __shared__ TO tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int j = ty; j < 64; j += 4) {
    const int r = r0 + j, c = c0 + tx;
    if (r < rows && c < cols) tile[j][tx] = (TO)in[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int j = ty; j < 64; j += 4) {
    const int c = c0 + j, r = r0 + tx;
    if (r < rows && c < cols) {
      int oc = c;
      if (MAP == 1) oc = (c / kInterleave) * (2 * kInterleave) + c % kInterleave;
      if (MAP == 2) oc = (c / kInterleave) * (2 * kInterleave) + kInterleave + c % kInterleave;
      if constexpr (std::is_same<TO, __bf16>::value)
        out[bf16_block_index(oc, r, rows)] = tile[tx][j];
      else
        out[(size_t)oc * rows + r] = tile[tx][j];
    }
  }
}

__global__ void k_pack_scales(const float *sg, const float *su, const float *sd, int d, int I,
                              float *s1, float *s2) {
  const int kb_n = d / 128, ib_n = I / 128;
  const int n1 = (2 * I / kInterleave) * kb_n;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < n1 + kb_n * ib_n;
       t += gridDim.x * blockDim.x) {
    if (t < n1) {
      // S1[g][kb] = scale of the gate (g even) or up (g odd) block holding
      // original column (g/2)*32, at k-block kb.  s_gate is [d/128][I/128].
      const int g = t / kb_n, kb = t % kb_n;
      const int col = (g / 2) * kInterleave;
      s1[t] = ((g & 1) ? su : sg)[kb * ib_n + col / 128];
    } else {
      // S2[nb][kb] = s_down[kb][nb]; s_down is [I/128][d/128]
      const int u = t - n1;
      const int nb = u / ib_n, kb = u % ib_n;
      s2[u] = sd[kb * kb_n + nb];
    }
  }
}

// MXFP4 experts.  W1p row n' is row (n'/64)*32 + n'%32 of the gate
// (n'/32 even) or up (odd) codes [I][d/2]: the caller's layout is already K
// packed, so packing is a row gather, one block per row.
// Row n of packed e2m1 weights into mx_block_index order; interleave (W1p):
// row n is gathered from gate (wg) or up (wu) like the bf16 W1p, otherwise
// (W2p) it is row n of wg.
__global__ __launch_bounds__(256) void k_pack_mx_rows(const uint8_t *wg, const uint8_t *wu,
                                                      int row_bytes, int interleave,
                                                      uint8_t *dst) {
  const int n = blockIdx.x;
  const uint8_t *src =
      interleave ? (((n / kInterleave) & 1) ? wu : wg) +
                       (size_t)((n / (2 * kInterleave)) * kInterleave + n % kInterleave) * row_bytes
                 : wg + (size_t)n * row_bytes;
  const uint4 *s4 = (const uint4 *)src;
  for (int c = threadIdx.x; c < row_bytes / 16; c += blockDim.x)
    *(uint4 *)(dst + mx_block_index(n, c * 16, row_bytes)) = s4[c];
}

// E8M0 scales [N][K/32] (row n of B) into mx_weight_scale_offset order;
// interleave: N = 2I rows gathered from gate (sa) and up (sb) like W1p.
__global__ void k_pack_mx_scales(const uint8_t *sa, const uint8_t *sb, int N, int K,
                                 int interleave, uint8_t *dst) {
  const int nblk = K / kMxBlock;
  const size_t total = (size_t)N * nblk;
  for (size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (size_t)gridDim.x * blockDim.x) {
    const int n = (int)(t / nblk), b = (int)(t % nblk);
    const uint8_t *src = sa;
    int row = n;
    if (interleave) {
      src = ((n / kInterleave) & 1) ? sb : sa;
      row = (n / (2 * kInterleave)) * kInterleave + n % kInterleave;
    }
    dst[mx_weight_scale_offset(n, b, K)] = src[(size_t)row * nblk + b];
  }
}

}  // namespace

// ================================================================ launchers
hipError_t launch_pack_mx(const uint8_t *wg, const uint8_t *wu, const uint8_t *wd,
                          const uint8_t *sg, const uint8_t *su, const uint8_t *sd, int d, int I,
                          uint8_t *blob, const BlobLayout &L, hipStream_t s) {
  hipLaunchKernelGGL(k_pack_mx_rows, dim3(2 * I), dim3(256), 0, s, wg, wu, d / 2, 1,
                     blob + L.w1_off);
  hipLaunchKernelGGL(k_pack_mx_rows, dim3(d), dim3(256), 0, s, wd, (const uint8_t *)nullptr, I / 2,
                     0, blob + L.w2_off);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pack_mx_scales, dim3(256), dim3(256), 0, s, sg, su, 2 * I, d, 1,
                     blob + L.s1_off);
  hipLaunchKernelGGL(k_pack_mx_scales, dim3(256), dim3(256), 0, s, sd, (const uint8_t *)nullptr,
                     d, I, 0, blob + L.s2_off);
  return hipGetLastError();
}

hipError_t launch_pack_w1(const void *wg, const void *wu, int w_dtype, int d, int I,
                          uint8_t *dst, hipStream_t s) {
  dim3 grid((I + 63) / 64, (d + 63) / 64);
  if (w_dtype == 2) {
    hipLaunchKernelGGL((k_transpose<uint8_t, uint8_t, 1>), grid, dim3(256), 0, s,
                       (const uint8_t *)wg, dst, d, I);
    hipLaunchKernelGGL((k_transpose<uint8_t, uint8_t, 2>), grid, dim3(256), 0, s,
                       (const uint8_t *)wu, dst, d, I);
  } else if (w_dtype == 1) {
    hipLaunchKernelGGL((k_transpose<__bf16, __bf16, 1>), grid, dim3(256), 0, s,
                       (const __bf16 *)wg, (__bf16 *)dst, d, I);
    hipLaunchKernelGGL((k_transpose<__bf16, __bf16, 2>), grid, dim3(256), 0, s,
                       (const __bf16 *)wu, (__bf16 *)dst, d, I);
  } else {
    hipLaunchKernelGGL((k_transpose<float, __bf16, 1>), grid, dim3(256), 0, s,
                       (const float *)wg, (__bf16 *)dst, d, I);
    hipLaunchKernelGGL((k_transpose<float, __bf16, 2>), grid, dim3(256), 0, s,
                       (const float *)wu, (__bf16 *)dst, d, I);
  }
  return hipGetLastError();
}

hipError_t launch_pack_w2(const void *wd, int w_dtype, int d, int I, uint8_t *dst,
                          hipStream_t s) {
  dim3 grid((d + 63) / 64, (I + 63) / 64);
  if (w_dtype == 2)
    hipLaunchKernelGGL((k_transpose<uint8_t, uint8_t, 0>), grid, dim3(256), 0, s,
                       (const uint8_t *)wd, dst, I, d);
  else if (w_dtype == 1)
    hipLaunchKernelGGL((k_transpose<__bf16, __bf16, 0>), grid, dim3(256), 0, s,
                       (const __bf16 *)wd, (__bf16 *)dst, I, d);
  else
    hipLaunchKernelGGL((k_transpose<float, __bf16, 0>), grid, dim3(256), 0, s,
                       (const float *)wd, (__bf16 *)dst, I, d);
  return hipGetLastError();
}

hipError_t launch_pack_scales(const float *sg, const float *su, const float *sd, int d, int I,
                              float *s1, float *s2, hipStream_t s) {
  hipLaunchKernelGGL(k_pack_scales, dim3(64), dim3(256), 0, s, sg, su, sd, d, I, s1, s2);
  return hipGetLastError();
}

hipError_t launch_ingest(const Arena &a, const IngestGroup &grp, int k, int E, int t_max,
                         size_t x_row_bytes, uint32_t *err, hipStream_t s) {
  int rows = 0;
  for (int i = 0; i < grp.n; ++i) rows = std::max(rows, grp.c[i].n_rows);
  if (grp.n <= 0 || rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_ingest, dim3((rows + 255) / 256, grp.n), dim3(256), 0, s, a, grp, k, E,
                     t_max, x_row_bytes, err);
  return hipGetLastError();
}

hipError_t launch_route(const Arena &a, const Scratch &sc, int row0, int n_rows, int k, int E,
                        int align, int expected_pairs, int max_mpad, int max_tiles,
                        uint64_t fetched_mask, int x_dtype, int wk, int d, int split_cu,
                        int n_tiles_n, int list2, uint32_t *err, hipStream_t s) {
  const int n_flat = n_rows * k;
  const int nb = (n_flat + kRoutePairs - 1) / kRoutePairs;
  if (nb == 0) return hipSuccess;
  const PlanArgs pa{E, align, expected_pairs, max_mpad, max_tiles, fetched_mask, split_cu,
                    n_tiles_n, list2, err};
  if (n_flat <= kFusedRoutePairs) {
    hipLaunchKernelGGL(k_route_fused, dim3(1), dim3(64 * kFusedWaves), 0, s, a, sc, row0,
                       n_flat, k, pa);
  } else {
    hipLaunchKernelGGL(k_route_count, dim3(nb), dim3(kRouteThreads), 0, s,
                       a.ids + (size_t)row0 * k, n_flat, E, sc.blk_cnt);
    hipLaunchKernelGGL(k_route_scan_scatter, dim3(nb + 1), dim3(kRouteThreads), 0, s, a, sc,
                       row0, n_flat, k, nb, pa);
  }
  // grouped rows: at most every pair plus one partial tile per expert
  const long long bound = ((long long)(expected_pairs + align - 1) / align + E) * align;
  const int n_pad = (int)std::min<long long>(bound, max_mpad);
  if (wk == kWMx || wk == kWFp8) {
    hipLaunchKernelGGL(k_pack_tokens, dim3((n_rows + 3) / 4), dim3(256), 0, s, a, sc, row0, n_rows,
                       k, d);
    const int nb = d / kMxBlock;
    hipLaunchKernelGGL(k_scale_layout, dim3((n_pad + 127) / 128, (nb + kScaleCols - 1) / kScaleCols),
                       dim3(256), 0, s, sc, nb);
  }
  else if (x_dtype == 0)
    hipLaunchKernelGGL(k_pack_rows, dim3((n_pad + kPackRows - 1) / kPackRows), dim3(256), 0, s, a,
                       sc, row0, k, E, d, n_pad);
  // bf16 rows with bf16 weights: GEMM1 reads them in place
  return hipGetLastError();
}

hipError_t launch_combine(const Arena &a, const Scratch &sc, int row0, int n_rows, int k, int d,
                          bool y_f32, bool skip_solo, float *out, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  if (y_f32)
    hipLaunchKernelGGL(k_combine<true>, dim3(n_rows), dim3(256), 0, s, a, sc, row0, k, d,
                       skip_solo, out);
  else
    hipLaunchKernelGGL(k_combine<false>, dim3(n_rows), dim3(256), 0, s, a, sc, row0, k, d,
                       skip_solo, out);
  return hipGetLastError();
}

}  // namespace cep
