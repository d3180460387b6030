// bf16 grouped expert GEMMs for gfx950 (CDNA4) MFMA.
//
// Appendix C, "Grouped FFN invocations": within an invocation the two expert
// GEMMs and the intervening activation run in stream order.  GEMM1 computes
// the gate and up projections of every grouped row against its expert's
// weights and applies SwiGLU in the epilogue; GEMM2 computes the down
// projection and scales each row by its routing coefficient (the one place
// the coefficient is applied).
//
// One kernel template, three uses:
//   large batches: 256 x 256 tile, K steps of 32 through 4 LDS stages, one
//     workgroup per CU -- MFMA-bound, each 16-byte LDS read feeds 4 MFMAs;
//   small batches (few rows per expert): 64 x 128 tile, K steps of 64 through
//     3 stages, two workgroups per CU -- weight-streaming (HBM) bound, sized
//     for many weight bytes in flight per CU;
//   mid-size batches (VAR): 128 x 128 tiles whose last tile per expert may be
//     a 64-row half (it loads and multiplies its first 64 rows only), the
//     weights three stages deep and the rows two, so that two workgroups
//     still fit a CU: a hot expert streams its weights once per 128 rows;
//   weight-streaming batches (LIN): the small tile's schedule over 64-row
//     tiles listed by rows, one work item per workgroup in list order, each
//     wave loading only its 8-row segments that hold rows.
// All accumulate each output over K in the same order (ascending 16-wide
// steps of v_mfma_f32_32x32x16_bf16), so a row's result does not depend on
// which tile its batch used.  With bf16 token rows GEMM1 runs as GATHER: its
// A rows are the batch's input rows themselves, found through the
// permutation (the layout transform's row pack reduced to an address lookup).
#include "gemm_common.h"

#include <algorithm>
#include <type_traits>
#include <utility>

namespace cep {
namespace {

template <int V>
using ic = std::integral_constant<int, V>;
template <class F, int... I>
__device__ inline void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(ic<I>{}), ...);
}
// f(ic<0>{}), ..., f(ic<N-1>{}): indices that stay compile-time constants
template <int N, class F>
__device__ inline void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// BM x BN output tile, NW waves as WGM x (NW/WGM), each wave owning a
// (BM/WGM) x (BN/(NW/WGM)) block of 32x32 MFMA fragments (for SwiGLU a
// wave's columns hold whole gate/up pairs of 32).  K advances in steps of BK through a ring of STAGES
// LDS buffers filled by direct global->LDS loads (no staging registers), one
// barrier per step.  An LDS row holds BK bf16 = CH 16-byte chunks; chunk c of
// row r lives at slot c ^ swz(r), with swz chosen so that sixteen consecutive
// rows read at one chunk (what one LDS cycle serves of an MFMA operand read)
// cover all sixteen 16-byte slots of a 256-byte bank window.  A load
// instruction fills 64 consecutive slots, so each lane fetches the global
// chunk that belongs in its slot; weight chunks come from the 1 KB blocks of
// the packed layout, so one load reads one block (BK 32) or two halves.
//
// Two schedules.  PIPE (MFMA-bound tile): each 16-wide sub-step multiplies
// fragments read during the previous sub-step, so LDS latency hides behind
// the MFMAs; loads run STAGES-2 steps ahead.  Otherwise (weight-streaming
// tile): fragments are read right before their MFMAs and loads run STAGES-1
// steps ahead, which keeps more weight bytes in flight per LDS byte.
template <int BM, int BN, int BK, int STAGES, int OCC, bool PIPE, bool SWIGLU, int WGM = 2,
          int NW = 4, int GM = kGroupM, bool GATHER = false, bool VAR = false, int ASTG = 0,
          bool LIN = false>
__global__ __launch_bounds__(64 * NW, OCC) void k_gemm_bf16(GemmArgs g) {
  static_assert(BK == 32 || BK == 64, "LDS swizzle covers 4 or 8 chunks per row");
  static_assert(!VAR || (!PIPE && WGM == 2 && BM == 128), "VAR: 128-row tile, two wave rows");
  static_assert(ASTG == 0 || (ASTG == 2 && !PIPE && STAGES >= 3), "A ring: all stages or two");
  constexpr int AS = ASTG ? ASTG : STAGES;  // depth of the A ring (B: STAGES)
  static_assert(STAGES >= 3 && STAGES <= 8, "wait counts below");
  constexpr int CH = BK / 8;                  // 16-byte chunks per LDS row
  constexpr int RPS = 1024 / (BK * 2);        // rows per 1 KB load segment
  constexpr int SH = CH == 4 ? 2 : 1;         // swz(r) = (r >> SH) & (CH - 1)
  constexpr int WGN = NW / WGM;  // waves along M x along N
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int A_LD = BM * BK * 2 / 1024 / NW, B_LD = BN * BK * 2 / 1024 / NW;  // per wave
  static_assert(A_LD * NW * 1024 == BM * BK * 2 && B_LD * NW * 1024 == BN * BK * 2,
                "loads split evenly over the waves");
  // SwiGLU: a wave's columns hold whole gate/up pairs of 32, or (XCH, two
  // wave columns of 32) wave column 0 holds the gate and 1 the up columns
  // and they meet in LDS after the K loop
  constexpr bool XCH = SWIGLU && !PIPE && WGN == 2 && WN == 32;
  static_assert(!SWIGLU || XCH || (BN / WGN) % 64 == 0,
                "a wave's columns hold whole gate/up pairs");
  constexpr int PER = A_LD + B_LD;            // loads per thread per step
  // PIPE workgroups are persistent (one per CU) and take every grid-th work
  // item of their XCD's share: the next tile's first loads then start while
  // the previous tile's output stores drain.  Others take one work item.
  const int n_live = *g.n_tiles;
  for (int it = 0;; ++it) {
  int mt, nt;
  if constexpr (LIN) {
    // work item = workgroup id, tile-major (every column slice of tile 0
    // first): the hardware starts the items in list order
    if (it > 0) return;
    const int ntn = g.N / BN, L = blockIdx.x;
    if (L >= n_live * ntn) return;
    mt = L / ntn;
    nt = L % ntn;
  } else if (!work_item<GM, PIPE>(it, n_live, g.N / BN, &mt, &nt)) {
    return;
  }
  const Tile t = g.tiles[mt];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid / WGN, wn = wid % WGN;
  const int K = g.K, nk = K / BK;
  const char *Ag = GATHER ? nullptr : (const char *)(g.A + (size_t)t.row0 * K * 2);
  const char *Bg = (const char *)(blob_of(g.bt, t.expert) + g.b_off);

  __shared__ u32x4 sA[AS][BM * CH];
  __shared__ u32x4 sB[STAGES][BN * CH];
  // GEMM2 of the non-PIPE tiles: direct output rows (GemmArgs::ydst; the
  // 256-row tile's epilogue has no registers to spare and gets none)
  const bool direct = !SWIGLU && !PIPE && g.ydst;

  // Lane l of a load fills slot l of a 1 KB segment (RPS rows x CH chunks):
  // row seg*RPS + l/CH, slot l%CH, which holds chunk (l%CH) ^ swz(row).  The
  // swizzle uses the full row index (with 8 chunks per row, swz depends on
  // the segment's position too).
  const int seg_row = lane / CH;
#define CEP_LANE_OFF(seg)                                                           \
  ((uint32_t)((seg) * RPS + seg_row) * K * 2 +                                      \
   (uint32_t)(((lane % CH) ^ ((((seg) * RPS + seg_row) >> SH) & (CH - 1))) * 16))
  // B (packed weights, bf16_block_index layout): the byte offset of the
  // lane's chunk of segment seg in K step 0; step kt adds kt * BK/32 times
  // the layout's 8 KB per 32 K.
  auto b_lane_off = [&](int seg) -> size_t {
    const int tr = seg * RPS + seg_row, n = nt * BN + tr;
    const int kc = ((lane % CH) ^ ((tr >> SH) & (CH - 1))) * 8;  // K element of the chunk
    return bf16_block_index(n, kc, K) * 2;
  };
  // GATHER: each lane's A rows are fixed for the whole K loop, so their
  // input-row addresses (plus the lane's chunk) are looked up once.  NAL_
  // (the A loads per wave in the current schedule) is defined in each scope
  // that expands these macros.
#define CEP_AROWS(arow_)                                                            \
  if constexpr (GATHER) {                                                           \
    _Pragma("unroll") for (int i = 0; i < NAL_; ++i) {                              \
      const int r = (wid * SEGW_ + i) * RPS + seg_row;                              \
      const int p = g.perm[t.row0 + r];                                             \
      arow_[i] = (const char *)g.xrow[g.arow0 + (p >= 0 ? p / g.k : 0)] +           \
                 ((lane % CH) ^ ((r >> SH) & (CH - 1))) * 16;                       \
    }                                                                               \
  }
#define CEP_DMA_A(kt)                                                               \
  {                                                                                 \
    const int buf_ = (kt) % AS;                                                     \
    _Pragma("unroll") for (int i = 0; i < NAL_; ++i) {                              \
      const int seg = wid * SEGW_ + i;                                              \
      dma16(GATHER ? arow[i] + (size_t)(kt) * BK * 2                                \
                   : Ag + (size_t)(kt) * BK * 2 + CEP_LANE_OFF(seg),                \
            __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf_][seg * 64])));       \
    }                                                                               \
  }
#define CEP_DMA_B(kt)                                                               \
  {                                                                                 \
    const int buf_ = (kt) % STAGES;                                                 \
    _Pragma("unroll") for (int i = 0; i < B_LD; ++i) {                              \
      const int seg = wid * B_LD + i;                                               \
      dma16(Bg + b_lane_off(seg) + (size_t)(kt) * (BK / 32) * kBf16BlockStepBytes,                 \
            __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf_][seg * 64])));       \
    }                                                                               \
  }
#define CEP_DMA_STAGE(kt) { CEP_DMA_A(kt) CEP_DMA_B(kt) }

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

  // First row of A fragment i of this wave.  VAR interleaves the waves'
  // fragments (i*64 + wm*32) so that a half tile's 64 rows are fragment 0
  // of every wave.  Every fragment row r = base + lane%32 has
  // swz(r) == swz(lane % 32) because the bases are multiples of 32.
  auto frow = [&](int i) { return VAR ? i * (BM / FM) + wm * 32 : wm * WM + i * 32; };
  const int rsw = ((lane & 31) >> SH) & (CH - 1);
#define CEP_LOAD_FRAG(fa_, fb_, abuf_, bbuf_, kk_, nfa_)                            \
  {                                                                                 \
    const int slot_ = ((kk_) * 2 + (lane >> 5)) ^ rsw;                              \
    _Pragma("unroll") for (int i = 0; i < (nfa_); ++i) fa_[i] = __builtin_bit_cast( \
        bf16x8, sA[abuf_][(frow(i) + (lane & 31)) * CH + slot_]);                   \
    _Pragma("unroll") for (int j = 0; j < FN; ++j) fb_[j] = __builtin_bit_cast(     \
        bf16x8, sB[bbuf_][(wn * WN + j * 32 + (lane & 31)) * CH + slot_]);          \
  }

  constexpr int KK = BK / 16;
  static_assert(!PIPE || KK % 2 == 0, "fragment double buffer alternates per sub-step");
  // a VAR tile of at most BM/2 rows loads and multiplies its first half only
  const bool half = VAR && t.rows <= BM / 2;
  if constexpr (PIPE) {
    constexpr int NAL_ = A_LD, SEGW_ = A_LD;
    const char *arow[NAL_];
    CEP_AROWS(arow)
    // Stage s is issued at the barrier of step s - STAGES + 1 (the prologue
    // below issues stages 0 .. STAGES-2), into the buffer of stage s - STAGES,
    // whose last fragment reads completed before the MFMAs of step
    // s - STAGES.
    //
    // Every step issues one stage of loads, so the vmcnt waits are constants
    // and the loop body is one basic block: steps past the end reload the
    // last K step into a buffer nobody reads again.  Sub-steps 0 .. KK-2 of
    // step kt read the fragments of the next sub-step, then multiply the
    // current ones; sub-step 0 also issues the loads of stage kt+STAGES-1
    // into the buffer of step kt-1, which every wave stopped reading before
    // the previous step's barrier.  The last sub-step multiplies while it
    // waits for stage kt+1, passes the barrier and reads the first fragments
    // of kt+1.  Loads, waits, the barrier and reads sit between MFMAs, so the
    // matrix pipe always has the next MFMA queued, and the LDS-read wait
    // before an MFMA never counts the reads issued after it.
    bf16x8 fa[2][FM], fb[2][FN];
    constexpr int NM = FM * FN;   // MFMAs per sub-step
    constexpr int NR = FM + FN;   // fragment reads per sub-step
    constexpr int PL = (KK - 1) & 1, QL = PL ^ 1;
    static_assert(NM >= 2 + PER + NR / 2 && NR % 2 == 0,
                  "enough MFMAs to spread the last sub-step over");
    auto mfma_one = [&](auto p_c, auto idx_c) {
      constexpr int p = decltype(p_c)::value, idx = decltype(idx_c)::value;
      constexpr int i = idx / FN, j = idx % FN;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
    };
    auto read_one = [&](auto q_c, int buf, auto idx_c) {
      constexpr int q = decltype(q_c)::value, idx = decltype(idx_c)::value;
      const int slot = (lane >> 5) ^ rsw;  // K sub-step 0
      if constexpr (idx < FM)
        fa[q][idx] = __builtin_bit_cast(bf16x8, sA[buf][(frow(idx) + (lane & 31)) * CH + slot]);
      else
        fb[q][idx - FM] = __builtin_bit_cast(
            bf16x8, sB[buf][(wn * WN + (idx - FM) * 32 + (lane & 31)) * CH + slot]);
    };
    // load piece idx of K step ks into LDS buffer buf: idx < A_LD is an A
    // segment, the rest B segments
    auto dma_one = [&](int ks, int buf, auto idx_c) {
      constexpr int idx = decltype(idx_c)::value;
      if constexpr (idx < A_LD) {
        const int seg = wid * A_LD + idx;
        dma16(GATHER ? arow[idx] + (size_t)ks * BK * 2
                     : Ag + (size_t)ks * BK * 2 + CEP_LANE_OFF(seg),
              __builtin_amdgcn_readfirstlane(lds_offset(&sA[buf][seg * 64])));
      } else {
        const int seg = wid * B_LD + (idx - A_LD);
        dma16(Bg + b_lane_off(seg) + (size_t)ks * (BK / 32) * kBf16BlockStepBytes,
              __builtin_amdgcn_readfirstlane(lds_offset(&sB[buf][seg * 64])));
      }
    };
    // sub-steps 0 .. KK-2 of the step in buffer cur
    // sub-steps 0 .. KK-2 of the step in buffer cur; with DMA, sub-step 0
    // also issues the loads of K step ks into buffer kbuf between its MFMAs
    auto early_subs = [&](int cur, auto dma_c, int ks, int kbuf) {
      constexpr bool DMA = decltype(dma_c)::value;
#pragma unroll
      for (int kk = 0; kk + 1 < KK; ++kk) {
        const int p = kk & 1, q = p ^ 1;
        CEP_LOAD_FRAG(fa[q], fb[q], cur, cur, kk + 1, FM);
        __builtin_amdgcn_sched_barrier(0);
        if (DMA && kk == 0) {
          static_for<PER>([&](auto d) {
            if (p == 0) mfma_one(ic<0>{}, d); else mfma_one(ic<1>{}, d);
            __builtin_amdgcn_sched_barrier(0);
            dma_one(ks, kbuf, d);
            __builtin_amdgcn_sched_barrier(0);
          });
          static_for<NM - PER>([&](auto m) {
            constexpr int M = PER + decltype(m)::value;
            if (p == 0) mfma_one(ic<0>{}, ic<M>{}); else mfma_one(ic<1>{}, ic<M>{});
          });
        } else {
          static_for<NM>([&](auto m) {
            if (p == 0) mfma_one(ic<0>{}, m); else mfma_one(ic<1>{}, m);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    static_for<STAGES - 1>([&](auto st) {
      constexpr int S = decltype(st)::value;
      static_for<PER>([&](auto d) { dma_one(min(S, nk - 1), S, d); });
    });
    // stage 0 landed when at most the later prologue stages are outstanding
    wait_vmcnt<(STAGES - 2) * PER>();
    __builtin_amdgcn_s_barrier();
    CEP_LOAD_FRAG(fa[0], fb[0], 0, 0, 0, FM);
    for (int kt = 0; kt + 1 < nk; ++kt) {
      const int cur = kt % STAGES, nxt = (kt + 1) % STAGES;
      const int ks = min(kt + STAGES - 1, nk - 1), kbuf = (kt + STAGES - 1) % STAGES;
      early_subs(cur, std::true_type{}, ks, kbuf);
      mfma_one(ic<PL>{}, ic<0>{});
      __builtin_amdgcn_sched_barrier(0);
      // this thread's loads of stage kt+1 are done when at most the
      // STAGES-2 stages issued after it are outstanding
      wait_vmcnt<(STAGES - 2) * PER>();
      mfma_one(ic<PL>{}, ic<1>{});
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();  // stage kt+1 landed; step kt's buffer free
      __builtin_amdgcn_sched_barrier(0);
      static_for<NR / 2>([&](auto r) {
        constexpr int R = decltype(r)::value;
        mfma_one(ic<PL>{}, ic<2 + R>{});
        __builtin_amdgcn_sched_barrier(0);
        read_one(ic<QL>{}, nxt, ic<2 * R>{});
        read_one(ic<QL>{}, nxt, ic<2 * R + 1>{});
        __builtin_amdgcn_sched_barrier(0);
      });
      static_for<NM - 2 - NR / 2>(
          [&](auto m) { mfma_one(ic<PL>{}, ic<2 + NR / 2 + decltype(m)::value>{}); });
      __builtin_amdgcn_sched_barrier(0);
    }
    // the last step: no loads, no barrier
    early_subs((nk - 1) % STAGES, std::false_type{}, 0, 0);
    static_for<NM>([&](auto m) { mfma_one(ic<PL>{}, m); });
    // the tail's reloads must land before the workgroup's LDS is released
    wait_vmcnt<0>();
  } else {
    // NFA A fragments per wave and NAL_ A loads per wave and step, the
    // first NAL_ of the wave's SEGW_ load segments (wave w loads segments
    // w*SEGW_ ..: all of them, or for a VAR half tile those of its first
    // BM/2 rows); the wave's vmcnt waits count its own loads per step.
    auto run = [&](auto nfa_c, auto nal_c, auto segw_c) {
      constexpr int NFA = decltype(nfa_c)::value, NAL_ = decltype(nal_c)::value;
      constexpr int SEGW_ = decltype(segw_c)::value;
      constexpr int PERX = NAL_ + B_LD;
      const char *arow[NAL_ > 0 ? NAL_ : 1];
      CEP_AROWS(arow)
      if constexpr (ASTG == 2) {
        // B (weights, from HBM) runs STAGES-1 steps ahead, A (rows, mostly
        // L2 hits) one step ahead in a ring of two: the top of step j issues
        // A(j+1), then B(j+STAGES-1), into buffers last read in step j-1.
        // The prologue is "step -1" after B(0 .. STAGES-3).
#pragma unroll
        for (int s = 0; s < STAGES - 2; ++s)
          if (s < nk) CEP_DMA_B(s);
        CEP_DMA_A(0);
        if (STAGES - 2 < nk) CEP_DMA_B(STAGES - 2);
      } else {
        // Stage s is issued at the top of step s - STAGES + 1, into the
        // buffer of stage s - STAGES, which every wave finished reading in
        // step s - STAGES (before this step's barrier).
#pragma unroll
        for (int s = 0; s < STAGES - 1; ++s)
          if (s < nk) CEP_DMA_STAGE(s);
      }
      for (int kt = 0; kt < nk; ++kt) {
        if constexpr (ASTG == 2) {
          // A(kt) and B(kt) are done when only B(kt+STAGES-2), issued after
          // A(kt) at the top of step kt-1, may be outstanding
          if (kt + STAGES - 2 < nk)
            wait_vmcnt<B_LD>();
          else
            wait_vmcnt<0>();
        } else {
          // this thread's loads of step kt are done when at most the loads
          // of the steps issued after it are outstanding
          wait_stages<PERX, STAGES - 2>(min(nk - 1, kt + STAGES - 2) - kt);
        }
        // every wave's loads of step kt landed; step kt-1 fully consumed.  A
        // bare barrier: __syncthreads() would also drain the later loads.
        __builtin_amdgcn_s_barrier();
        if constexpr (ASTG == 2) {
          if (kt + 1 < nk) CEP_DMA_A(kt + 1);
          if (kt + STAGES - 1 < nk) CEP_DMA_B(kt + STAGES - 1);
        } else {
          if (kt + STAGES - 1 < nk) CEP_DMA_STAGE(kt + STAGES - 1);
        }
        const int acur = kt % AS, cur = kt % STAGES;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          bf16x8 fa[FM], fb[FN];
          CEP_LOAD_FRAG(fa, fb, acur, cur, kk, NFA);
#pragma unroll
          for (int i = 0; i < NFA; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
              acc[i][j] =
                  __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
      }
    };
    // LIN: a wave loads only those of its load segments (RPS rows each)
    // that hold rows of the tile (its MFMAs then read stale LDS rows for the
    // rest, whose outputs are never stored): a tile of a few rows requests
    // little more than its weights
    auto run_rows = [&](auto nfa_c, auto segw_c) {
      constexpr int SEGW = decltype(segw_c)::value;
      if constexpr (LIN) {
        const int n = min(SEGW, max(0, (t.rows - wid * SEGW * RPS + RPS - 1) / RPS));
        static_for<SEGW + 1>([&](auto k) {
          if (n == decltype(k)::value) run(nfa_c, k, segw_c);
        });
      } else {
        run(nfa_c, segw_c, segw_c);
      }
    };
    if constexpr (VAR) {
      if (half)
        run_rows(ic<1>{}, ic<A_LD / 2>{});
      else
        run_rows(ic<FM>{}, ic<A_LD>{});
    } else {
      run_rows(ic<FM>{}, ic<A_LD>{});
    }
  }
#undef CEP_LOAD_FRAG
#undef CEP_DMA_STAGE
#undef CEP_DMA_A
#undef CEP_DMA_B
#undef CEP_AROWS
#undef CEP_LANE_OFF

  // 32x32 accumulator layout: lane l, element r -> column l%32,
  // row 8*(r/4) + 4*(l/32) + r%4.
  // GEMM2: routing coefficients of the 16 rows the lane holds in row group
  // i.  The epilogues load group i+1's before storing group i's outputs, so
  // that waiting for a group's coefficients never waits for earlier stores.
  auto coef16 = [&](int i, float(&w)[16]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = frow(i) + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      w[r] = lr < t.rows ? g.wrow[(size_t)t.row0 + lr] : 0.0f;
    }
  };
  if constexpr (PIPE && !SWIGLU) {
    // float32 outputs straight from the accumulators: one store instruction
    // writes 32 consecutive columns (128 bytes) of two rows
    static_assert(WGM == 2 && !VAR, "two wave rows");
    float *Y = (float *)g.out;
    float wc[16], wx[16];
    coef16(0, wc);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (i + 1 < FM) coef16(i + 1, wx);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (lr >= t.rows) continue;
        const size_t row = (size_t)t.row0 + lr;
        const size_t ybase = row * g.N + nt * BN + wn * WN + (lane & 31);
#pragma unroll
        for (int j = 0; j < FN; ++j) Y[ybase + j * 32] = acc[i][j][r] * wc[r];
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) wc[r] = wx[r];
    }
    // every wave's last operand reads completed: the ring is free for the
    // next tile's loads (the stores may still be in flight)
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    continue;
  }
  if constexpr (PIPE) {
    // The h tile goes through LDS: each wave writes its bf16 results
    // into the (now idle) operand ring, rows of wave row 0 in sA and of wave
    // row 1 in sB, then the workgroup writes whole rows with 16-byte stores
    // (a store instruction covers two to four full rows instead of 64
    // two-byte pieces).  Chunk c of a staged row r sits at c ^ (4 * ((r/4) % 4)),
    // so the two half-waves of one element write (rows r and r+4) use
    // different banks.
    static_assert(WGM == 2 && !VAR, "staged epilogue: two wave rows");
    constexpr int CB = BN / 2;   // h columns of the tile
    constexpr int CPR = CB / 8;  // 16-byte chunks per output row
    constexpr int WCB = WN / 2;  // h columns of one wave
    static_assert(WM * CB * 2 <= (int)sizeof(sA) && WM * CB * 2 <= (int)sizeof(sB),
                  "a wave row's outputs fit one operand ring");
    static_assert(CPR % 4 == 0 && CPR >= 16, "swizzle stays inside the row");
    // every wave's tail loads landed (wait_vmcnt<0> above) and its last
    // operand reads completed: the ring is free
    __syncthreads();
    __bf16 *st = (__bf16 *)(wm == 0 ? (void *)&sA[0][0] : (void *)&sB[0][0]);
    auto soff = [](int r, int c) {
      return r * CB + ((((c >> 3) ^ (((r >> 2) & 3) << 2))) << 3) + (c & 7);
    };
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        // fragment pairs (2*j2, 2*j2+1) are the gate and up columns of h
        // columns wn*WCB + j2*32 + [0, 32) of the tile
#pragma unroll
        for (int j2 = 0; j2 < FN / 2; ++j2)
          st[soff(lr, wn * WCB + j2 * 32 + (lane & 31))] =
              (__bf16)silu_mul(acc[i][2 * j2][r], acc[i][2 * j2 + 1][r]);
      }
    }
    __syncthreads();
    const size_t ldo = g.N / 2;
    __bf16 *O = (__bf16 *)g.out + (size_t)t.row0 * ldo + (size_t)nt * CB;
#pragma unroll 4
    for (int q = tid; q < BM * CPR; q += 64 * NW) {
      const int row = q / CPR, c = q % CPR;
      if (row >= t.rows) break;  // q grows with the row
      const int lr = row % WM;
      const u32x4 *src = row < WM ? &sA[0][0] : &sB[0][0];
      *(u32x4 *)(O + (size_t)row * ldo + c * 8) = src[lr * CPR + (c ^ (((lr >> 2) & 3) << 2))];
    }
    // every wave's reads of the staged rows completed: the ring is free for
    // the next tile's loads (the stores may still be in flight)
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    continue;
  }
  if constexpr (XCH) {
    // the up waves hand their accumulators to the gate waves through the
    // idle A ring (every load of the K loop landed: the last step waited
    // for all of them)
    static_assert(FN == 1 && WGM * FM * 16 * 64 * 4 <= (int)sizeof(sA), "exchange fits the A ring");
    float *xch = (float *)&sA[0][0];
    __syncthreads();  // every wave's last operand reads completed
    if (wn == 1) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) xch[((wm * FM + i) * 16 + r) * 64 + lane] = acc[i][0][r];
    }
    __syncthreads();
    if (wn == 1) return;
    __bf16 *H = (__bf16 *)g.out;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (half && i > 0) break;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rt = frow(i) + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (rt >= t.rows) continue;
        const size_t row = (size_t)t.row0 + rt;
        // gate columns nt*BN + [0, 32) and up columns nt*BN + [32, 64) are
        // h columns nt*BN/2 + [0, 32)
        H[row * (g.N / 2) + nt * BN / 2 + (lane & 31)] =
            (__bf16)silu_mul(acc[i][0][r], xch[((wm * FM + i) * 16 + r) * 64 + lane]);
      }
    }
    return;
  }
  // GEMM2: direct output rows of the lane's 16 rows of group i (ydst), -1
  // for a grouped output row; rotated with the coefficients
  auto dst16 = [&](int i, int(&o)[16]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = frow(i) + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      o[r] = direct && lr < t.rows ? g.ydst[(size_t)t.row0 + lr] : -1;
    }
  };
  float wc[16], wx[16];
  int dc[16], dx[16];
  if (!SWIGLU) {
    coef16(0, wc);
    dst16(0, dc);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    if (half && i > 0) break;
    if (!SWIGLU && i + 1 < FM && !half) {
      coef16(i + 1, wx);
      dst16(i + 1, dx);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rt = frow(i) + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
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
        // a row with dc >= 0 goes to that output row (+0 for -0)
        const size_t col = (size_t)nt * BN + wn * WN + (lane & 31);
        float *yr = (dc[r] >= 0 ? g.yout + (size_t)dc[r] * g.N : (float *)g.out + row * g.N) + col;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const float v = acc[i][j][r] * wc[r];
          yr[j * 32] = dc[r] >= 0 ? __uint_as_float(plus_zero(__float_as_uint(v))) : v;
        }
      }
    }
    if (!SWIGLU) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        wc[r] = wx[r];
        dc[r] = dx[r];
      }
    }
  }
  }  // work items
}

}  // namespace

template <bool SWIGLU, bool GATHER>
hipError_t launch_bf16_as(const GemmArgs &g, int grid_tiles, int align, hipStream_t s) {
  if (align == kBf16TileM) {
    constexpr int BN = 256;
    if (g.N % BN) return hipErrorInvalidValue;
    const int grid = std::min(balanced_grid(grid_tiles, kGroupM, g.N / BN), persistent_grid());
    hipLaunchKernelGGL((k_gemm_bf16<kBf16TileM, BN, 32, 4, 1, true, SWIGLU, 2, 4, kGroupM, GATHER>),
                       dim3(grid), dim3(256), 0, s, g);
  } else if (align == kBf16SmallTileM) {
    constexpr int BN = 128;
    if (g.N % BN || g.K % 64) return hipErrorInvalidValue;
    const int grid = balanced_grid(grid_tiles, kGroupM, g.N / BN);
    hipLaunchKernelGGL(
        (k_gemm_bf16<kBf16SmallTileM, BN, 64, 3, 2, false, SWIGLU, 2, 4, kGroupM, GATHER>),
        dim3(grid), dim3(256), 0, s, g);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Remainder tiles run alone after the 256-row launch and touch one or two
// experts, so few workgroups stream their weights; each CU's streaming rate
// is bounded, so they use 64-column tiles: twice the workgroups of the
// streaming tile, half the weight bytes each (GEMM1's gate and up halves
// meet in LDS).
template <bool SWIGLU, bool GATHER>
hipError_t launch_bf16_rem_as(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  constexpr int BN = 64;
  if (g.N % BN || g.K % 64) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / BN);
  hipLaunchKernelGGL(
      (k_gemm_bf16<kBf16SmallTileM, BN, 64, 3, 2, false, SWIGLU, 2, 4, kGroupM, GATHER>),
      dim3(grid), dim3(256), 0, s, g);
  return hipGetLastError();
}

template <bool SWIGLU>
hipError_t launch_bf16_rem(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  if constexpr (SWIGLU) {
    if (g.A == nullptr) {
      if (!g.xrow || !g.perm || g.k < 1) return hipErrorInvalidValue;
      return launch_bf16_rem_as<true, true>(g, grid_tiles, s);
    }
  }
  return launch_bf16_rem_as<SWIGLU, false>(g, grid_tiles, s);
}
template hipError_t launch_bf16_rem<true>(const GemmArgs &, int, hipStream_t);
template hipError_t launch_bf16_rem<false>(const GemmArgs &, int, hipStream_t);

template <bool SWIGLU>
hipError_t launch_bf16(const GemmArgs &g, int grid_tiles, int align, hipStream_t s) {
  if constexpr (SWIGLU) {
    if (g.A == nullptr) {
      if (!g.xrow || !g.perm || g.k < 1) return hipErrorInvalidValue;
      return launch_bf16_as<true, true>(g, grid_tiles, align, s);
    }
  }
  return launch_bf16_as<SWIGLU, false>(g, grid_tiles, align, s);
}

template <bool SWIGLU, bool GATHER>
hipError_t launch_bf16_var_as(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  constexpr int BN = 128;
  if (g.N % BN || g.K % 64) return hipErrorInvalidValue;
  const int grid = balanced_grid(grid_tiles, kGroupM, g.N / BN);
  hipLaunchKernelGGL(
      (k_gemm_bf16<kBf16VarTileM, BN, 64, 3, 2, false, SWIGLU, 2, 4, kGroupM, GATHER, true, 2>),
      dim3(grid), dim3(256), 0, s, g);
  return hipGetLastError();
}

template <bool SWIGLU>
hipError_t launch_bf16_var(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  if constexpr (SWIGLU) {
    if (g.A == nullptr) {
      if (!g.xrow || !g.perm || g.k < 1) return hipErrorInvalidValue;
      return launch_bf16_var_as<true, true>(g, grid_tiles, s);
    }
  }
  return launch_bf16_var_as<SWIGLU, false>(g, grid_tiles, s);
}

// Weight-streaming batches (a few hundred pairs over all local experts, one
// of them hot).  A CU's load rate bounds these launches, and it counts every
// byte requested, rows from L2 as much as weights from HBM, so a launch lasts
// as long as its most loaded CU.  The scan lists the batch's 64-row tiles by
// rows, most first; the work items (GEMM1: 64 rows x 64 columns, 32 h
// columns; GEMM2: 64 x 128) follow that list one per workgroup, so the items
// of the largest tiles start first and the small ones fill in behind them,
// and each wave loads only its 8-row segments that hold rows (a tile of a
// few rows requests little more than its weights).  Straggler workload,
// per-chunk batches: GEMM1 108 -> 98 us, GEMM2 48.5 -> 46 us per batch on
// average.
template <bool GATHER>
hipError_t launch_bf16_stream_as(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  constexpr int BN = 64;
  if (g.N % BN || g.K % 64) return hipErrorInvalidValue;
  const int grid = grid_tiles * (g.N / BN);
  hipLaunchKernelGGL((k_gemm_bf16<kBf16SmallTileM, BN, 64, 3, 2, false, true, 2, 4, kGroupM,
                                  GATHER, false, 0, true>),
                     dim3(grid), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_bf16_stream2(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  constexpr int BN = 128;
  if (g.N % BN || g.K % 64) return hipErrorInvalidValue;
  const int grid = grid_tiles * (g.N / BN);
  hipLaunchKernelGGL((k_gemm_bf16<kBf16SmallTileM, BN, 64, 3, 2, false, false, 2, 4, kGroupM,
                                  false, false, 0, true>),
                     dim3(grid), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_bf16_stream(const GemmArgs &g, int grid_tiles, hipStream_t s) {
  if (g.A == nullptr) {
    if (!g.xrow || !g.perm || g.k < 1) return hipErrorInvalidValue;
    return launch_bf16_stream_as<true>(g, grid_tiles, s);
  }
  return launch_bf16_stream_as<false>(g, grid_tiles, s);
}

template hipError_t launch_bf16_var<true>(const GemmArgs &, int, hipStream_t);
template hipError_t launch_bf16_var<false>(const GemmArgs &, int, hipStream_t);
template hipError_t launch_bf16<true>(const GemmArgs &, int, int, hipStream_t);
template hipError_t launch_bf16<false>(const GemmArgs &, int, int, hipStream_t);

}  // namespace cep
