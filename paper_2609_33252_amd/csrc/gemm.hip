// Launchers of the grouped expert GEMMs (Appendix C, "Grouped FFN
// invocations"): GEMM1 = gate/up projection with SwiGLU (and, for e4m3
// and MXFP4 weights, the h re-quantisation) in the epilogue; GEMM2 = down
// projection scaled by each row's routing coefficient.  Kernels:
// gemm_bf16.hip, gemm_fp8.hip, gemm_mx.hip.
#include "gemm_common.h"

namespace cep {
namespace {

GemmArgs base_args(const Scratch &sc, int list, int list_cap, int grid_tiles,
                   const BlobTable &bt) {
  GemmArgs g{};
  g.tiles = sc.tiles + (size_t)list * list_cap;
  g.n_tiles = sc.n_tiles + list;
  g.max_tiles = grid_tiles;
  g.bt = bt;
  g.s_ld = sc.s_ld;
  return g;
}

template <bool SWIGLU>
hipError_t launch_any(const GemmArgs &g, int grid_tiles, int split_tiles, int align, int wk,
                      const Scratch &sc, int which, int list_cap, hipStream_t s) {
  if (wk == kWFp8) return launch_fp8<SWIGLU>(g, grid_tiles, align, s);
  if (wk == kWMx) return launch_mx<SWIGLU>(g, grid_tiles, align, s);
  hipError_t e = launch_bf16<SWIGLU>(g, grid_tiles, align, s);
  if (e != hipSuccess || split_tiles <= 0) return e;
  // remainder tiles: same operands and output, the 64-row list
  GemmArgs r = g;
  r.tiles = sc.tiles + (size_t)(2 * which + 1) * list_cap;
  r.n_tiles = sc.n_tiles + 2 * which + 1;
  r.max_tiles = split_tiles;
  return launch_bf16_rem<SWIGLU>(r, split_tiles, s);
}

// the scan's second list of `which`: the batch's 128-row tiles (kListVar)
// or its 64-row tiles ordered by rows (kListSorted)
GemmArgs var_list(GemmArgs g, const Scratch &sc, int which, int list_cap) {
  g.tiles = sc.tiles + (size_t)(2 * which + 1) * list_cap;
  g.n_tiles = sc.n_tiles + 2 * which + 1;
  return g;
}

}  // namespace

hipError_t launch_gemm1(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        int split_tiles, int align, bool var, bool stream, const BlobTable &bt,
                        const BlobLayout &L, int wk, int d, int I, const Arena *gather, int row0,
                        int k, hipStream_t s) {
  if (grid_tiles <= 0) return hipSuccess;
  GemmArgs g = base_args(sc, 2 * which, list_cap, grid_tiles, bt);
  g.A = (const uint8_t *)sc.xg;
  if (gather) {  // bf16 rows read in place through the permutation
    g.A = nullptr;
    g.xrow = gather->xrow;
    g.perm = sc.perm;
    g.arow0 = row0;
    g.k = k;
  }
  g.As = sc.xs;
  g.K = d;
  g.N = 2 * I;
  g.b_off = L.w1_off;
  g.bs_off = L.s1_off;
  g.out = sc.h;
  g.out_s = sc.hs;
  if (var) return launch_bf16_var<true>(var_list(g, sc, which, list_cap), grid_tiles, s);
  if (stream) return launch_bf16_stream(var_list(g, sc, which, list_cap), grid_tiles, s);
  return launch_any<true>(g, grid_tiles, split_tiles, align, wk, sc, which, list_cap, s);
}

hipError_t launch_gemm2(const Scratch &sc, int which, int list_cap, int grid_tiles,
                        int split_tiles, int align, bool var, bool stream, const BlobTable &bt,
                        const BlobLayout &L, int wk, int d, int I, float *out, hipStream_t s) {
  if (grid_tiles <= 0) return hipSuccess;
  GemmArgs g = base_args(sc, 2 * which, list_cap, grid_tiles, bt);
  if (out && gemm2_writes_solo(wk, align)) {
    g.yout = out;
    g.ydst = sc.ydst;
  }
  g.A = (const uint8_t *)sc.h;
  g.As = sc.hs;
  g.K = I;
  g.N = d;
  g.b_off = L.w2_off;
  g.bs_off = L.s2_off;
  g.out = sc.y;
  g.wrow = sc.wrow;
  if (var) return launch_bf16_var<false>(var_list(g, sc, which, list_cap), grid_tiles, s);
  if (stream) return launch_bf16_stream2(var_list(g, sc, which, list_cap), grid_tiles, s);
  return launch_any<false>(g, grid_tiles, split_tiles, align, wk, sc, which, list_cap, s);
}

}  // namespace cep
