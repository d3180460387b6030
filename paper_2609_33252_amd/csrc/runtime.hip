// Host runtime of libcep: context, chunk arena, launch policy, stream slots,
// weight fetch, layer barrier and statistics.  Implements include/cep.h.
//
// Section 3.2 ("Launch threshold", "Multi-stream execution"), Appendix C
// ("Asynchronous dispatch", "Grouped FFN invocations", "One-shot weight
// fetching", "Output return and combine").
//
// Threading: one host thread per context.  Every entry point except the
// introspection calls only enqueues work.
#include "common.h"
#include "../../include/cep.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace cep;

namespace {

struct ChunkRec {
  int replica;
  int row0, n_rows, n_pairs;
  hipEvent_t arrival;  // caller-owned, may be null
  const int32_t *token_idx;
  const void *x;
  const int32_t *topk_id;
  const float *topk_w;
};

struct BatchRec {
  int64_t first_chunk;
  int n_chunks;
  int row0, n_rows, n_pairs;
  int slot;
  int align;  // per-expert row alignment of the grouped layout (GEMM M tile)
  bool fetched;  // the batch has fetched experts' tiles (run after the copy)
  hipEvent_t ev_start, ev_end;
  // on the batch stream after: routing, GEMM1, GEMM2, combine
  hipEvent_t ev_phase[4];
  // fetched experts' GEMMs, on the batch stream after the resident experts'
  // GEMMs: after the wait for the copy, after GEMM1, after GEMM2
  hipEvent_t ev_fphase[3];
  bool phases;  // ev_phase (and ev_fphase for batches with fetched tiles) recorded
  // recorded routing (record_routing only), pinned host memory
  int32_t *h_cnt = nullptr, *h_off = nullptr, *h_off_pad = nullptr, *h_perm = nullptr,
          *h_pos = nullptr;
  int mpad_bound = 0;
};

enum LayerState { kIdle = 0, kOpen = 1 };

}  // namespace

struct cep_ctx {
  cep_config cfg{};
  int device = 0;
  std::string err;
  int wk = kWBf16;  // expert weight format
  BlobLayout L{};
  uint8_t *w_res = nullptr;  // E blobs
  std::vector<uint8_t> resident;
  uint64_t nonres_mask = 0;  // experts without resident weights
  uint8_t *fetch_buf = nullptr;
  int fetch_mode = CEP_FETCH_COPY;
  Arena arena{};
  int arena_cap = 0;
  uint32_t *d_err = nullptr;
  int max_pairs = 0, max_mpad = 0, max_tiles = 0, max_blocks = 0, max_rows = 0;
  int n_cu = 0;  // compute units of the device (tile-plan makespan estimate)
  hipStream_t ingest = nullptr;
  hipStream_t st[8] = {};
  hipStream_t copy = nullptr;  // the fetch's copies when the caller gives no stream
  // slot streams that ran batches (or hold arrival waits) since the last
  // layer barrier; the next layer's staging waits for exactly these
  unsigned used_st = 0;
  Scratch sc[8] = {};
  std::vector<void *> allocs;
  // policy
  int policy = CEP_WAIT_ALL, theta = 1, n_streams = 1;
  // layer state
  int state = kIdle;
  uint32_t gen = 0;
  int n_rep = 0, expected_chunks = 0;
  float *out = nullptr;
  int rows_used = 0;
  int64_t staged = 0;  // chunks [0, staged) have their metadata in the arena
  bool phase_timing = true;  // record per-phase events in each batch
  std::vector<ChunkRec> chunks;
  int64_t pending_first = 0;
  int pending_pairs = 0, pending_rows = 0;
  std::vector<BatchRec> batches;
  bool origin_set = false;
  hipEvent_t ev_origin = nullptr;
  // fetch: the one decision of this layer; fetched_mask = the fetched
  // experts, whose tiles run after the resident experts' GEMMs; copied: their
  // weights come from the fetch buffer and their tiles wait for the copy
  // (else they are read from the donor region in place: no copy, or a copy
  // that failed to start)
  bool fetched = false;
  uint64_t fetched_mask = 0;
  bool copied = false;
  bool fetch_copy_issued = false;  // a copy was enqueued (this layer)
  bool fetch_copy_prev = false;    // ev_fetch_ready holds an earlier layer's copy
  bool fetch_fallback = false;     // this layer's copy failed: read in place
  // where each expert's weights are read from in this layer (null: none)
  const uint8_t *blob_ptr[kMaxExperts] = {};
  hipEvent_t ev_fetch_start = nullptr, ev_fetch_ready = nullptr;
  // sync-only events, one set per slot (re-recorded per batch)
  hipEvent_t ev_ingest[8] = {};
  hipEvent_t ev_layer_done = nullptr, ev_layer_ingest = nullptr;
  // the last event recorded on the ingest stream with no kernel after it
  // (the end event of a batch that ran there), or null
  hipEvent_t ingest_tail = nullptr;
  std::vector<hipEvent_t> timing_pool[2];  // [fenced]
  size_t timing_used[2] = {0, 0};
};

namespace {

// message of the last failure of a call that had no context yet
thread_local std::string g_err;

int fail(cep_ctx *c, int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  (c ? c->err : g_err) = buf;
  return code;
}

}  // namespace

namespace cep {
// records the message of a failure that has no context (cep_last_error(NULL))
int set_global_error(int code, const char *msg) {
  g_err = msg;
  return code;
}
}  // namespace cep

namespace {

#define HIPCHK(ctx, call)                                                              \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail((ctx), CEP_EHIP, "%s: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, \
                  __LINE__);                                                           \
  } while (0)

bool valid_config(const cep_config *c, std::string *why) {
  auto bad = [&](const char *m) { *why = m; return false; };
  if (!c) return bad("cfg is NULL");
  if (c->d_model <= 0 || c->d_model % 256 || c->d_model > kMaxDim)
    return bad("d_model must be a positive multiple of 256, at most 32768");
  if (c->d_ff <= 0 || c->d_ff % 128 || c->d_ff > kMaxDim)
    return bad("d_ff must be a positive multiple of 128, at most 32768");
  if (c->n_local_experts < 1 || c->n_local_experts > kMaxExperts) return bad("n_local_experts must be in 1..64");
  if (c->top_k < 1 || c->top_k > kMaxTopK) return bad("top_k must be in 1..16");
  if (c->max_replicas < 1 || c->max_tokens_per_replica < 1) return bad("max_replicas and max_tokens_per_replica must be >= 1");
  if ((long long)c->max_replicas * c->max_tokens_per_replica > (1LL << 24)) return bad("max_replicas * max_tokens_per_replica too large");
  if (c->w_dtype < CEP_F32 || c->w_dtype > CEP_MXFP4) return bad("bad w_dtype");
  if (c->x_dtype != CEP_F32 && c->x_dtype != CEP_BF16) return bad("x_dtype must be CEP_F32 or CEP_BF16");
  if (c->w_dtype == CEP_FP8_E4M3_B128 && c->x_dtype != CEP_BF16) return bad("fp8 weights need bf16 token rows");
  if (c->w_dtype == CEP_MXFP4 && c->x_dtype != CEP_BF16) return bad("MXFP4 weights need bf16 token rows");
  if (c->n_streams < 1 || c->n_streams > 8) return bad("n_streams must be in 1..8");
  if (c->max_pairs_per_batch < 0) return bad("max_pairs_per_batch must be >= 0");
  return true;
}

int weight_kind(int w_dtype) {
  return w_dtype == CEP_FP8_E4M3_B128 ? kWFp8 : (w_dtype == CEP_MXFP4 ? kWMx : kWBf16);
}

void *dalloc(cep_ctx *c, size_t bytes, hipError_t *e) {
  void *p = nullptr;
  *e = hipMalloc(&p, std::max<size_t>(bytes, 256));
  if (*e == hipSuccess) c->allocs.push_back(p);
  return p;
}

// Timing events from per-layer pools.  Phase markers only measure time, so
// they skip the system-scope fence (an L2 writeback and invalidate between
// the phases); a batch's end event keeps it, because the host reads the
// batch's routing copies after synchronising on it.
// Events that only order streams of this device: a device-scope release.
constexpr unsigned kDepEvent = hipEventDisableTiming | hipEventReleaseToDevice;

hipEvent_t timing_event(cep_ctx *c, bool fenced) {
  std::vector<hipEvent_t> &pool = c->timing_pool[fenced];
  size_t &used = c->timing_used[fenced];
  if (used == pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, fenced ? hipEventDefault : hipEventDisableSystemFence) !=
        hipSuccess)
      return nullptr;
    pool.push_back(e);
  }
  return pool[used++];
}

void free_batch_records(cep_ctx *c) {
  for (auto &b : c->batches) {
    (void)hipHostFree(b.h_cnt);
    (void)hipHostFree(b.h_off);
    (void)hipHostFree(b.h_off_pad);
    (void)hipHostFree(b.h_perm);
    (void)hipHostFree(b.h_pos);
  }
  c->batches.clear();
}

// Stages the metadata of chunks [c->staged, upto) into the arena on stream s
// (one launch per group of chunks), after their arrival waits.
int stage_chunks(cep_ctx *c, int64_t upto, hipStream_t s) {
  const size_t xrb = (size_t)c->cfg.d_model * (c->cfg.x_dtype == CEP_F32 ? 4 : 2);
  while (c->staged < upto) {
    IngestGroup g{};
    while (g.n < kIngestGroup && c->staged < upto) {
      const ChunkRec &ch = c->chunks[c->staged++];
      if (ch.n_rows > 0)
        g.c[g.n++] = IngestChunk{ch.token_idx, ch.x, ch.topk_id, ch.topk_w, ch.row0, ch.n_rows,
                                 ch.replica};
    }
    HIPCHK(c, launch_ingest(c->arena, g, c->cfg.top_k, c->cfg.n_local_experts,
                            c->cfg.max_tokens_per_replica, xrb, c->d_err, s));
    if (s == c->ingest) c->ingest_tail = nullptr;
  }
  return CEP_OK;
}

// Stream slot and stream of the batch that will hold the chunks pending now
// (the next batch to launch).  With one stream, batches run on the ingest
// stream itself.
int pending_slot(const cep_ctx *c) { return (int)(c->batches.size() % c->n_streams); }
hipStream_t pending_stream(const cep_ctx *c) {
  return c->n_streams == 1 ? c->ingest : c->st[pending_slot(c)];
}

// Experts that have pairs routed to them but no weights this layer: neither
// resident nor fetched (copied or read in place).
uint64_t missing_experts(const cep_ctx *c) {
  return c->nonres_mask & ~c->fetched_mask;
}

// Launch all pending chunks as one grouped invocation on the next stream slot.
int launch_pending(cep_ctx *c) {
  const int64_t nch = (int64_t)c->chunks.size() - c->pending_first;
  if (nch <= 0 || c->pending_pairs == 0) {
    c->pending_first = c->chunks.size();
    c->pending_pairs = c->pending_rows = 0;
    return CEP_OK;
  }
  const cep_config &cfg = c->cfg;
  const int E = cfg.n_local_experts, k = cfg.top_k, d = cfg.d_model, I = cfg.d_ff;
  // every expert without resident weights must have been fetched (copied or
  // read in place) before a batch launches
  if (const uint64_t miss = missing_experts(c))
    return fail(c, CEP_ESTATE,
                "expert %d has no resident weights and no fetch this layer; the chunk stays "
                "pending (cep_weight_fetch, then cep_flush)",
                __builtin_ctzll(miss));

  BatchRec b{};
  b.first_chunk = c->pending_first;
  b.n_chunks = (int)nch;
  b.row0 = c->chunks[c->pending_first].row0;
  b.n_rows = c->pending_rows;
  b.n_pairs = c->pending_pairs;
  b.slot = pending_slot(c);
  const int slot = b.slot;
  // one stream: batches run on the ingest stream itself, in submission
  // order after their chunks' staging, without a cross-stream hop
  hipStream_t s = pending_stream(c);
  if (s != c->ingest) c->used_st |= 1u << slot;
  const Scratch &sc = c->sc[slot];
  const int P = b.n_pairs;
  const int A = batch_align(c->wk, b.n_pairs, E);
  b.align = A;
  const int tiles = std::min(c->max_tiles, (P + A - 1) / A + E);
  b.mpad_bound = std::min(c->max_mpad, tiles * A);
  // the end event is fenced only when the host reads routing copies after it
  b.phases = c->phase_timing;
  b.ev_start = b.phases ? timing_event(c, false) : nullptr;
  b.ev_end = timing_event(c, cfg.record_routing != 0);
  b.fetched = c->fetched_mask != 0;
  for (hipEvent_t &e : b.ev_phase) e = b.phases ? timing_event(c, false) : nullptr;
  for (hipEvent_t &e : b.ev_fphase) e = b.phases && b.fetched ? timing_event(c, false) : nullptr;
  if ((b.phases && !b.ev_start) || !b.ev_end ||
      (b.phases && (!b.ev_phase[0] || !b.ev_phase[1] || !b.ev_phase[2] || !b.ev_phase[3])) ||
      (b.phases && b.fetched && (!b.ev_fphase[0] || !b.ev_fphase[1] || !b.ev_fphase[2])))
    return fail(c, CEP_EHIP, "hipEventCreate failed");

  // the batch's chunks' arrival waits already sit on this stream (enqueued
  // at submit); the ingest stream carries the layer's start (after the
  // previous layer's batches, which read the arena), which the batch stream
  // follows; then it stages every chunk submitted so far (the batch's, and
  // chunks without local pairs before it) in one launch per group
  if (s != c->ingest) {
    HIPCHK(c, hipEventRecord(c->ev_ingest[slot], c->ingest));
    HIPCHK(c, hipStreamWaitEvent(s, c->ev_ingest[slot], 0));
  }
  if (b.phases) HIPCHK(c, hipEventRecord(b.ev_start, s));
  {
    const int rc = stage_chunks(c, (int64_t)c->chunks.size(), s);
    if (rc != CEP_OK) return rc;
  }
  // 256-row bf16 tiles: the scan may move small remainders to 64-row tiles
  // (at most two per expert), run by a second launch of the 64-row kernel
  const bool split = c->wk == kWBf16 && A == kBf16TileM;
  const int split_tiles = split ? 2 * E : 0;
  // 64-row bf16 batches with enough rows per expert: 128-row tiles
  const bool var = batch_var_tiles(c->wk, A, P, E);
  // smaller 64-row bf16 batches: GEMM1 over the tiles sorted by rows
  const bool stream = batch_stream_tiles(c->wk, A, P, E);
  HIPCHK(c, launch_route(c->arena, sc, b.row0, b.n_rows, k, E, A, P, c->max_mpad, c->max_tiles,
                         c->fetched_mask, cfg.x_dtype, c->wk, d, split ? c->n_cu : 0,
                         2 * I / kBf16TileN,
                         var ? kListVar : stream ? kListSorted : kListNone, c->d_err, s));
  if (b.phases) HIPCHK(c, hipEventRecord(b.ev_phase[0], s));

  BlobTable bt{};
  for (int e = 0; e < E; ++e) bt.blob[e] = c->blob_ptr[e];
  // bf16 rows with bf16 weights are not packed: GEMM1 reads them in place
  const Arena *gather = c->wk == kWBf16 && cfg.x_dtype == CEP_BF16 ? &c->arena : nullptr;

  HIPCHK(c, launch_gemm1(sc, 0, c->max_tiles, tiles, split_tiles, A, var, stream, bt, c->L,
                         c->wk, d, I, gather, b.row0, k, s));
  if (b.phases) HIPCHK(c, hipEventRecord(b.ev_phase[1], s));
  HIPCHK(c, launch_gemm2(sc, 0, c->max_tiles, tiles, split_tiles, A, var, stream, bt, c->L,
                         c->wk, d, I, c->out, s));
  if (b.phases) HIPCHK(c, hipEventRecord(b.ev_phase[2], s));
  // fetched experts' tiles (the scan's second tile lists) run after the
  // resident experts' GEMMs, once their weights are in: the copy overlaps
  // the resident work and delays nothing before it (Appendix C, "One-shot
  // weight fetching": the donor-side work does not wait for the copy)
  if (b.fetched) {
    if (c->copied) HIPCHK(c, hipStreamWaitEvent(s, c->ev_fetch_ready, 0));
    if (b.phases) HIPCHK(c, hipEventRecord(b.ev_fphase[0], s));
    HIPCHK(c, launch_gemm1(sc, 1, c->max_tiles, tiles, split_tiles, A, var, stream, bt, c->L,
                           c->wk, d, I, gather, b.row0, k, s));
    if (b.phases) HIPCHK(c, hipEventRecord(b.ev_fphase[1], s));
    HIPCHK(c, launch_gemm2(sc, 1, c->max_tiles, tiles, split_tiles, A, var, stream, bt, c->L,
                           c->wk, d, I, c->out, s));
    if (b.phases) HIPCHK(c, hipEventRecord(b.ev_fphase[2], s));
  }
  HIPCHK(c, launch_combine(c->arena, sc, b.row0, b.n_rows, k, d, c->wk == kWBf16,
                           gemm2_writes_solo(c->wk, A), c->out, s));
  if (b.phases) HIPCHK(c, hipEventRecord(b.ev_phase[3], s));

  if (cfg.record_routing) {
    HIPCHK(c, hipHostMalloc((void **)&b.h_cnt, sizeof(int32_t) * E, 0));
    HIPCHK(c, hipHostMalloc((void **)&b.h_off, sizeof(int32_t) * (E + 1), 0));
    HIPCHK(c, hipHostMalloc((void **)&b.h_off_pad, sizeof(int32_t) * (E + 1), 0));
    HIPCHK(c, hipHostMalloc((void **)&b.h_perm, sizeof(int32_t) * b.mpad_bound, 0));
    HIPCHK(c, hipHostMalloc((void **)&b.h_pos, sizeof(int32_t) * (size_t)b.n_rows * k, 0));
    HIPCHK(c, hipMemcpyAsync(b.h_cnt, sc.cnt, sizeof(int32_t) * E, hipMemcpyDeviceToHost, s));
    HIPCHK(c, hipMemcpyAsync(b.h_off, sc.off, sizeof(int32_t) * (E + 1), hipMemcpyDeviceToHost, s));
    HIPCHK(c, hipMemcpyAsync(b.h_off_pad, sc.off_pad, sizeof(int32_t) * (E + 1),
                             hipMemcpyDeviceToHost, s));
    HIPCHK(c, hipMemcpyAsync(b.h_perm, sc.perm, sizeof(int32_t) * b.mpad_bound,
                             hipMemcpyDeviceToHost, s));
    HIPCHK(c, hipMemcpyAsync(b.h_pos, sc.pos_of, sizeof(int32_t) * (size_t)b.n_rows * k,
                             hipMemcpyDeviceToHost, s));
  }
  HIPCHK(c, hipEventRecord(b.ev_end, s));
  if (s == c->ingest) c->ingest_tail = b.ev_end;
  c->batches.push_back(b);
  c->pending_first = c->chunks.size();
  c->pending_pairs = c->pending_rows = 0;
  return CEP_OK;
}

}  // namespace

// ================================================================== ABI

CEP_API size_t cep_packed_expert_bytes(const cep_config *cfg) {
  std::string why;
  if (!valid_config(cfg, &why)) return 0;
  return blob_layout(cfg->d_model, cfg->d_ff, weight_kind(cfg->w_dtype)).bytes;
}

static int pack_range(const cep_config *cfg, const cep_weights *w, int first, int n, uint8_t *dst,
                      hipStream_t s, cep_ctx *c, const uint8_t *mask) {
  const int d = cfg->d_model, I = cfg->d_ff;
  const int wk = weight_kind(cfg->w_dtype);
  const bool fp8 = wk == kWFp8;
  const BlobLayout L = blob_layout(d, I, wk);
  const size_t es = cfg->w_dtype == CEP_F32 ? 4 : (fp8 ? 1 : 2);
  const size_t mat = (size_t)d * I * es;
  const size_t smat = (size_t)(d / 128) * (I / 128);
  for (int q = 0; q < n; ++q) {
    const int e = first + q;
    if (mask && !mask[e]) continue;
    uint8_t *blob = dst + (size_t)q * L.bytes;
    if (wk == kWMx) {
      // codes: gate/up [I][d/2], down [d][I/2]; E8M0 scales [I][d/32], [d][I/32]
      const size_t cm = (size_t)d * I / 2, sm = (size_t)d * I / kMxBlock;
      const uint8_t *sg = (const uint8_t *)w->s_gate, *su = (const uint8_t *)w->s_up,
                    *sd = (const uint8_t *)w->s_down;
      HIPCHK(c, launch_pack_mx((const uint8_t *)w->w_gate + e * cm, (const uint8_t *)w->w_up + e * cm,
                               (const uint8_t *)w->w_down + e * cm, sg + e * sm, su + e * sm,
                               sd + e * sm, d, I, blob, L, s));
      continue;
    }
    HIPCHK(c, launch_pack_w1((const uint8_t *)w->w_gate + e * mat, (const uint8_t *)w->w_up + e * mat,
                             cfg->w_dtype, d, I, blob + L.w1_off, s));
    HIPCHK(c, launch_pack_w2((const uint8_t *)w->w_down + e * mat, cfg->w_dtype, d, I,
                             blob + L.w2_off, s));
    if (fp8)
      HIPCHK(c, launch_pack_scales((const float *)w->s_gate + e * smat,
                                   (const float *)w->s_up + e * smat,
                                   (const float *)w->s_down + e * smat,
                                   d, I, (float *)(blob + L.s1_off), (float *)(blob + L.s2_off), s));
  }
  return CEP_OK;
}

CEP_API int cep_pack_experts(const cep_config *cfg, const cep_weights *w, int first, int n,
                             void *dst, hipStream_t s) {
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, CEP_EINVAL, "cep_pack_experts: %s", why.c_str());
  if (!w || !dst || first < 0 || n < 0 || first + n > cfg->n_local_experts)
    return fail(nullptr, CEP_EINVAL, "cep_pack_experts: bad weights, dst or expert range");
  if (!w->w_gate || !w->w_up || !w->w_down ||
      (weight_kind(cfg->w_dtype) != kWBf16 && (!w->s_gate || !w->s_up || !w->s_down)))
    return fail(nullptr, CEP_EINVAL, "cep_pack_experts: NULL weight or scale pointer");
  return pack_range(cfg, w, first, n, (uint8_t *)dst, s, nullptr, nullptr);
}

namespace {
void scratch_setup(int dev);
}  // namespace

CEP_API int cep_init_experts(cep_ctx **out, const cep_config *cfg, const cep_weights *w,
                             const uint8_t *resident, hipStream_t s) {
  if (!out) return fail(nullptr, CEP_EINVAL, "cep_init_experts: out is NULL");
  *out = nullptr;
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, CEP_EINVAL, "cep_init_experts: %s", why.c_str());
  if (!w || !w->w_gate || !w->w_up || !w->w_down ||
      (weight_kind(cfg->w_dtype) != kWBf16 && (!w->s_gate || !w->s_up || !w->s_down)))
    return fail(nullptr, CEP_EINVAL, "cep_init_experts: NULL weight or scale pointer");
  cep_ctx *c = new cep_ctx();
  c->cfg = *cfg;
  if (hipGetDevice(&c->device) != hipSuccess ||
      hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device) !=
          hipSuccess) {
    delete c;
    return fail(nullptr, CEP_EHIP, "cep_init_experts: device query failed");
  }
  // the device's copy of the allocation-free call's scratch (once per device)
  scratch_setup(c->device);
  const int E = cfg->n_local_experts, k = cfg->top_k, d = cfg->d_model, I = cfg->d_ff;
  c->wk = weight_kind(cfg->w_dtype);
  c->L = blob_layout(d, I, c->wk);
  c->resident.assign(E, 1);
  if (resident)
    for (int e = 0; e < E; ++e) c->resident[e] = resident[e] ? 1 : 0;
  for (int e = 0; e < E; ++e)
    if (!c->resident[e]) c->nonres_mask |= 1ull << e;
  c->arena_cap = cfg->max_replicas * cfg->max_tokens_per_replica;
  c->max_rows = c->arena_cap;
  const long long def_pairs = (long long)c->arena_cap * k;
  c->max_pairs = cfg->max_pairs_per_batch > 0 ? (int)std::min<long long>(cfg->max_pairs_per_batch, def_pairs)
                                              : (int)def_pairs;
  // capacities cover every batch alignment: most tiles with the smallest,
  // most padded rows with the largest
  c->max_tiles = (c->max_pairs + kMinAlign - 1) / kMinAlign + E;
  c->max_mpad = (int)align_up((size_t)c->max_pairs, kMaxAlign) + kMaxAlign * (E + 1);
  c->max_blocks = (int)(((long long)c->max_rows * k + kRoutePairs - 1) / kRoutePairs);
  c->policy = CEP_WAIT_ALL;
  c->n_streams = cfg->n_streams;

  hipError_t e = hipSuccess;
  auto A = [&](size_t bytes) { return e == hipSuccess ? dalloc(c, bytes, &e) : nullptr; };
  c->w_res = (uint8_t *)A(c->L.bytes * E);
  if (cfg->fetch_buffer_bytes) c->fetch_buf = (uint8_t *)A(cfg->fetch_buffer_bytes);
  c->arena.ids = (int32_t *)A(sizeof(int32_t) * c->arena_cap * k);
  c->arena.w = (float *)A(sizeof(float) * c->arena_cap * k);
  c->arena.dst = (int32_t *)A(sizeof(int32_t) * c->arena_cap);
  c->arena.solo = (int32_t *)A(sizeof(int32_t) * c->arena_cap);
  c->arena.xrow = (const void **)A(sizeof(void *) * c->arena_cap);
  c->d_err = (uint32_t *)A(sizeof(uint32_t));
  const size_t xes = c->wk != kWBf16 ? 1 : 2;
  for (int i = 0; i < cfg->n_streams; ++i) {
    Scratch &sc = c->sc[i];
    sc.blk_cnt = (int32_t *)A(sizeof(int32_t) * c->max_blocks * E);
    sc.cnt = (int32_t *)A(sizeof(int32_t) * E);
    sc.off = (int32_t *)A(sizeof(int32_t) * (E + 1));
    sc.off_pad = (int32_t *)A(sizeof(int32_t) * (E + 1));
    sc.tiles = (Tile *)A(sizeof(Tile) * 4 * c->max_tiles);
    sc.n_tiles = (int32_t *)A(sizeof(int32_t) * 4);
    sc.pos_of = (int32_t *)A(sizeof(int32_t) * (size_t)c->max_rows * k);
    sc.perm = (int32_t *)A(sizeof(int32_t) * c->max_mpad);
    sc.wrow = (float *)A(sizeof(float) * c->max_mpad);
    sc.ydst = (int32_t *)A(sizeof(int32_t) * c->max_mpad);
    // bf16 rows with bf16 weights are read in place by GEMM1 (no packed copy)
    if (!(c->wk == kWBf16 && cfg->x_dtype == CEP_BF16)) sc.xg = A(xes * c->max_mpad * d);
    sc.h = A(xes * c->max_mpad * I);
    sc.y = A((c->wk == kWBf16 ? 4 : 2) * (size_t)c->max_mpad * d);
    if (c->wk != kWBf16) {  // E8M0 bytes per 32 channels
      sc.xs = (float *)A(sizeof(float) * c->max_mpad * (d / 128));
      sc.hs = (float *)A(sizeof(float) * c->max_mpad * (I / 128));
      sc.s_ld = c->max_mpad;
      sc.xs_pitch = (int)align_up((size_t)d / 32, 16);
      sc.xs_rows = (uint8_t *)A((size_t)c->max_mpad * sc.xs_pitch);
    }
  }
  if (e != hipSuccess) {
    cep_destroy(c);
    return fail(nullptr, CEP_ENOMEM, "cep_init_experts: device allocation failed: %s",
                hipGetErrorString(e));
  }
  // streams at default priority; events for ordering only skip timing
  bool ok = hipStreamCreateWithFlags(&c->ingest, hipStreamNonBlocking) == hipSuccess;
  for (int i = 0; i < cfg->n_streams && ok; ++i) {
    ok = hipStreamCreateWithFlags(&c->st[i], hipStreamNonBlocking) == hipSuccess &&
         hipEventCreateWithFlags(&c->ev_ingest[i], kDepEvent) == hipSuccess;
  }
  if (ok && cfg->fetch_buffer_bytes)
    ok = hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking) == hipSuccess;
  ok = ok && hipEventCreateWithFlags(&c->ev_origin, hipEventDisableSystemFence) == hipSuccess &&
       hipEventCreateWithFlags(&c->ev_fetch_start, hipEventDisableSystemFence) == hipSuccess &&
       hipEventCreate(&c->ev_fetch_ready) == hipSuccess &&
       hipEventCreateWithFlags(&c->ev_layer_done, hipEventDisableTiming) == hipSuccess &&
       hipEventCreateWithFlags(&c->ev_layer_ingest, kDepEvent) == hipSuccess;
  ok = ok && hipMemsetAsync(c->d_err, 0, sizeof(uint32_t), s) == hipSuccess;
  if (!ok) {
    cep_destroy(c);
    return fail(nullptr, CEP_EHIP, "cep_init_experts: stream/event creation failed");
  }
  int rc = pack_range(cfg, w, 0, E, c->w_res, s, c, c->resident.data());
  if (rc == CEP_OK && hipStreamSynchronize(s) != hipSuccess)
    rc = fail(c, CEP_EHIP, "cep_init_experts: weight packing failed");
  if (rc != CEP_OK) {
    g_err = c->err;
    cep_destroy(c);
    return rc;
  }
  *out = c;
  return CEP_OK;
}

CEP_API int cep_set_phase_timing(cep_ctx *c, int on) {
  if (!c) return CEP_EINVAL;
  if (c->state != kIdle) return fail(c, CEP_ESTATE, "cep_set_phase_timing inside an open layer");
  c->phase_timing = on != 0;
  return CEP_OK;
}

CEP_API int cep_set_policy(cep_ctx *c, int policy, int threshold_pairs, int n_streams) {
  if (!c) return CEP_EINVAL;
  if (c->state != kIdle) return fail(c, CEP_ESTATE, "cep_set_policy inside an open layer");
  if (policy < CEP_WAIT_ALL || policy > CEP_THRESHOLD)
    return fail(c, CEP_EINVAL, "unknown policy %d", policy);
  if (policy == CEP_THRESHOLD && threshold_pairs < 1)
    return fail(c, CEP_EINVAL, "threshold must be >= 1");
  if (n_streams < 1 || n_streams > c->cfg.n_streams)
    return fail(c, CEP_EINVAL, "n_streams must be in 1..%d", c->cfg.n_streams);
  c->policy = policy;
  c->theta = policy == CEP_THRESHOLD ? threshold_pairs : (policy == CEP_PER_CHUNK ? 1 : 0);
  c->n_streams = n_streams;
  return CEP_OK;
}

CEP_API int cep_begin_layer(cep_ctx *c, uint32_t generation, int n_replicas,
                            const int *chunks_per_replica, float *out) {
  if (!c) return CEP_EINVAL;
  if (c->state != kIdle) return fail(c, CEP_ESTATE, "previous layer not combined");
  if (n_replicas < 1 || n_replicas > c->cfg.max_replicas || !chunks_per_replica || !out)
    return fail(c, CEP_EINVAL, "bad n_replicas / chunks_per_replica / out");
  long long tot = 0;
  for (int r = 0; r < n_replicas; ++r) {
    if (chunks_per_replica[r] < 0) return fail(c, CEP_EINVAL, "negative chunk count");
    tot += chunks_per_replica[r];
  }
  // The previous layer's last batch end event, when nothing was enqueued on
  // the ingest stream after it and it is still pending, already marks where
  // this layer's ingest work can start: it becomes the clock origin (its
  // event object trades places with the origin's in the timing pool) and
  // the stream carries one marker fewer between layers.
  hipEvent_t prev_tail = c->used_st == 0 ? c->ingest_tail : nullptr;
  // the previous layer's batches may still read the arena: stage after them
  for (int i = 0; i < c->cfg.n_streams; ++i) {
    if ((c->used_st >> i) & 1) {
      HIPCHK(c, hipEventRecord(c->ev_ingest[i], c->st[i]));
      HIPCHK(c, hipStreamWaitEvent(c->ingest, c->ev_ingest[i], 0));
    }
  }
  c->used_st = 0;
  free_batch_records(c);
  c->timing_used[0] = c->timing_used[1] = 0;
  c->gen = generation;
  c->n_rep = n_replicas;
  c->expected_chunks = (int)tot;
  c->out = out;
  c->rows_used = 0;
  c->staged = 0;
  c->chunks.clear();
  c->pending_first = 0;
  c->pending_pairs = c->pending_rows = 0;
  bool aliased = false;
  if (prev_tail) {
    const hipError_t q = hipEventQuery(prev_tail);
    (void)hipGetLastError();  // a pending event's status is not an error
    if (q == hipErrorNotReady) {
      for (hipEvent_t &e : c->timing_pool[0]) {
        if (e == prev_tail) {
          std::swap(e, c->ev_origin);
          aliased = true;
          break;
        }
      }
    }
  }
  // clock origin of this layer's stats
  if (!aliased) HIPCHK(c, hipEventRecord(c->ev_origin, c->ingest));
  c->ingest_tail = nullptr;
  c->origin_set = true;
  c->fetched = false;
  c->fetched_mask = 0;
  c->copied = false;
  c->fetch_copy_prev = c->fetch_copy_prev || c->fetch_copy_issued;
  c->fetch_copy_issued = false;
  c->fetch_fallback = false;
  for (int e = 0; e < c->cfg.n_local_experts; ++e)
    c->blob_ptr[e] = c->resident[e] ? c->w_res + (size_t)e * c->L.bytes : nullptr;
  c->state = kOpen;
  return CEP_OK;
}

CEP_API int cep_submit_chunk(cep_ctx *c, uint32_t generation, int replica, int n_rows, int n_pairs,
                             const int32_t *token_idx, const void *x, const int32_t *topk_id,
                             const float *topk_w, hipEvent_t arrival, int64_t *chunk_id) {
  if (!c) return CEP_EINVAL;
  if (c->state != kOpen) return fail(c, CEP_ESTATE, "no open layer");
  if (generation != c->gen) return fail(c, CEP_ESTATE, "generation %u, layer is %u", generation, c->gen);
  if ((int)c->chunks.size() >= c->expected_chunks)
    return fail(c, CEP_ESTATE, "all %d expected chunks already submitted", c->expected_chunks);
  if (replica < 0 || replica >= c->n_rep) return fail(c, CEP_EINVAL, "replica %d out of range", replica);
  if (n_rows < 0 || n_pairs < 0 || (long long)n_pairs > (long long)n_rows * c->cfg.top_k)
    return fail(c, CEP_EINVAL, "bad n_rows %d / n_pairs %d", n_rows, n_pairs);
  if (n_rows > 0 && (!token_idx || !x || !topk_id || !topk_w))
    return fail(c, CEP_EINVAL, "NULL chunk array");
  if (((uintptr_t)x & 15) != 0) return fail(c, CEP_EINVAL, "x must be 16-byte aligned");
  if (c->rows_used + n_rows > c->arena_cap)
    return fail(c, CEP_ENOMEM, "layer rows exceed max_replicas * max_tokens_per_replica");
  if (n_pairs > c->max_pairs)
    return fail(c, CEP_ENOMEM, "chunk pairs %d exceed max_pairs_per_batch %d", n_pairs, c->max_pairs);
  // a chunk that would overflow a batch first launches what is pending,
  // before anything of this chunk is recorded (a failure leaves the layer as
  // it was before the call)
  if (n_pairs > 0 && c->pending_pairs > 0 && c->pending_pairs + n_pairs > c->max_pairs) {
    int rc = launch_pending(c);
    if (rc != CEP_OK) return rc;
  }
  // readiness (Appendix C, "Asynchronous dispatch": a lane's inputs become
  // eligible on its own signal): the wait goes on the stream of the batch
  // that will hold this chunk, ahead of that batch's staging, so no other
  // batch waits for this chunk's arrival
  if (arrival) {
    hipStream_t s = pending_stream(c);
    HIPCHK(c, hipStreamWaitEvent(s, arrival, 0));
    if (s == c->ingest)
      c->ingest_tail = nullptr;
    else
      c->used_st |= 1u << pending_slot(c);
  }
  ChunkRec ch{replica, c->rows_used, n_rows, n_pairs, arrival, token_idx, x, topk_id, topk_w};
  c->rows_used += n_rows;
  const int64_t id = (int64_t)c->chunks.size();
  if (chunk_id) *chunk_id = id;
  c->chunks.push_back(ch);
  if (n_pairs > 0) {
    if (c->pending_pairs == 0) c->pending_first = id;
    c->pending_pairs += n_pairs;
    c->pending_rows = (int)(c->rows_used - c->chunks[c->pending_first].row0);
  } else if (c->pending_pairs == 0) {
    c->pending_first = id + 1;
  }
  const bool last = (int)c->chunks.size() == c->expected_chunks;
  const bool thresh = c->policy != CEP_WAIT_ALL && c->pending_pairs >= c->theta && c->pending_pairs > 0;
  // a launch that fails here (an expert without weights) leaves the chunk
  // pending: cep_weight_fetch and then cep_flush launch it
  if (thresh || last) return launch_pending(c);
  return CEP_OK;
}

CEP_API int cep_flush(cep_ctx *c) {
  if (!c) return CEP_EINVAL;
  if (c->state != kOpen) return fail(c, CEP_ESTATE, "no open layer");
  return launch_pending(c);
}

CEP_API int cep_weight_fetch(cep_ctx *c, const int *ids, int n, const void *const *src_blobs,
                             hipStream_t side, hipEvent_t *ready) {
  if (!c) return CEP_EINVAL;
  if (c->state != kOpen) return fail(c, CEP_ESTATE, "no open layer");
  if (c->fetched) return fail(c, CEP_EBUSY, "one weight fetch per layer");
  if (n < 0 || (n > 0 && (!ids || !src_blobs)))
    return fail(c, CEP_EINVAL, "bad fetch arguments");
  uint64_t mask = 0;
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= c->cfg.n_local_experts)
      return fail(c, CEP_EINVAL, "fetch id %d out of range", ids[i]);
    if ((mask >> ids[i]) & 1) return fail(c, CEP_EINVAL, "duplicate fetch id %d", ids[i]);
    if (!src_blobs[i]) return fail(c, CEP_EINVAL, "NULL source blob");
    mask |= 1ull << ids[i];
  }
  const size_t need = (size_t)n * c->L.bytes;
  if (need > c->cfg.fetch_buffer_bytes)
    return fail(c, CEP_ENOMEM, "fetch of %zu bytes exceeds the %zu-byte buffer", need,
                c->cfg.fetch_buffer_bytes);
  c->fetched = true;  // one decision per layer, also when it copies nothing
  if (ready) *ready = nullptr;
  if (n == 0) return CEP_OK;
  bool in_place = c->fetch_mode == CEP_FETCH_IN_PLACE;
  if (!in_place) {
    hipStream_t s = side ? side : c->copy;
    // do not overwrite the buffer while an earlier layer's batches may still
    // read it (the earlier layer's barrier event covers all of them), nor
    // while an earlier layer's copy may still write it
    if (c->fetch_copy_prev) {
      HIPCHK(c, hipStreamWaitEvent(s, c->ev_layer_done, 0));
      HIPCHK(c, hipStreamWaitEvent(s, c->ev_fetch_ready, 0));
    }
    HIPCHK(c, hipEventRecord(c->ev_fetch_start, s));
    // expert e goes to slot = number of fetched experts with a smaller id.  A
    // copy that fails to start ends the copying; the fetch then falls back to
    // reading the donor blobs in place (Appendix C, "FFN reassignment commit
    // and fallback": a failed copy never triggers another fetch decision)
    for (int i = 0; i < n && !in_place; ++i) {
      const int slot = __builtin_popcountll(mask & ((1ull << ids[i]) - 1));
      uint8_t *dst = c->fetch_buf + (size_t)slot * c->L.bytes;
      const hipError_t e =
          c->fetch_mode == CEP_FETCH_FAIL_COPY
              ? hipErrorInvalidValue
              : hipMemcpyAsync(dst, src_blobs[i], c->L.bytes, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        in_place = true;
        c->fetch_fallback = true;
      }
    }
    // the copies already enqueued finish before `ready`, which the layer
    // barrier also waits for
    HIPCHK(c, hipEventRecord(c->ev_fetch_ready, s));
    c->fetch_copy_issued = true;
  }
  if (in_place) {
    // fetched experts read their donor blobs where they are: their tiles still
    // run after the resident experts' GEMMs, with no copy to wait for
    for (int i = 0; i < n; ++i) c->blob_ptr[ids[i]] = (const uint8_t *)src_blobs[i];
    c->fetched_mask = mask;
    return CEP_OK;
  }
  for (int i = 0; i < n; ++i) {
    const int slot = __builtin_popcountll(mask & ((1ull << ids[i]) - 1));
    c->blob_ptr[ids[i]] = c->fetch_buf + (size_t)slot * c->L.bytes;
  }
  c->fetched_mask = mask;
  c->copied = true;
  if (ready) *ready = c->ev_fetch_ready;
  return CEP_OK;
}

CEP_API int cep_set_fetch_mode(cep_ctx *c, int mode) {
  if (!c) return CEP_EINVAL;
  if (c->state != kIdle) return fail(c, CEP_ESTATE, "cep_set_fetch_mode inside an open layer");
  if (mode < CEP_FETCH_COPY || mode > CEP_FETCH_FAIL_COPY)
    return fail(c, CEP_EINVAL, "unknown fetch mode %d", mode);
  c->fetch_mode = mode;
  return CEP_OK;
}

CEP_API int cep_combine(cep_ctx *c, hipStream_t s, hipEvent_t *done) {
  if (!c) return CEP_EINVAL;
  if (c->state != kOpen) return fail(c, CEP_ESTATE, "no open layer");
  if ((int)c->chunks.size() < c->expected_chunks)
    return fail(c, CEP_ESTATE, "%d of %d chunks submitted; cep_flush ends a layer early",
                (int)c->chunks.size(), c->expected_chunks);
  int rc = launch_pending(c);
  if (rc != CEP_OK) return rc;
  // chunks after the last batch (no local pairs) are still staged, so their
  // ids are validated and the caller may release them after `done`; their
  // arrival waits sit on the stream of the batch that would have held them
  if (c->staged < (int64_t)c->chunks.size()) {
    hipStream_t ps = pending_stream(c);
    if (ps != c->ingest) {
      HIPCHK(c, hipEventRecord(c->ev_ingest[pending_slot(c)], c->ingest));
      HIPCHK(c, hipStreamWaitEvent(ps, c->ev_ingest[pending_slot(c)], 0));
      c->used_st |= 1u << pending_slot(c);
    }
    rc = stage_chunks(c, (int64_t)c->chunks.size(), ps);
    if (rc != CEP_OK) return rc;
  }
  // every batch of the layer ran on a used slot stream or on the ingest
  // stream
  for (int i = 0; i < c->cfg.n_streams; ++i) {
    if ((c->used_st >> i) & 1) {
      HIPCHK(c, hipEventRecord(c->ev_ingest[i], c->st[i]));
      HIPCHK(c, hipStreamWaitEvent(s, c->ev_ingest[i], 0));
    }
  }
  if (s != c->ingest) {
    // a batch end event with no kernel after it already marks the end of
    // the ingest stream's work: one marker fewer between layers
    if (!c->ingest_tail) HIPCHK(c, hipEventRecord(c->ev_layer_ingest, c->ingest));
    HIPCHK(c, hipStreamWaitEvent(s, c->ingest_tail ? c->ingest_tail : c->ev_layer_ingest, 0));
  }
  // the layer's copy (also one no batch consumed) has finished reading the
  // donor blobs and writing the fetch buffer before `done`
  if (c->fetch_copy_issued) HIPCHK(c, hipStreamWaitEvent(s, c->ev_fetch_ready, 0));
  HIPCHK(c, hipEventRecord(c->ev_layer_done, s));
  if (done) *done = c->ev_layer_done;
  c->state = kIdle;
  return CEP_OK;
}

CEP_API int cep_get_batch_count(const cep_ctx *c) { return c ? (int)c->batches.size() : 0; }

CEP_API int cep_get_batch_routing(cep_ctx *c, int batch, int *align, int *n_pairs, int *n_rows,
                                  int32_t *cnt, int32_t *off, int32_t *off_pad, int32_t *perm_src,
                                  int32_t *pos_of, int64_t *chunks, int *n_chunks) {
  if (!c) return CEP_EINVAL;
  if (batch < 0 || batch >= (int)c->batches.size()) return fail(c, CEP_EINVAL, "no batch %d", batch);
  const BatchRec &b = c->batches[batch];
  const int E = c->cfg.n_local_experts, k = c->cfg.top_k;
  if (align) *align = b.align;
  if (n_pairs) *n_pairs = b.n_pairs;
  if (n_rows) *n_rows = b.n_rows;
  if (n_chunks) *n_chunks = b.n_chunks;
  if (chunks)
    for (int i = 0; i < b.n_chunks; ++i) chunks[i] = b.first_chunk + i;
  if (!(cnt || off || off_pad || perm_src || pos_of)) return CEP_OK;
  if (!c->cfg.record_routing) return fail(c, CEP_ESTATE, "record_routing is off");
  HIPCHK(c, hipEventSynchronize(b.ev_end));
  if (cnt) memcpy(cnt, b.h_cnt, sizeof(int32_t) * E);
  if (off) memcpy(off, b.h_off, sizeof(int32_t) * (E + 1));
  if (off_pad) memcpy(off_pad, b.h_off_pad, sizeof(int32_t) * (E + 1));
  if (pos_of) memcpy(pos_of, b.h_pos, sizeof(int32_t) * (size_t)b.n_rows * k);
  if (perm_src) {
    for (int e = 0; e < E; ++e)
      for (int q = 0; q < b.h_cnt[e]; ++q) {
        const int p = b.h_off_pad[e] + q;
        if (p < b.mpad_bound && b.h_off[e] + q < b.n_pairs) perm_src[b.h_off[e] + q] = b.h_perm[p];
      }
  }
  return CEP_OK;
}

CEP_API int cep_get_stats(cep_ctx *c, char *buf, size_t cap) {
  if (!c || !buf) return CEP_EINVAL;
  std::string js = "{\"batches\":[";
  char tmp[1024];
  for (size_t i = 0; i < c->batches.size(); ++i) {
    const BatchRec &b = c->batches[i];
    HIPCHK(c, hipEventSynchronize(b.ev_end));
    float t0 = -1, t1 = 0, ph[4] = {-1, -1, -1, -1};
    if (b.phases) HIPCHK(c, hipEventElapsedTime(&t0, c->ev_origin, b.ev_start));
    HIPCHK(c, hipEventElapsedTime(&t1, c->ev_origin, b.ev_end));
    hipEvent_t prev = b.ev_start;
    for (int p = 0; b.phases && p < 4; ++p) {
      HIPCHK(c, hipEventElapsedTime(&ph[p], prev, b.ev_phase[p]));
      prev = b.ev_phase[p];
    }
    // fetched experts' GEMMs sit between GEMM2 and the combine
    float h0 = -1, hg1 = -1, hg2 = -1;
    if (b.phases && b.fetched) {
      HIPCHK(c, hipEventElapsedTime(&h0, c->ev_origin, b.ev_fphase[0]));
      HIPCHK(c, hipEventElapsedTime(&hg1, b.ev_fphase[0], b.ev_fphase[1]));
      HIPCHK(c, hipEventElapsedTime(&hg2, b.ev_fphase[1], b.ev_fphase[2]));
      HIPCHK(c, hipEventElapsedTime(&ph[3], b.ev_fphase[2], b.ev_phase[3]));
    }
    snprintf(tmp, sizeof tmp,
             "%s{\"first_chunk\":%lld,\"n_chunks\":%d,\"rows\":%d,\"pairs\":%d,\"slot\":%d,"
             "\"fetched\":%s,\"start_ms\":%.6f,\"end_ms\":%.6f,\"route_ms\":%.6f,"
             "\"gemm1_ms\":%.6f,\"gemm2_ms\":%.6f,\"combine_ms\":%.6f,"
             "\"fetched_start_ms\":%.6f,\"fetched_gemm1_ms\":%.6f,\"fetched_gemm2_ms\":%.6f}",
             i ? "," : "", (long long)b.first_chunk, b.n_chunks, b.n_rows, b.n_pairs, b.slot,
             b.fetched ? "true" : "false", t0, t1, ph[0], ph[1], ph[2], ph[3], h0, hg1, hg2);
    js += tmp;
  }
  js += "],\"chunks\":[";
  for (size_t i = 0; i < c->chunks.size(); ++i) {
    const ChunkRec &ch = c->chunks[i];
    float ta = -1;
    if (ch.arrival && c->origin_set) {
      // an arrival event without timing has no timestamp: report -1 and
      // clear the runtime's sticky error so later launches do not see it
      if (hipEventSynchronize(ch.arrival) != hipSuccess ||
          hipEventElapsedTime(&ta, c->ev_origin, ch.arrival) != hipSuccess) {
        ta = -1;
        (void)hipGetLastError();
      }
    }
    snprintf(tmp, sizeof tmp, "%s{\"replica\":%d,\"rows\":%d,\"pairs\":%d,\"arrival_ms\":%.6f}",
             i ? "," : "", ch.replica, ch.n_rows, ch.n_pairs, ta);
    js += tmp;
  }
  js += "]";
  if (c->fetched && c->fetched_mask) {
    float f0 = -1, f1 = -1;
    if (c->fetch_copy_issued) {
      HIPCHK(c, hipEventSynchronize(c->ev_fetch_ready));
      if (c->origin_set) {
        (void)hipEventElapsedTime(&f0, c->ev_origin, c->ev_fetch_start);
        (void)hipEventElapsedTime(&f1, c->ev_origin, c->ev_fetch_ready);
      }
    }
    // bytes: what the copy moved into the fetch buffer (0 when read in place)
    snprintf(tmp, sizeof tmp,
             ",\"fetch\":{\"start_ms\":%.6f,\"end_ms\":%.6f,\"bytes\":%zu,\"experts\":%d,"
             "\"in_place\":%s,\"fallback\":%s}",
             f0, f1, c->copied ? (size_t)__builtin_popcountll(c->fetched_mask) * c->L.bytes : 0,
             __builtin_popcountll(c->fetched_mask), c->copied ? "false" : "true",
             c->fetch_fallback ? "true" : "false");
    js += tmp;
  }
  js += "}";
  if (js.size() + 1 > cap) return fail(c, CEP_ENOMEM, "stats need %zu bytes", js.size() + 1);
  memcpy(buf, js.c_str(), js.size() + 1);
  return CEP_OK;
}

CEP_API int cep_get_status(cep_ctx *c) {
  if (!c) return CEP_EINVAL;
  HIPCHK(c, hipDeviceSynchronize());
  uint32_t w = 0;
  HIPCHK(c, hipMemcpy(&w, c->d_err, sizeof w, hipMemcpyDeviceToHost));
  HIPCHK(c, hipMemset(c->d_err, 0, sizeof w));
  if (!w) return CEP_OK;
  return fail(c, CEP_EINVAL, "device-side check failed:%s%s%s%s", (w & kErrBadId) ? " expert id out of range" : "",
              (w & kErrPairCount) ? " n_pairs mismatch" : "", (w & kErrBadToken) ? " token index out of range" : "",
              (w & kErrOverflow) ? " batch exceeded scratch capacity" : "");
}

CEP_API const char *cep_last_error(const cep_ctx *c) {
  if (!c) return g_err.c_str();
  return c->err.c_str();
}

CEP_API int cep_destroy(cep_ctx *c) {
  if (!c) return CEP_OK;
  (void)hipDeviceSynchronize();
  free_batch_records(c);
  for (auto &pool : c->timing_pool)
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  hipEvent_t evs[] = {c->ev_origin, c->ev_fetch_start, c->ev_fetch_ready, c->ev_layer_done,
                      c->ev_layer_ingest};
  for (hipEvent_t e : evs)
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < 8; ++i) {
    if (c->ev_ingest[i]) (void)hipEventDestroy(c->ev_ingest[i]);
    if (c->st[i]) (void)hipStreamDestroy(c->st[i]);
  }
  if (c->ingest) (void)hipStreamDestroy(c->ingest);
  if (c->copy) (void)hipStreamDestroy(c->copy);
  for (void *p : c->allocs) (void)hipFree(p);
  delete c;
  return CEP_OK;
}

// ===================================================== allocation-free call
// One grouped invocation whose scratch (arena, routing arrays, tile lists,
// grouped rows, h and expert outputs) is carved from a file-scope device
// array instead of the context's buffers, for callers that cannot allocate.
// Each device holds its own copy of the array at its own address, found once
// per device by cep_init_experts; every call on a device shares it.
namespace {

constexpr size_t kNoAllocBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
hipError_t g_scratch_err[kMaxDevices] = {};

// With device `dev` current: the device address of that device's copy of
// `scratch`, looked up once.
void scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev]) return;
  void *p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e == hipSuccess && p) {
    g_scratch_ptr[dev] = p;
  } else {
    g_scratch_err[dev] = e;
    (void)hipGetLastError();
  }
}

// Sub-allocation of `bytes` (256-byte aligned) from a carve cursor.
struct Carver {
  size_t used = 0;
  uint8_t *base = nullptr;  // null: only count
  void *take(size_t bytes) {
    void *p = base ? base + used : nullptr;
    used += align_up(std::max<size_t>(bytes, 1), 256);
    return p;
  }
};

}  // namespace

CEP_API int cep_ffn_noalloc(cep_ctx *c, int replica, int n_rows, int n_pairs,
                            const int32_t *token_idx, const void *x, const int32_t *topk_id,
                            const float *topk_w, float *out, hipStream_t s) {
  if (!c) return CEP_EINVAL;
  const cep_config &cfg = c->cfg;
  const int E = cfg.n_local_experts, k = cfg.top_k, d = cfg.d_model, I = cfg.d_ff;
  if (replica < 0 || replica >= cfg.max_replicas)
    return fail(c, CEP_EINVAL, "replica %d out of range", replica);
  if (n_rows < 0 || n_rows > cfg.max_tokens_per_replica || n_pairs < 0 ||
      (long long)n_pairs > (long long)n_rows * k)
    return fail(c, CEP_EINVAL, "bad n_rows %d / n_pairs %d", n_rows, n_pairs);
  if (n_rows > 0 && (!token_idx || !x || !topk_id || !topk_w || !out))
    return fail(c, CEP_EINVAL, "NULL chunk array or output");
  if (((uintptr_t)x & 15) != 0) return fail(c, CEP_EINVAL, "x must be 16-byte aligned");
  if (c->nonres_mask)
    return fail(c, CEP_ESTATE, "the allocation-free call needs every expert resident");
  if (n_pairs == 0) return CEP_OK;
  // capacities of this one invocation: its row alignment A is known here, so
  // the grouped rows need at most P + E*(A-1) (each expert's last tile
  // padded), rounded up to whole 256-row groups of the scale layouts
  const int P = n_pairs;
  const int A = batch_align(c->wk, P, E);
  const int mpad = (int)align_up((size_t)P + (size_t)E * A, kMaxAlign);
  const int tiles_cap = (P + kMinAlign - 1) / kMinAlign + E;
  const int blocks = (int)(((long long)n_rows * k + kRoutePairs - 1) / kRoutePairs);
  const size_t xes = c->wk != kWBf16 ? 1 : 2;
  const bool packed = !(c->wk == kWBf16 && cfg.x_dtype == CEP_BF16);
  Carver cv;
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1) {
      if (cv.used > kNoAllocBytes)
        return fail(c, CEP_ENOMEM,
                    "%d rows with %d pairs need %zu bytes of scratch; the allocation-free "
                    "call has %zu",
                    n_rows, n_pairs, cv.used, kNoAllocBytes);
      const int dev = c->device;
      if (dev < 0 || dev >= kMaxDevices || !g_scratch_ptr[dev])
        return fail(c, CEP_EHIP, "scratch address of device %d unavailable: %s", dev,
                    hipGetErrorString(dev >= 0 && dev < kMaxDevices ? g_scratch_err[dev]
                                                                   : hipErrorInvalidDevice));
      cv = Carver{};
      cv.base = (uint8_t *)g_scratch_ptr[dev];
    }
    Arena a{};
    a.ids = (int32_t *)cv.take(sizeof(int32_t) * (size_t)n_rows * k);
    a.w = (float *)cv.take(sizeof(float) * (size_t)n_rows * k);
    a.dst = (int32_t *)cv.take(sizeof(int32_t) * (size_t)n_rows);
    a.solo = (int32_t *)cv.take(sizeof(int32_t) * (size_t)n_rows);
    a.xrow = (const void **)cv.take(sizeof(void *) * (size_t)n_rows);
    Scratch sc{};
    sc.blk_cnt = (int32_t *)cv.take(sizeof(int32_t) * (size_t)blocks * E);
    sc.cnt = (int32_t *)cv.take(sizeof(int32_t) * E);
    sc.off = (int32_t *)cv.take(sizeof(int32_t) * (E + 1));
    sc.off_pad = (int32_t *)cv.take(sizeof(int32_t) * (E + 1));
    sc.tiles = (Tile *)cv.take(sizeof(Tile) * 4 * (size_t)tiles_cap);
    sc.n_tiles = (int32_t *)cv.take(sizeof(int32_t) * 4);
    sc.pos_of = (int32_t *)cv.take(sizeof(int32_t) * (size_t)n_rows * k);
    sc.perm = (int32_t *)cv.take(sizeof(int32_t) * (size_t)mpad);
    sc.wrow = (float *)cv.take(sizeof(float) * (size_t)mpad);
    sc.ydst = (int32_t *)cv.take(sizeof(int32_t) * (size_t)mpad);
    if (packed) sc.xg = cv.take(xes * (size_t)mpad * d);
    sc.h = cv.take(xes * (size_t)mpad * I);
    sc.y = cv.take((c->wk == kWBf16 ? 4 : 2) * (size_t)mpad * d);
    if (c->wk != kWBf16) {
      sc.xs = (float *)cv.take(sizeof(float) * (size_t)mpad * (d / 128));
      sc.hs = (float *)cv.take(sizeof(float) * (size_t)mpad * (I / 128));
      sc.s_ld = mpad;
      sc.xs_pitch = (int)align_up((size_t)d / 32, 16);
      sc.xs_rows = (uint8_t *)cv.take((size_t)mpad * sc.xs_pitch);
    }
    if (pass == 0) continue;

    // the same kernels as a one-chunk wait-all layer, on stream s
    IngestGroup g{};
    g.c[0] = IngestChunk{token_idx, x, topk_id, topk_w, 0, n_rows, replica};
    g.n = 1;
    const size_t xrb = (size_t)d * (cfg.x_dtype == CEP_F32 ? 4 : 2);
    HIPCHK(c, launch_ingest(a, g, k, E, cfg.max_tokens_per_replica, xrb, c->d_err, s));
    const bool split = c->wk == kWBf16 && A == kBf16TileM;
    const int split_tiles = split ? 2 * E : 0;
    const bool var = batch_var_tiles(c->wk, A, P, E);
    const bool stream = batch_stream_tiles(c->wk, A, P, E);
    const int tiles = std::min(tiles_cap, (P + A - 1) / A + E);
    HIPCHK(c, launch_route(a, sc, 0, n_rows, k, E, A, P, mpad, tiles_cap, 0, cfg.x_dtype, c->wk,
                           d, split ? c->n_cu : 0, 2 * I / kBf16TileN,
                           var ? kListVar : stream ? kListSorted : kListNone, c->d_err, s));
    BlobTable bt{};
    for (int e = 0; e < E; ++e) bt.blob[e] = c->w_res + (size_t)e * c->L.bytes;
    const Arena *gather = packed ? nullptr : &a;
    HIPCHK(c, launch_gemm1(sc, 0, tiles_cap, tiles, split_tiles, A, var, stream, bt, c->L, c->wk,
                           d, I, gather, 0, k, s));
    HIPCHK(c, launch_gemm2(sc, 0, tiles_cap, tiles, split_tiles, A, var, stream, bt, c->L, c->wk,
                           d, I, out, s));
    HIPCHK(c, launch_combine(a, sc, 0, n_rows, k, d, c->wk == kWBf16, gemm2_writes_solo(c->wk, A),
                             out, s));
  }
  return CEP_OK;
}
