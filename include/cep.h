/*
 * cep.h -- C ABI of libcep, the per-GPU streamFFN routed-expert path of
 * CascadeEP ("Asynchronous Expert Execution for MoE Prefill under Attention
 * Imbalance") for AMD Instinct MI355X (gfx950).
 *
 * One GPU holds E local experts (its expert-parallel share).  Routed token
 * chunks arrive from R attention replicas at different times (Section 3.2,
 * "Asynchronous EP and streaming FFN"; Appendix C, "Asynchronous dispatch").
 * The library batches ready chunks under a launch policy (Section 3.2,
 * "Launch threshold"), and runs every batch as one grouped FFN invocation
 * on one of several HIP streams (Section 3.2, "Multi-stream execution"):
 *
 *   1. histogram of local expert ids over the batch's valid (token, slot) pairs
 *   2. exclusive scan -> per-expert row offsets, aligned to the GEMM M tile
 *   3. stable permute/pack of token rows into expert-contiguous order, with an
 *      inverse map (e4m3 / MXFP4 weights: activations quantised to MXFP8 on
 *      the way)
 *   4. grouped gate/up GEMM with fused SwiGLU (e4m3 / MXFP4 weights: h
 *      re-quantised to MXFP8)
 *   5. grouped down GEMM, scaled by the routing coefficient
 *   6. combine: each source token's local contributions summed in slot order
 *      and written to its (replica, token) row of the output (e4m3 / MXFP4
 *      weights: step 5 writes the row of a token with one local pair itself,
 *      with the same value)
 *   (steps 1-6: Appendix C, "Grouped FFN invocations" and "Output return and
 *   combine").
 *
 * The single-GPU part of opportunistic expert weight fetching (Section 3.3;
 * Appendix C, "One-shot weight fetching") is a side-stream device-to-device
 * copy of whole expert weight blobs into a preallocated buffer; the fetched
 * experts' grouped GEMMs of a batch run after its resident experts' GEMMs,
 * gated by the copy, so the copy overlaps the resident work.
 *
 * Conventions for every entry point:
 *   - Return value: CEP_OK or a negative cep_status.  Nothing aborts or
 *     throws across the ABI.  cep_last_error() gives a message for the last
 *     failure on a context (HIP failures carry hipGetErrorString text).
 *   - "device" pointers are HIP device memory on the context's device;
 *     "host" pointers are ordinary host memory.  Dense arrays are row-major.
 *   - A context is used by one host thread at a time.
 *   - Work is enqueued asynchronously; only cep_destroy, cep_get_stats,
 *     cep_get_batch_routing and cep_get_status wait for the GPU.
 */
#ifndef CEP_H
#define CEP_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct cep_ctx cep_ctx; /* opaque, library-owned */

enum cep_status {
  CEP_OK = 0,
  CEP_EINVAL = -1, /* bad argument: shape, id, pointer, dtype, unknown batch */
  CEP_ENOMEM = -2, /* allocation failed, or a size exceeds a configured capacity */
  CEP_EHIP = -3,   /* a HIP runtime call failed (message in cep_last_error) */
  CEP_ESTATE = -4, /* call not valid in the current layer state / generation */
  CEP_EBUSY = -5   /* the one weight fetch of this layer was already issued */
};

enum cep_dtype {
  CEP_F32 = 0,          /* float32 (converted to bf16 inside the library)     */
  CEP_BF16 = 1,         /* bfloat16                                            */
  CEP_FP8_E4M3_B128 = 2, /* weights only: OCP e4m3fn codes, one float32 scale
                           per 128x128 block; activations and h run as MXFP8
                           (e4m3, one E8M0 scale per 32) inside the library */
  CEP_MXFP4 = 3          /* weights only: OCP MXFP4 (e2m1 codes, one E8M0 scale
                           per 32 along K; Section 4.1's DeepSeek-V4 experts);
                           activations and h run as MXFP8 inside the library */
};

/* How cep_weight_fetch brings a fetched expert's weights (Appendix C,
 * "One-shot weight fetching"; "FFN reassignment commit and fallback"). */
enum cep_fetch_mode {
  CEP_FETCH_COPY = 0,      /* copy the blobs into the fetch buffer on the side
                              stream; the experts' tiles wait for the copy.  A
                              copy that fails to start falls back to IN_PLACE */
  CEP_FETCH_IN_PLACE = 1,  /* no copy: the experts' tiles read the donor blobs
                              where they are (a peer region read in place)    */
  CEP_FETCH_FAIL_COPY = 2  /* test aid: behave as if the first copy failed to
                              start, which takes the fallback of COPY          */
};

enum cep_policy {
  CEP_WAIT_ALL = 0,  /* synchronous EP: one batch after every expected chunk  */
  CEP_PER_CHUNK = 1, /* asynchronous EP without threshold: one batch per chunk */
  CEP_THRESHOLD = 2  /* streamFFN: launch when pending pairs >= threshold      */
};

typedef struct {
  int d_model;                /* hidden size d, multiple of 256, <= 32768     */
  int d_ff;                   /* expert intermediate size I, mult. of 128, <= 32768 */
  int n_local_experts;        /* E, 1..64                                     */
  int top_k;                  /* k routing slots per token, 1..16             */
  int max_replicas;           /* R_max                                        */
  int max_tokens_per_replica; /* T_max; also the row stride of `out` per replica */
  int w_dtype;                /* cep_dtype of the expert weights              */
  int x_dtype;                /* cep_dtype of the token rows (F32 or BF16)    */
  int n_streams;              /* stream slots for batches, 1..8               */
  int max_pairs_per_batch;    /* capacity of one batch in valid pairs; 0 means
                                 max_replicas * max_tokens_per_replica * top_k */
  size_t fetch_buffer_bytes;  /* capacity of the temporary weight buffer      */
  int record_routing;         /* nonzero: keep every batch's routing metadata
                                 for cep_get_batch_routing (test/debug aid)   */
} cep_config;

/* Expert weights, device memory.
 * F32 / BF16 / FP8, math orientation (y = x W):
 *   w_gate, w_up : [E][d][I]     w_down : [E][I][d]   (element type w_dtype)
 *   FP8 only, float32 block scales (value = code * scale of its block):
 *   s_gate, s_up : [E][d/128][I/128]   s_down : [E][I/128][d/128]
 * MXFP4, output-major with K packed (the layout MX checkpoints use for a
 * linear layer's weight), two e2m1 codes per byte, the even K in the low
 * nibble, and uint8 E8M0 scales (2^(s-127)) per 32 consecutive K:
 *   w_gate, w_up : [E][I][d/2]   s_gate, s_up : [E][I][d/32]
 *   w_down       : [E][d][I/2]   s_down       : [E][d][I/32]
 * Scale pointers are unused (may be NULL) for F32 and BF16.                  */
typedef struct {
  const void *w_gate, *w_up, *w_down;
  const void *s_gate, *s_up, *s_down; /* float32 (FP8) or uint8 E8M0 (MXFP4) */
} cep_weights;

/* Bytes of one expert's packed weight blob (the library's device layout of
 * gate/up, down and scales).  0 if cfg is invalid.  The unit of a weight
 * fetch (Appendix C, "One-shot weight fetching": experts are copied whole). */
size_t cep_packed_expert_bytes(const cep_config *cfg);

/* Pack experts [first, first+n) of w into dst (device, n blobs back to back,
 * n * cep_packed_expert_bytes bytes, caller-owned).  Builds the weight region
 * a donor GPU would hold.  Enqueued on stream s; w must stay valid until then. */
int cep_pack_experts(const cep_config *cfg, const cep_weights *w, int first, int n,
                     void *dst, hipStream_t s);

/* Create a context: validates cfg, allocates every scratch buffer, the chunk
 * arena and the fetch buffer, creates the streams, and packs the weights of
 * resident experts into library-owned memory.  The library's streams are
 * non-blocking streams at default priority.  HIP runs a process's streams on
 * at most GPU_MAX_HW_QUEUES hardware queues (4 by default) and streams that
 * share a queue run its packets in order: a batch waiting for a late chunk
 * then also holds back the other streams on its queue.  A process with more
 * streams in use than that should raise GPU_MAX_HW_QUEUES (it is read when
 * HIP initialises).  These are the expert weights
 * every grouped invocation reads (Appendix C, "Grouped FFN invocations"),
 * and the preallocated temporary weight buffer of a helper (Appendix C,
 * "One-shot weight fetching": its capacity bounds the fetch byte budget).
 * resident: host [E] flags, NULL = all resident; an expert with flag 0 has
 * no local weights (its weights live with a donor, Section 3.3) and its work
 * can only run after cep_weight_fetch brings them (w is not read for it).
 * Synchronises s before returning, so the caller may free w after.  Errors:
 * CEP_EINVAL for a bad cfg or NULL weights, CEP_ENOMEM when a device
 * allocation fails, CEP_EHIP; *out is NULL then (message in
 * cep_last_error(NULL)). */
int cep_init_experts(cep_ctx **out, const cep_config *cfg, const cep_weights *w,
                     const uint8_t *resident, hipStream_t s);

/* Launch policy (Section 3.2; baselines of Section 4.3).  threshold_pairs is
 * theta in valid local (token, slot) pairs, used by CEP_THRESHOLD (>= 1).
 * n_streams in 1..cfg.n_streams.  Only between layers (CEP_ESTATE otherwise). */
int cep_set_policy(cep_ctx *ctx, int policy, int threshold_pairs, int n_streams);

/* Open layer `generation` (Appendix C, "Asynchronous dispatch": each
 * dispatch instance carries a generation tag, and every chunk submitted for
 * this layer must carry it; "Output return and combine": the next layer is
 * admitted only after the previous one's outputs are in, so the previous
 * layer must have been combined, CEP_ESTATE otherwise).  n_replicas <= R_max;
 * chunks_per_replica: host [n_replicas], the number of chunks each replica
 * will submit (the final flush of Section 3.2, "Launch threshold", fires
 * after the last of them).  out: device float32 [n_replicas][T_max][d],
 * caller-owned; the combine writes each delivered token's row once (its sum
 * over local slots) and leaves the rows of tokens never delivered untouched
 * (pass zeroed memory for y = 0 there; a zero fill of every row would cost as
 * much HBM traffic as the combine itself).  `out` must stay valid until
 * cep_combine's event completes.  Errors: CEP_EINVAL for a bad n_replicas,
 * a negative chunk count or a NULL pointer. */
int cep_begin_layer(cep_ctx *ctx, uint32_t generation, int n_replicas,
                    const int *chunks_per_replica, float *out);

/* Submit one chunk of replica `replica`'s routed tokens (a dispatch lane
 * becoming ready, Appendix C).  Device arrays, borrowed until the batch that
 * contains the chunk has finished (cep_combine's event covers all):
 *   token_idx [n_rows] int32 token slot in [0, T_max), each (replica, token)
 *             at most once per layer
 *   x         [n_rows][d] rows (x_dtype), 16-byte aligned.  With bf16 rows
 *             and bf16 weights the first grouped GEMM reads them in place
 *             (no packed copy): keeping a layer's chunks in one receive
 *             region keeps that gather within few pages
 *   topk_id   [n_rows][k] int32 local expert id in [0, E) or -1 (remote slot)
 *   topk_w    [n_rows][k] float32 routing coefficients
 * n_pairs: host-known count of valid (id >= 0) entries.  arrival: event after
 * which the data is valid (NULL: valid now).  The wait is enqueued here, on
 * the stream of the batch that will hold this chunk, so that only that
 * batch waits for it (a chunk becomes eligible on its own signal, not behind
 * other replicas' chunks); the event may be recorded again afterwards.  The
 * chunk's metadata is read when its batch launches (all chunks of a batch in
 * one staging launch).  May launch batches per policy; never blocks.
 * chunk_id (optional) receives the chunk's sequence number.
 * Errors: CEP_ESTATE for a wrong generation or a closed layer, CEP_EINVAL
 * for bad sizes, CEP_ENOMEM if the layer's rows exceed the arena
 * (R_max * T_max rows) or n_pairs exceeds max_pairs_per_batch; nothing of
 * the chunk is recorded then.  CEP_ESTATE also when a batch would launch
 * while an expert without resident weights has no fetch this layer: the
 * chunk is recorded and stays pending (cep_weight_fetch, then cep_flush,
 * launch it).  Ids outside [-1, E) or a wrong n_pairs are detected on the
 * device and reported by cep_get_status. */
int cep_submit_chunk(cep_ctx *ctx, uint32_t generation, int replica, int n_rows, int n_pairs,
                     const int32_t *token_idx, const void *x, const int32_t *topk_id,
                     const float *topk_w, hipEvent_t arrival, int64_t *chunk_id);

/* Launch everything pending now (explicit final flush, Section 3.2).
 * No-op when nothing is pending.  CEP_ESTATE as for cep_submit_chunk when an
 * expert without resident weights has no fetch this layer. */
int cep_flush(cep_ctx *ctx);

/* One-shot weight fetch (Section 3.3, Algorithm 1's AsyncFetch; Appendix C,
 * "One-shot weight fetching").  Copies the packed blobs src_blobs[i] (device
 * pointers, each cep_packed_expert_bytes, e.g. from cep_pack_experts) of local
 * experts ids[i] into the context's fetch buffer on stream `side` and returns
 * a library-owned event `ready` that completes with the copy (side NULL: a
 * library stream).  In later batches of this layer, the grouped GEMMs of
 * these experts run after the batch's resident experts' GEMMs and wait for
 * `ready`; the resident experts' work is not delayed.  When the
 * fetch mode is CEP_FETCH_IN_PLACE, or a copy fails to start (Appendix C,
 * "FFN reassignment commit and fallback": a failed copy leaves the work
 * where it can run and triggers no new decision), nothing is copied: the
 * experts' tiles (still after the resident experts' GEMMs) read src_blobs
 * in place, *ready is NULL, and cep_get_stats
 * reports the fetch as in place (with "fallback" after a failed copy).  The
 * output is the same, bit for bit, in every mode.  One fetch per layer: a
 * second call returns CEP_EBUSY.  Total bytes above fetch_buffer_bytes:
 * CEP_ENOMEM and nothing is copied.  Duplicate or out-of-range ids:
 * CEP_EINVAL.  Batches launched before the fetch use the resident weights;
 * an expert without resident weights must be fetched before the first batch
 * of the layer launches.  src_blobs must stay valid until cep_combine's
 * `done` event completes (the layer barrier also waits for the copy). */
int cep_weight_fetch(cep_ctx *ctx, const int *ids, int n, const void *const *src_blobs,
                     hipStream_t side, hipEvent_t *ready);

/* Fetch mode of the following layers' cep_weight_fetch (enum cep_fetch_mode).
 * Only between layers (CEP_ESTATE otherwise); CEP_EINVAL for an unknown mode. */
int cep_set_fetch_mode(cep_ctx *ctx, int mode);

/* Layer barrier (Appendix C, "Output return and combine": the next layer is
 * admitted only after all outputs are in).  Flushes pending chunks, makes
 * stream s wait for every batch of the layer (and for the layer's weight
 * copy), and returns a library-owned event `done` (may be NULL) recorded on
 * s after which `out` is final.
 * Closes the layer.  CEP_ESTATE if the layer is not open or chunks are still
 * expected (call cep_flush first to end a layer early). */
int cep_combine(cep_ctx *ctx, hipStream_t s, hipEvent_t *done);

/* Routing metadata of batch `batch` of the last layer: the per-expert row
 * counts, the tile-aligned offsets and the inverse map of one grouped
 * invocation (Appendix C, "Grouped FFN invocations"), for checking against a
 * reference (requires cfg.record_routing; waits for that batch).  CEP_EINVAL
 * for an unknown batch, CEP_ESTATE if record_routing is off and an array
 * was asked for.  Host outputs, any may be NULL:
 *   align [1]: M-tile alignment A;  n_pairs [1]; n_rows [1]
 *   cnt [E]; off [E+1] unpadded; off_pad [E+1] A-aligned
 *   perm_src [n_pairs]: flat pair index (row_in_batch * k + slot) of each
 *            unpadded grouped row, expert-major, stable
 *   pos_of   [n_rows * k]: padded grouped row of each flat pair, -1 if remote
 *   chunks   [n_chunks_max]: chunk sequence numbers in the batch (n_chunks [1])
 * Sizes: call with NULL arrays first to read n_pairs / n_rows / n_chunks. */
int cep_get_batch_routing(cep_ctx *ctx, int batch, int *align, int *n_pairs, int *n_rows,
                          int32_t *cnt, int32_t *off, int32_t *off_pad, int32_t *perm_src,
                          int32_t *pos_of, int64_t *chunks, int *n_chunks);

/* Per-phase timing of the following layers' batches: on (default) records
 * a HIP event after each phase (routing, GEMM1, GEMM2, combine) on the batch
 * stream, each costing a few microseconds of launch gap; off reports the
 * batch start and the phase durations as -1 in cep_get_stats (the batch end
 * stays).  Only between layers (CEP_ESTATE otherwise). */
int cep_set_phase_timing(cep_ctx *ctx, int on);

/* Number of batches launched in the current (or last) layer. */
int cep_get_batch_count(const cep_ctx *ctx);

/* Timing of the last layer, for the measurements of Section 4.3 (per-chunk
 * latency, FFN throughput of streamed against synchronous launches) and the
 * readiness timing of Appendix A ("Timing and readiness gaps": when each
 * replica's inputs arrived).  Waits for the layer's work and writes a JSON
 * object to buf (host, cap bytes, NUL-terminated; CEP_ENOMEM if too small;
 * CEP_EINVAL for NULL): per batch its chunks,
 * rows, pairs, stream slot, start/end in ms from the layer's origin
 * (cep_begin_layer) and the durations of its routing, GEMM1, GEMM2 and
 * combine phases (HIP events on the batch stream between the launches; for
 * a batch with fetched experts also when its fetched experts' GEMMs started,
 * after the copy, and their GEMM1 and GEMM2 durations, -1 otherwise); per
 * chunk its arrival (when a timing event was given, else -1) in the same
 * clock; and the fetch (interval, bytes copied, experts, in place or not). */
int cep_get_stats(cep_ctx *ctx, char *buf, size_t cap);

/* Waits for all work and reads the device-side error word: CEP_OK, or
 * CEP_EINVAL if a submitted chunk had an id outside [-1, E) or a pair count
 * different from its n_pairs (message in cep_last_error).  Clears it. */
int cep_get_status(cep_ctx *ctx);

/* Message for the last failure on ctx ("" if none).  With ctx NULL: the last
 * failure, on the calling thread, of a call that had no context to hold it
 * (cep_init_experts, cep_pack_experts). */
const char *cep_last_error(const cep_ctx *ctx);

/* Wait for all work, release every resource.  NULL is a no-op. */
int cep_destroy(cep_ctx *ctx);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): one chunk
 * of replica `replica` run as a one-batch layer, i.e. what cep_begin_layer,
 * cep_submit_chunk (policy CEP_WAIT_ALL, arrival NULL) and cep_combine do,
 * with the same kernels and the same bits in `out`, enqueued on stream s.
 * Arguments as for cep_submit_chunk; out: device float32 [R_max][T_max][d]
 * as for cep_begin_layer (delivered rows written, others untouched).  All
 * scratch (the chunk's routing arrays, tile lists, grouped rows, h, expert
 * outputs) lives in one 64 MiB device array of the library, one per device,
 * so nothing is allocated or freed: CEP_ENOMEM (before any work) when the
 * chunk needs more.  The need is about (2*d_ff + 4*d) bytes per grouped row
 * with bf16 weights and rows ((2*d_ff + 6*d) with float32 rows, (d_ff + 3*d)
 * with e4m3 or MXFP4 weights), for n_pairs rows
 * plus up to one M tile (64 or 256 rows; 128 or 256 with e4m3 / MXFP4) of
 * padding per expert: about 2 K pairs at d = 4096, d_ff = 2048, 8 experts.
 * Every call on a device shares that array, and it keeps the last call's
 * contents: calls that overlap on one device (on different streams, or with
 * kernels of an earlier call still running on another stream) race.  Work of
 * the context's layers uses its own buffers and does not conflict.  Needs
 * every expert resident (CEP_ESTATE otherwise); n_pairs 0 does nothing.
 * Device-side checks (ids, token slots, the pair count) are reported by
 * cep_get_status. */
int cep_ffn_noalloc(cep_ctx *ctx, int replica, int n_rows, int n_pairs, const int32_t *token_idx,
                    const void *x, const int32_t *topk_id, const float *topk_w, float *out,
                    hipStream_t s);

/* ------------------------------------------------------------------------
 * FFN throughput profile (host only; no GPU work).
 *
 * streamFFN's launch threshold theta is the smallest profiled expert-token
 * count whose FFN throughput reaches a fraction rho of the observed peak
 * (Section 3.2, "Launch threshold"); the FFN latency model is
 * F(N) = N / (eta(N) * P_peak), eta(N) in (0, 1] the throughput normalised
 * to the observed peak P_peak (Section 3.3, Eq. ffn-throughput-latency).
 * Between profiled counts eta is linear in N; below the smallest profiled
 * count n_0, F(N) = F(n_0); above the largest, eta keeps its last value.
 * Failures return CEP_EINVAL / CEP_ENOMEM with a message in
 * cep_last_error(NULL).
 */
typedef struct cep_ffn_profile cep_ffn_profile;

/* n[count]: profiled expert-token counts, positive and strictly increasing;
 * tput[count]: FFN throughput measured at each, positive and finite, in
 * expert tokens per time unit (F is then in that unit).  Both host arrays,
 * copied.  *out receives a profile owned by the caller. */
int cep_profile_create(const int64_t *n, const double *tput, int count, cep_ffn_profile **out);

/* Observed peak throughput P_peak (0 for NULL). */
double cep_profile_peak(const cep_ffn_profile *p);

/* *theta = smallest profiled count with tput / P_peak >= rho, rho in (0, 1]. */
int cep_profile_theta(const cep_ffn_profile *p, double rho, int64_t *theta);

/* *eta = eta(N) for N >= 1. */
int cep_profile_eta(const cep_ffn_profile *p, int64_t N, double *eta);

/* *latency = F(N) for N >= 0 (F(0) = 0). */
int cep_profile_latency(const cep_ffn_profile *p, int64_t N, double *latency);

/* Release a profile; NULL is a no-op. */
void cep_profile_destroy(cep_ffn_profile *p);

/* ------------------------------------------------------------------------
 * Opportunistic expert weight fetching: the coordinator (host only).
 *
 * The joint plan S of one MoE layer over R ranks (each an attention replica
 * and an expert-parallel rank; Section 3.3).  Per rank: whether it still
 * computes attention (a candidate donor), its remaining attention time A
 * (Eq. attention-remaining) and dispatch latency D, the expert tokens N it
 * receives, and, once out of attention, the completion time T of its own FFN
 * work.  A donor's predicted completion is T_d(S) = A_d + D_d + F(N_d)
 * (Eq. donor-completion), F from an FFN profile.  All times share one clock
 * measured from the decision instant, in the profile's time unit.
 *
 * cep_oewf_select is Algorithm 1 (SelectWeights): the donor with the latest
 * T_d(S) among the other ranks still in attention (lowest rank on ties); its
 * experts that hold tokens of the helper, by descending tokens / bytes
 * (ascending id on ties), taken greedily while they fit the byte budget B_h.
 * One decision per rank per layer (Appendix C, "One-shot weight fetching");
 * the helper then copies the selected experts with cep_weight_fetch.
 * cep_oewf_evaluate is the cost-based reassignment test (Eqs.
 * swf-completion-times, swf-admission) on the latest plan, with the helper's
 * completion max{T_h(S), s_h + F(N_trans)} for a reassigned invocation
 * planned to launch s_h after the decision, s_h in [0, T_h(S)] (Appendix E;
 * alpha_h = max{0, s_h + F(N_trans) - T_h(S)} / F(N_trans)).
 * cep_oewf_commit applies an admitted decision only if the donor's and the
 * helper's plan entries are unchanged since the evaluation, the plan's
 * tokens are unclaimed and the donor has not submitted them (Appendix C,
 * "FFN reassignment commit and fallback"); then the donor's N and the
 * helper's T change together.  Otherwise execution stays with the donor.
 * Calls on one coordinator are serialised internally.  Failures return
 * CEP_EINVAL / CEP_ENOMEM / CEP_EBUSY with a message in cep_last_error(NULL).
 */
#define CEP_OEWF_MAX_EXPERTS 64

typedef struct cep_oewf cep_oewf;

typedef struct {
  int helper, donor;     /* donor -1: no candidate donor                      */
  int n_experts;         /* selected experts; 0 = empty selection (no fetch)  */
  int experts[CEP_OEWF_MAX_EXPERTS];     /* donor expert ids, selection order */
  int64_t tokens[CEP_OEWF_MAX_EXPERTS];  /* helper's tokens per selected expert */
  int64_t bytes;         /* bytes to fetch (sum of the selected b_e)          */
  int64_t plan_id;       /* the coordinator's record of this plan (-1: none)  */
} cep_oewf_fetch;

typedef struct {
  int admit;             /* Eq. swf-admission holds                           */
  double Td, Th;         /* T_d(S), T_h(S)                                    */
  double Td2, Th2;       /* T_d(S'), T_h(S')                                  */
  double alpha;          /* alpha_h                                           */
  int64_t plan_id, n_trans;
  uint64_t donor_version, helper_version; /* plan entries the test read       */
} cep_oewf_decision;

/* A coordinator for n_ranks ranks (1..4096) with FFN model F (copied). */
int cep_oewf_create(int n_ranks, const cep_ffn_profile *F, cep_oewf **out);

/* New layer: every rank may decide once more; earlier plans and decisions
 * become stale (they no longer commit).  Rank entries are kept. */
int cep_oewf_begin_layer(cep_oewf *o);

/* Set rank r's entry (times and counts >= 0); bumps its version. */
int cep_oewf_set_rank(cep_oewf *o, int r, int in_attention, double A, double D, int64_t N,
                      double T);

/* *t = T_r(S): the donor model while r is in attention, else its T. */
int cep_oewf_completion(cep_oewf *o, int r, double *t);

/* *t = max_r T_r(S). */
int cep_oewf_makespan(cep_oewf *o, double *t);

/* Algorithm 1 for helper h.  tokens: host [n_ranks][n_experts], tokens h
 * dispatched to expert e of rank d; expert_bytes: host [n_experts] (> 0),
 * bytes of one expert's weights and scales; budget: B_h bytes.  n_experts
 * <= CEP_OEWF_MAX_EXPERTS.  CEP_EBUSY if h already decided this layer. */
int cep_oewf_select(cep_oewf *o, int helper, int n_experts, const int64_t *tokens,
                    const int64_t *expert_bytes, int64_t budget, cep_oewf_fetch *plan);

/* Reassignment test for moving n_trans (0 <= n_trans <= min(plan tokens,
 * N_d)) of a plan's unstarted tokens to its helper, launched s_h after the
 * decision.  Changes nothing. */
int cep_oewf_evaluate(cep_oewf *o, const cep_oewf_fetch *plan, int64_t n_trans, double s_h,
                      cep_oewf_decision *dec);

/* Version-checked commit; *committed = 1 if applied, 0 on fallback (also
 * for a decision taken before the last cep_oewf_begin_layer). */
int cep_oewf_commit(cep_oewf *o, const cep_oewf_decision *dec, int donor_submitted,
                    int *committed);

/* Release a coordinator; NULL is a no-op. */
void cep_oewf_destroy(cep_oewf *o);

#ifdef __cplusplus
}
#endif
#endif /* CEP_H */
