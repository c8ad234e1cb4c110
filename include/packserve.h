/*
 * packserve.h -- C ABI of the MI355X (gfx950) window scorer for PackServe's
 * KVC-first, SLO-aware request packing (Algorithm 1 of the paper).
 *
 * One call scores a whole scheduling window: for every request of the window
 * and every serving instance it finds the longest cached block prefix, runs
 * the white-box latency model (prefill Eq. 7 with the empirical C and C^2
 * terms of Sec. 5.3, decode Eq. 8 per batch-size segment with its EMA factor,
 * the TPOT estimate of Eq. 10, the TTFT decomposition of Eq. 4), applies the
 * capacity guard, the normalised recomputation filter of Eq. 9 and the TPOT
 * filter, and picks the instance with the decode-batch-size-centric key
 * (Sec. 6.2, D-C-Q of Table 4) or, when no instance meets the TPOT target,
 * the cache-aware load-balancing fallback (the LMetric product, Sec. 7 and
 * Sec. 8.1).  Every request of a window is scored against the same instance
 * snapshot; ps_commit then applies the chosen placements in order.
 *
 * Conventions shared by every entry point:
 *   - Return value: PS_OK (0) or a negative PS_E_* code.  Nothing is thrown
 *     or aborted across the ABI; ps_last_error() gives the message.  On an
 *     error the outputs are unspecified and the context state is unchanged.
 *   - Host pointers are owned by the caller; the library copies what it
 *     needs before returning and keeps no pointer to them.
 *   - "_dev" entry points take device pointers owned by the caller, enqueue
 *     work on the given HIP stream (NULL = the default stream) and return
 *     without waiting; the caller synchronises.  They use the context's
 *     tables and scratch, so two calls on one context must not overlap.
 *   - A context is not thread-safe; separate contexts are independent.
 *   - Block hashes are nonzero 64-bit values (0 is the empty-slot sentinel).
 *     A request's chain is pool[pre_off, pre_off + pre_len) followed by
 *     pool[tail_off, tail_off + tail_len): chained hashes, so one hash names
 *     a whole prefix, as a node of a prefix tree does.
 */
#ifndef PACKSERVE_H
#define PACKSERVE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define PS_OK 0
#define PS_E_INVAL (-1)  /* bad argument: null pointer, zero hash, malformed CSR/model */
#define PS_E_NOMEM (-2)  /* device or host allocation failed */
#define PS_E_DEVICE (-3) /* a HIP call failed */
#define PS_E_STATE (-4)  /* call order: scoring or commit before ps_load_instances */
#define PS_E_RANGE (-5)  /* a value is outside the limits below */

/* limits (validated) */
#define PS_MAX_SEG 32          /* decode batch-size segments */
#define PS_MAX_INST 65536      /* instances: ids fit the 16-bit key field */
#define PS_MAX_DQ 4095         /* decoding / queued requests per instance */
#define PS_MAX_CHAIN 16777215  /* blocks per request chain (2^24 - 1) */
#define PS_MAX_PENDING 17179869184LL  /* pending prefill tokens per instance (2^34) */
#define PS_MAX_CONTEXT 70368744177664LL /* context tokens per instance (2^46) */
#define PS_MAX_BLOCK_TOKENS 1024
#define PS_MAX_BATCH 8191      /* B_max */
#define PS_MAX_TABLE_CAP 67108864 /* distinct cached blocks per instance (2^26) */

/*
 * ps_model.flags.  The admission layers of the paper's layer ablation
 * (Table 3) are: G = NO_KVC_FILTER | NO_TPOT_FILTER, C = NO_TPOT_FILTER,
 * T = NO_KVC_FILTER | FALLBACK_DCQ, CT = FALLBACK_DCQ, F (full) = 0.
 */
#define PS_F_TTFT_ADMIT 1u     /* also require predicted TTFT <= the TTFT budget for T */
#define PS_F_NO_KVC_FILTER 2u  /* skip the recomputation filter: C = A */
#define PS_F_NO_TPOT_FILTER 4u /* skip the TPOT test: T = C (minus TTFT admission if on) */
#define PS_F_FALLBACK_DCQ 8u   /* when T is empty choose over C by the D-C-Q key, not LMetric */
/*
 * Selection order within T (bits 8..11 of flags; the selector ablation of
 * Table 4, plus LMetric alone).  D = most decoding requests, C = most cached
 * blocks, Q = fewest queued requests, H = smallest TPOT headroom
 * (tpot_slo - predicted TPOT); every order ends with the lowest id.  RANDOM
 * takes the k-th member of T in id order, k = floor(z_hi * |T| / 2^32) with
 * z the (r + 1)-th output of a SplitMix64 stream seeded with rand_seed for
 * request r of the window.
 */
#define PS_SEL_DCQ 0u
#define PS_SEL_D 1u
#define PS_SEL_DQ 2u
#define PS_SEL_DC 3u
#define PS_SEL_DQC 4u
#define PS_SEL_HCQ 5u
#define PS_SEL_RANDOM 6u
#define PS_SEL_LMETRIC 7u
#define PS_F_SELECTOR(sel) ((uint32_t)(sel) << 8)

/* ps_result.flags */
#define PS_R_REJECT 1u    /* no capacity-eligible instance (Algorithm 1 returns Reject) */
#define PS_R_FALLBACK 2u  /* T was empty: chosen by the load-balancing fallback over C */
#define PS_R_TTFT_MISS 4u /* predicted TTFT of the choice exceeds the TTFT budget */
#define PS_R_INVALID 8u   /* (_dev only) malformed request descriptor; instance -1 */

typedef struct ps_ctx ps_ctx; /* opaque: device tables, instance state, stream */
typedef int32_t ps_status;

/*
 * Pool-wide latency profile and policy; copied at load.
 *  alpha: prefill model T_pf(N, C) = a0 + a1 N + a2 N C + a3 N^2 + a4 C + a5 C^2,
 *         seconds, N new and C cached tokens (Eq. 7 plus the C, C^2 terms of
 *         Sec. 5.3).
 *  seg_ub[0..n_seg): inclusive upper batch size of each decode segment,
 *         strictly ascending (CUDA-graph capture sizes in the paper, Sec. 5.3);
 *         a projected batch above the last bound uses the last segment.
 *  beta[s], gamma[s]: decode iteration T_iter(B, S) = gamma_s (b0 + b1 B + b2 S)
 *         (Eq. 8 per segment; gamma_s is the EMA factor of Sec. 5.3, > 0).
 *  eta: recomputation budget (>= 0, Eq. 9); tpot_slo: TPOT target tau (s,
 *         strict test); ttft_floor: minimum TTFT budget (s; the budget is
 *         max(floor, T_pf(L, 0)), Sec. 8.1); lout: recent median output length
 *         (tokens; the interference term divides by max(1, lout), Eq. 10).
 *  block_tokens: tokens per block; b_max: engine batch limit; kv_cap_tokens:
 *         KV capacity in tokens (capacity guard: A_i + 1 <= b_max and
 *         S_i + L <= kv_cap_tokens).
 *  flags: PS_F_* and PS_F_SELECTOR(PS_SEL_*).
 *  rand_seed: seed of the random selector's stream.
 */
typedef struct {
  float alpha[6];
  int32_t n_seg;
  int32_t seg_ub[PS_MAX_SEG];
  float beta[PS_MAX_SEG][3];
  float gamma[PS_MAX_SEG];
  float eta, tpot_slo, ttft_floor, lout;
  int32_t block_tokens, b_max;
  int64_t kv_cap_tokens;
  uint32_t flags;
  uint64_t rand_seed;
} ps_model;

/*
 * Instance snapshot (host memory).  Instance i caches the block hashes
 * blk[blk_off[i], blk_off[i+1]) (set semantics: duplicates allowed, order
 * irrelevant; at most table_cap_blocks per row; blk_off[0] = 0, ascending).
 * decoding = D_i, queued = Q_i (both in [0, PS_MAX_DQ]; A_i = D_i + Q_i),
 * pending_tok = P_i (pending uncached prefill tokens), ctx_tok = S_i (context
 * tokens of the A_i active requests).  table_cap_blocks also bounds later
 * inserts by ps_commit.
 */
typedef struct {
  int32_t n_inst, table_cap_blocks;
  const int64_t* blk_off;
  const uint64_t* blk;
  const int32_t* decoding;
  const int32_t* queued;
  const int64_t* pending_tok;
  const int64_t* ctx_tok;
} ps_instances;

/* One request: chain = pool[pre_off..+pre_len) ++ pool[tail_off..+tail_len). */
typedef struct {
  int64_t pre_off;
  int64_t tail_off;
  int32_t pre_len;
  int32_t tail_len;
} ps_req;

/* One decision (20 bytes).  instance -1 = Reject (hit 0, ttft = tpot = 0). */
typedef struct {
  int32_t instance;
  int32_t hit_blocks;
  float ttft;
  float tpot;
  uint32_t flags;
} ps_result;

/* Create a context on HIP device `device` (owns a default-priority stream). */
ps_status ps_create(int device, ps_ctx** out);

/* Free every device buffer and the stream.  NULL is accepted. */
ps_status ps_destroy(ps_ctx* ctx);

/*
 * Replace the snapshot: what Algorithm 1 reads about the instance pool.  The
 * cached block sets stand for each instance's local prefix tree (Sec. 7: the
 * scheduler keeps a prefix tree per instance and asks it for the longest
 * cached prefix); the counters D_i, Q_i, P_i, S_i are the scheduler-
 * observable instance state and the model the configuration profile that
 * Sec. 5.1 names as the latency model's inputs (Eqs. 4, 7, 8, 10).
 * Builds one open-addressing table per instance from the CSR block lists
 * (buckets of 8 x 64-bit slots, at least 2 * table_cap_blocks slots, a
 * per-instance salted bucket index) and uploads the load counters and the
 * model.  Synchronous.  PS_E_INVAL on a null pointer, a zero hash, a
 * malformed CSR or model; PS_E_RANGE when a limit above is exceeded.
 */
ps_status ps_load_instances(ps_ctx* ctx, const ps_instances* inst, const ps_model* model);

/*
 * Algorithm 1 (Sec. 6) for every request of a window: its input is the
 * request, the instance pool with its state, eta and tau; its output the
 * chosen instance or Reject; here each request's result also carries the
 * prefix hit and the predicted TTFT (Eq. 4) and TPOT (Eq. 10) of the choice.
 * Score a window held in host memory: copies pool[0, pool_len) and reqs to
 * the device, runs ps_score_window_dev on the context stream and copies the
 * n_req results back.  Synchronous.  Descriptors must lie inside the pool,
 * chains must be at most PS_MAX_CHAIN blocks and the pool free of zero
 * hashes (PS_E_RANGE / PS_E_INVAL otherwise).  n_req = 0 is a no-op.
 */
ps_status ps_score_window(ps_ctx* ctx, const uint64_t* pool, int64_t pool_len,
                          const ps_req* reqs, int32_t n_req, ps_result* out);

/*
 * Algorithm 1 (Sec. 6) for every request of a device-resident window, as
 * ps_score_window.  d_sizes is an addition to the boundary Algorithm 1
 * implies: the sizes of its candidate sets (capacity-eligible, after the
 * recomputation filter of Eq. 9, after the TPOT filter) are what the
 * parity tests check beside the decision, and a caller can read how many
 * instances each filter kept.  Pass NULL to skip them (the faster path).
 * Score a device-resident window into d_out[n_req] (and, if d_sizes is not
 * NULL, |A|, |C|, |T| per request into d_sizes[3 * n_req]), asynchronously
 * on `hip_stream`.  Descriptors are checked by the kernel: a malformed one
 * yields instance -1 with PS_R_INVALID.  A zero hash in a chain never
 * matches (it ends the prefix walk).  Requests with the same pre_off share
 * one walk of that segment per window (identical results); the context
 * keeps a group table for that, grown (hipMalloc) when a window has more
 * requests than any before it: under 620 bytes per request, none for
 * windows above 4,194,304 requests, which are scored without it.  Calls
 * that overlap on one context (two streams) race on that table.
 */
ps_status ps_score_window_dev(ps_ctx* ctx, const uint64_t* d_pool, int64_t pool_len,
                              const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                              uint32_t* d_sizes, void* hip_stream);

/*
 * ps_score_window_dev without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, results and asynchrony as
 * ps_score_window_dev (byte-identical results); the window's prefix-group
 * table lives in a fixed device array of about 37 MiB per GPU instead of
 * memory the context grows, set up by the first ps_create on the device and
 * held until the process ends.  No hipMalloc, hipFree, memset node or event
 * is issued (timing is not recorded).  Limit: n_req <= 65,536 per call
 * (PS_E_RANGE above; split larger windows); at most 16 MiB of popular-group
 * hit rows (a group beyond them takes the per-request path, same results).
 * Every call on one GPU, from any context, shares that array and leaves its
 * contents to the next: calls that overlap on one GPU (two streams, two
 * threads, two contexts) race.  PS_E_STATE if the context has no snapshot
 * or the array was not set up on its device.
 */
ps_status ps_score_window_dev_fixed(ps_ctx* ctx, const uint64_t* d_pool, int64_t pool_len,
                                    const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                                    uint32_t* d_sizes, void* hip_stream);

/*
 * Measurement: with on != 0, the next ps_score_window(_dev) calls (up to
 * 4,096 of them) record HIP events on their stream around their launches:
 * the prefix-group pass (claim, walk) and the scoring pass (lean scorer,
 * general scorer).
 * ps_read_timing waits for those calls and returns their number and the
 * mean duration of each part in milliseconds, then starts a new count.
 * PS_E_STATE if no call was recorded.  Switching it on or off resets the
 * count.  The events are kept until ps_destroy.
 */
ps_status ps_set_timing(ps_ctx* ctx, int32_t on);
ps_status ps_read_timing(ps_ctx* ctx, int32_t* n_calls, float* ms_group, float* ms_score);

/*
 * Measurement, per kernel: like ps_read_timing (same recorded calls; it
 * starts a new count too), but ms[0..3] receive the mean milliseconds of the
 * four launches of a scoring call: the group claim pass, the group walk, the
 * lean scorer and the general scorer (0 for a launch the call did not make).
 * ms points to 4 host floats.
 */
ps_status ps_read_kernel_timing(ps_ctx* ctx, int32_t* n_calls, float* ms);

/*
 * Diagnostic: the longest cached prefix (blocks) of every request on every
 * instance, ignoring capacity, into d_hits[r * n_inst + i], asynchronously on
 * `hip_stream`.  Same prefix walk as the scorer.  Malformed descriptors give
 * 0xFFFFFFFF rows.
 */
ps_status ps_probe_hits_dev(ps_ctx* ctx, const uint64_t* d_pool, int64_t pool_len,
                            const ps_req* d_reqs, int32_t n_req, uint32_t* d_hits,
                            void* hip_stream);

/*
 * Algorithm 1 per arrival (Sec. 6 and 7 of the paper: one request at a time,
 * the request path updating the chosen instance's counters and prefix tree
 * before the next request is routed).  The device-resident window's
 * requests are taken in array order; request r is scored against the state
 * left by requests 0..r-1 (same scoring as ps_score_window_dev) and, when
 * placed, committed as ps_commit would commit it, before request r + 1 is
 * scored.  Results into d_out[n_req]; |A|, |C|, |T| into d_sizes[3 * n_req]
 * if not NULL; blocks refused at the table cap into *n_dropped (host, may
 * be NULL).  Malformed descriptors yield PS_R_INVALID and change nothing.
 * Zero hashes in a chain are never inserted (nor counted as refused).
 * Runs on `hip_stream` and returns once the window is scheduled and the
 * context holds the final state.  PS_E_RANGE, before any change, if B_max
 * or M_KV would let a counter leave its limit (B_max - 1 - D_i above
 * PS_MAX_DQ; P_i or S_i plus M_KV - S_i above its limit).
 */
ps_status ps_schedule_window_dev(ps_ctx* ctx, const uint64_t* d_pool, int64_t pool_len,
                                 const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                                 uint32_t* d_sizes, int64_t* n_dropped, void* hip_stream);

/*
 * Device memory the two calls above may hold for the hits of the requests
 * one launch schedules (n_inst x 4 bytes per request): a window whose hits
 * exceed it is scheduled in several launches, in order, with identical
 * results.  0 restores the default, 256 MiB; any budget admits at least one
 * request per launch.  The memory is kept by the context until ps_destroy.
 */
ps_status ps_set_schedule_budget(ps_ctx* ctx, int64_t bytes);

/*
 * Speculative batches of ps_schedule_window_dev (Algorithm 1 per request,
 * Sec. 6, with the state moving along the request path, Sec. 7, as above;
 * the results do not depend on this setting).  The requests are taken in
 * batches of `batch`: every request of a batch is first scored in parallel
 * against the state at the batch's start, keeping |A|, |C|, |T|, W_min and
 * the first members of T and of C in key order; then, in arrival order, the
 * instances that earlier requests of the batch were placed on are scored
 * again against the current state, and when they cannot change W_min and
 * the speculative lists show the least key, the request is decided from
 * them; otherwise it is scored in full.  batch in [1, 256]; 0 scores every
 * request in full (one workgroup, no speculation).  Default 256.  The
 * Random and H-C-Q selectors are always scored in full.  PS_E_INVAL for a
 * batch outside [0, 256].
 */
ps_status ps_set_schedule_speculation(ps_ctx* ctx, int32_t batch);

/*
 * Of the requests the last ps_schedule_window_dev call scored (every valid
 * descriptor), how many were decided from their speculative result
 * (*n_spec) and how many were scored in full (*n_full; both 0 without
 * speculation).  Host pointers, either may be NULL.  Synchronous.
 */
ps_status ps_read_schedule_stats(ps_ctx* ctx, int64_t* n_spec, int64_t* n_full);

/*
 * Replay given placements (device array d_inst[n_req], -1 = none) in array
 * order: for each placed request, d_out gets the instance, the hit, TTFT
 * and TPOT that instance offers at the request's arrival (the state left by
 * the earlier entries; no capacity test) and PS_R_TTFT_MISS when TTFT
 * exceeds the request's SLO; then the request is committed as ps_commit
 * does.  Entries with -1 yield PS_R_REJECT.  Measures what placements made
 * against one snapshot do to the requests that follow them.  PS_E_RANGE,
 * before any change, for an instance outside [-1, n_inst) or a counter that
 * would leave its limit.  Synchronous on `hip_stream` as above.
 */
ps_status ps_replay_window_dev(ps_ctx* ctx, const uint64_t* d_pool, int64_t pool_len,
                               const ps_req* d_reqs, int32_t n_req, const int32_t* d_inst,
                               ps_result* d_out, int64_t* n_dropped, void* hip_stream);

/*
 * The request-path update of the instance state (Sec. 7: the scheduler's
 * view of each instance, its counters and its prefix tree, is updated as
 * requests are routed, with no round trip to the engine).  pool_len is an
 * addition to the placements Algorithm 1 outputs: the chains are named by
 * offsets into the caller's hash pool, and its length lets every
 * descriptor be checked before any change.
 * Apply placements (host memory) in array order: entry k places request
 * reqs[k] on instance inst[k] (-1 = skip).  For each placed request, against
 * the table as left by the earlier entries: Q_i += 1, P_i += uncached tokens
 * (L - block_tokens * hit), S_i += L, and the chain's blocks enter
 * the table in chain order until table_cap_blocks distinct blocks are held;
 * refused blocks are counted in *n_dropped.  No eviction.  Synchronous.
 * PS_E_RANGE if a counter would leave its limit.
 */
ps_status ps_commit(ps_ctx* ctx, const uint64_t* pool, int64_t pool_len, const ps_req* reqs,
                    const int32_t* inst, int32_t n, int64_t* n_dropped);

/*
 * Copy the current load counters and per-instance distinct cached-block
 * counts to host arrays of n_inst entries (any pointer may be NULL).
 */
ps_status ps_read_state(ps_ctx* ctx, int32_t* decoding, int32_t* queued, int64_t* pending_tok,
                        int64_t* ctx_tok, int64_t* cached_blocks);

/*
 * Layout facts for measurement: slots per instance table, total table bytes,
 * and whether per-candidate prefix hits stay in LDS (1) or in device scratch
 * (0) for the loaded instance count.  Any pointer may be NULL.
 */
ps_status ps_table_info(ps_ctx* ctx, int64_t* slots_per_table, int64_t* table_bytes,
                        int32_t* hits_in_lds);

/*
 * Response-path feedback (Sec. 5.3 and Sec. 7 of the paper; applied in array
 * order, between windows, never concurrently with scoring).
 */

/* Instance state transitions along the response path. */
#define PS_EV_PREFILL_DONE 1  /* a queued request produced its first token: Q -= 1, D += 1,
                                 P -= tokens (the request's uncached prefill tokens) */
#define PS_EV_DECODE_TOKENS 2 /* the instance's decoding requests generated `tokens` tokens:
                                 S += tokens */
#define PS_EV_FINISHED 3      /* a decoding request completed: D -= 1, S -= tokens (its final
                                 context length) */
typedef struct {
  int32_t instance;
  int32_t kind;   /* PS_EV_* */
  int64_t tokens;
} ps_event;

/*
 * Apply events to the load counters in array order, then refresh the derived
 * per-instance data (capacity room, decode segment, key order).  PS_E_RANGE if
 * any counter would leave its limits (D, Q in [0, PS_MAX_DQ], P in
 * [0, PS_MAX_PENDING], S in [0, PS_MAX_CONTEXT]); PS_E_INVAL on an unknown
 * kind or instance.  On error no event is applied.  Synchronous.
 */
ps_status ps_apply_events(ps_ctx* ctx, const ps_event* events, int32_t n);

/*
 * Online calibration of the decode model (Sec. 5.3).  Sample k is a measured
 * pure-decode forward: batch size batch[k] >= 1, total context ctx_tok[k]
 * tokens, duration measured_s[k] > 0 seconds.  For its segment s (the
 * segment of batch[k]) the base prediction is b0 + b1 B + b2 S (no factor);
 * ratio = clip(measured / prediction, 0.5, 2); gamma_s = clip(0.98 gamma_s +
 * 0.02 ratio, 1, 2).  Samples whose base prediction is not positive are
 * skipped.  The factors are kept in double precision between calls and used
 * by the scorer in fp32.  PS_E_INVAL on a non-finite or non-positive
 * duration or a batch below 1.
 */
ps_status ps_feedback_decode(ps_ctx* ctx, const int32_t* batch, const int64_t* ctx_tok,
                             const float* measured_s, int32_t n);

/*
 * Recent median output length (the L_out of Eq. 10): record completed
 * requests' output lengths (tokens, >= 0) in order; L_out becomes the lower
 * median (element floor((m - 1) / 2) of the sorted values) of the last
 * m = min(recorded, PS_LOUT_WINDOW) lengths.  Before any sample the model's
 * lout stays.
 */
#define PS_LOUT_WINDOW 1024
ps_status ps_feedback_output(ps_ctx* ctx, const int32_t* out_len, int32_t n);

/* Current EMA factors (n_seg entries) and L_out; either pointer may be NULL. */
ps_status ps_read_model(ps_ctx* ctx, float* gamma, float* lout, int32_t* n_seg);

/* Message of the last failed call on ctx (or of ps_create when ctx is NULL). */
const char* ps_last_error(const ps_ctx* ctx);

/* Identity of this build: the first 16 hex digits of the SHA-256 of the
 * library's sources (the csrc files in name order, then this header), as
 * the build computed it, so a caller can tell a library built from other
 * sources; "unknown" for a build that did not pass one.  A static string,
 * never freed; no error case. */
const char* ps_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* PACKSERVE_H */
