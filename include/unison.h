/*
 * unison.h -- C ABI of libunison, a batched, trace-driven simulator of the
 * UNISON session-KV residency policy on AMD Instinct MI355X (gfx950).
 *
 * The library runs many independent two-tier (SRAM over HBM) KV-pool
 * simulations at once.  At every session event each simulation writes the
 * event into its session register file, scores every table entry with SPEAR
 * (Sec. III-B, eq. (esp)) or a baseline key, evicts the argmax victim while
 * the pool violates eq. (cap), and on a gap onset lets TIDE (Sec. III-C,
 * eq. (budget), eq. (promote), eq. (demote)) spend the expected idle window
 * as a DMA budget -- the joint loop of Algorithm 1.  Hit, miss, AMAT
 * (eq. (hr-amat)), prefill (eq. (prered)) and TTFT-proxy counters
 * accumulate per simulation.  Separate entry points expose the scorers, the
 * register-file EMA and the Kendall tau-b ranking-fidelity statistics of
 * Sec. IV-C and Sec. VI-F.
 *
 * Conventions (all entry points):
 *  - Every call returns UNISON_OK (0) or a negative UNISON_E_* code and never
 *    throws.  unison_last_error() gives a message for calls on a context.
 *  - Pointers documented DEVICE are device memory on the context's device;
 *    HOST pointers are ordinary host memory.  All of them are BORROWED: the
 *    caller keeps them alive and unmodified until the stream work that uses
 *    them has completed.
 *  - The library allocates no device memory.  All per-simulation state lives
 *    in a caller-owned workspace of unison_workspace_size() bytes.
 *  - Work is enqueued on the caller's HIP stream and is asynchronous, except
 *    where a call says it synchronises.
 *  - A context is not thread-safe; use one per host thread.
 *
 * Binary trace format (struct-of-arrays, one entry per event, events of one
 * trace contiguous and in processing order):
 *   ev_t_ns    uint64  event time in ns, non-decreasing within a trace
 *   ev_sid     uint32  session index within the trace, < its session count
 *   ev_info    uint32  (kind << 24) | turn; kind is UNISON_EV_*, turn is the
 *                      0-based turn index (ARRIVE: the turn that starts;
 *                      GAP_START / DONE: the turn that ended)
 *   ev_len     uint32  ARRIVE: resident KV length of the turn in tokens
 *                      (non-decreasing per session, eq. (reuse)); else 0
 *   ev_next_ns uint64  GAP_START: time of the session's next ARRIVE (read
 *                      only by the Belady policy); else UINT64_MAX
 *   ev_tool    uint32  GAP_START: tool class of the gap that starts, below
 *                      UNISON_ETA_CLASSES (read only by the ETA policy); else
 *                      ignored.  Optional: without it every gap is class 0
 *   sess_kvb   uint32  per session: KV bytes per token (eq. (cap) in bytes)
 * A session's events must run ARRIVE(0), GAP_START(0), ARRIVE(1), ...,
 * ARRIVE(T-1), DONE(T-1).  A simulation that meets an event breaking this
 * order stops there; its counters then carry error = event index + 1 and
 * unison_read_counters() returns UNISON_E_BAD_TRACE.
 */
#ifndef UNISON_H
#define UNISON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- codes */
#define UNISON_OK 0
#define UNISON_E_INVALID (-1)   /* null pointer, bad size, bad parameter */
#define UNISON_E_BAD_TRACE (-2) /* an event breaks the trace format */
#define UNISON_E_CAPACITY (-3)  /* a trace has more sessions than supported */
#define UNISON_E_HIP (-4)       /* a HIP runtime call failed */
#define UNISON_E_NOT_READY (-5) /* run before traces, tables and parameters */

#define UNISON_EV_ARRIVE 0u     /* turn k starts; for k >= 1 this is gap_end */
#define UNISON_EV_GAP_START 1u  /* turn k ended, another turn follows */
#define UNISON_EV_DONE 2u       /* the final turn ended */

#define UNISON_POLICY_SPEAR 0u   /* SPEAR score eq. (esp) (+ TIDE if enabled) */
#define UNISON_POLICY_LRU 1u     /* recency: evict the longest-idle session */
#define UNISON_POLICY_TIMEOUT 2u /* recency plus expiry after an idle TTL */
#define UNISON_POLICY_BELADY 3u  /* offline oracle: evict the farthest next request */
#define UNISON_POLICY_ETA 4u     /* tool-type arrival table: evict the farthest predicted
                                    return, gap onset + the expected wait of its tool class */
#define UNISON_POLICY_PARAMS 0xFFu /* unison_run: use each simulation's own policy */

#define UNISON_RUN_CONTINUE 1u   /* resume every simulation where the last run stopped */
#define UNISON_RUN_LOG 2u        /* also record decisions (see unison_read_log) */
#define UNISON_RUN_LOG_VICTIM 4u /* with UNISON_RUN_LOG: also record each event's scan
                                    result as a UNISON_OP_VICTIM record (a = victim or
                                    0xFFFFFFFF), written before that event's decisions */

#define UNISON_LUT_LEN 51u       /* hazard table entries, t = 0..50 (eq. (hazard)) */
#define UNISON_MAX_SESSIONS (1u << 20) /* largest session count of one trace */
#define UNISON_ETA_CLASSES 16u   /* tool classes of an ETA table */

/* Decision record operations; `b` holds the second session or the tier. */
#define UNISON_OP_EVICT 1u    /* a = victim (Alg. 1, capacity branch) */
#define UNISON_OP_EXPIRE 2u   /* a = session whose idle TTL ran out */
#define UNISON_OP_BYPASS 3u   /* a = arriving session served but not retained */
#define UNISON_OP_PROMOTE 4u  /* a = HBM resident moved into free SRAM (TIDE) */
#define UNISON_OP_SWAP 5u     /* a = promoted (eq. (promote)), b = demoted (eq. (demote)) */
#define UNISON_OP_VICTIM 6u   /* a = the event's scan result (UNISON_RUN_LOG_VICTIM only) */
#define UNISON_OP_PLACE 7u    /* a = arriving session, b = tier (1 SRAM, 2 HBM) */

typedef struct unison_ctx unison_ctx;

/* Register-file organisation (Sec. IV-B, eq. (rf), eq. (stale)): the unified
 * file, or two private copies -- the eviction engine's and TIDE's -- that are
 * overwritten with the live file after every request and gap onset, after every
 * 8th request, or at gap onsets only. */
#define UNISON_DUAL_NONE 0u
#define UNISON_DUAL_EVERY 1u
#define UNISON_DUAL_EIGHT 2u
#define UNISON_DUAL_GAP 3u

/* Sizes that fix the workspace. */
typedef struct {
  uint32_t n_sims;       /* simulations in the batch, >= 1 */
  uint32_t n_traces;     /* traces they replay, >= 1 */
  uint32_t max_sessions; /* largest session count of any trace, 1..UNISON_MAX_SESSIONS */
  uint32_t n_luts;       /* hazard tables, >= 1 */
  uint32_t log_cap;      /* decision records kept per simulation (0: no log) */
  uint32_t views;        /* 1: reserve the two register-file copies of the dual design
                            (64 B per session slot), needed by any row with dual_sync != 0 */
} unison_dims;

/* One simulation's parameters (eq. (cap), eq. (esp), eq. (budget),
 * eq. (hr-amat), eq. (lock)); host array of n_sims rows. */
typedef struct {
  uint32_t policy;         /* UNISON_POLICY_SPEAR .. UNISON_POLICY_ETA */
  uint32_t tide;           /* 1: TIDE pass on gap onsets while the DMA is free */
  uint32_t score_mode;     /* 0: fp32 score; 1: fixed-point score_q (SPEAR only) */
  uint32_t lut;            /* hazard table index, < n_luts */
  uint32_t trace;          /* trace index, < n_traces */
  uint32_t hazard_online;  /* 0: the table set by unison_set_hazard; 1: the table starts
                              empty and is rebuilt from the first online_sessions
                              completions, each DONE adding its session's turn count to
                              the counts of eq. (hazard) before that event's scan (the
                              online-convergence study of eq. (attainment)) */
  uint64_t cap_sram_B;     /* C_S in bytes */
  uint64_t cap_hbm_B;      /* C_H in bytes */
  uint64_t n_slots;        /* N_sess, >= 1 */
  uint64_t dma_B_per_us;   /* DMA bandwidth B in bytes per microsecond, >= 1 */
  uint64_t ttl_ns;         /* idle TTL of the timeout policy */
  double t_s_ns_per_B;     /* SRAM read cost t_s */
  double t_h_ns_per_B;     /* HBM read cost t_h */
  double t_p_ns_per_tok;   /* prefill cost t_p */
  float penalty_us;        /* completion penalty P of eq. (esp), >= 0, microseconds */
  uint32_t b_h;            /* hazard bits b_h, 6..16 (below 6, floor(eps Lambda + 1/2) = 0 and
                              sigma_q of eq. (survq) can reach 0, where eq. (t1) is undefined) */
  uint32_t b_g;            /* gap register bits b_g, 1..64 */
  uint32_t online_sessions; /* completions an online table counts (hazard_online = 1) */
  uint64_t tau_ns;         /* gap time divisor tau, >= 1 */
  uint64_t p_z;            /* integer penalty P_Z = P / tau */
  uint32_t dual_sync;      /* UNISON_DUAL_*: one live register file (0), or the dual design of
                              eq. (stale) whose eviction and TIDE engines decide from private
                              copies refreshed at the given points */
  uint32_t recip_bits;     /* score_mode 1: 0 divides eq. (t1) by sigma_q exactly; W in 1..32
                              multiplies by floor(2^W / sigma_q + 1/2) instead and shifts right
                              by W (a reciprocal table of depth Lambda: the divider-type axis of
                              the format sweep) */
} unison_sim_params;

/* Per-simulation results. */
typedef struct {
  uint64_t requests, hit_sram, hit_hbm, miss, bypass, evict, expire, promote, swap;
  uint64_t dma_bytes;         /* bytes TIDE migrated */
  uint64_t tide_passes;       /* TIDE passes started */
  uint64_t tokens_total;      /* sum of request lengths, eq. (prered) denominator */
  uint64_t tokens_computed;   /* tokens prefilled, eq. (prered) numerator */
  uint64_t extra_prefill_tok; /* prefix tokens re-prefilled after a loss */
  uint64_t score_evals;       /* the register-file scan's domain: sum over events of |table|
                                 (every entry the paper's scan covers) */
  uint64_t resident_evals;    /* sum over events of the resident count */
  uint64_t digest;            /* sum mod 2^64 of hashes of every decision record:
                                 mix(w0 ^ w1 * 0x9e3779b97f4a7c15), w0 = ev << 8 | op,
                                 w1 = a << 32 | b, mix = the SplitMix64 finaliser */
  uint64_t victim_digest;     /* sum over events e of (v + 1) * (2e + 1) * 0x9e3779b97f4a7c15
                                 mod 2^64, v = the event's scan result (argmax victim,
                                 0xFFFFFFFF when nothing is evictable) */
  uint64_t events;            /* events processed so far */
  uint64_t error;             /* 0, or 1 + index of the event that broke the format */
  uint64_t prefetch_hits;     /* SRAM hits on sessions TIDE moved into SRAM since their previous
                                 request (prefetch accuracy = prefetch_hits / (promote + swap)) */
  uint64_t vict_diff;         /* dual-view runs: evictions whose victim the live table would not
                                 have picked (eq. (stale)) */
  uint64_t prom_diff;         /* dual-view runs: TIDE moves whose promoted session the live
                                 table would not have picked */
  double amat_sum_ns;         /* sum of per-request access costs, eq. (hr-amat) */
  double ttft_sum_ns;         /* sum of per-request first-token cost proxies */
} unison_counters;

typedef struct {
  uint32_t ev, op, a, b; /* event index, UNISON_OP_*, session / tier operands */
} unison_record;

/* Workspace bytes for these sizes.  Errors: UNISON_E_INVALID. */
int unison_workspace_size(const unison_dims* d, size_t* bytes);

/* Creates a context on the current HIP device.  `hip_stream` is a
 * hipStream_t (NULL = the null stream); `workspace` is DEVICE memory of at
 * least unison_workspace_size() bytes, 256-byte aligned.  Both are borrowed
 * for the context's lifetime. */
int unison_create(unison_ctx** out, const unison_dims* d, void* hip_stream, void* workspace,
                  size_t workspace_bytes);
/* Bytes of the library's static workspace (unison_create_static). */
#define UNISON_STATIC_WORKSPACE_BYTES (32u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): creates a
 * context like unison_create whose workspace is the library's own static
 * device array of UNISON_STATIC_WORKSPACE_BYTES (32 MiB), one per GPU,
 * reserved when the library is loaded and held until the process ends.  No
 * device memory is allocated (the context itself is host memory, as for
 * unison_create).  The array's address on the current device is taken once,
 * at the first call on that device.  Every other entry point works on such
 * a context as on any other.
 * All contexts made this way on one GPU share its array, which keeps the
 * contents the latest call left: each new context takes the array over, and
 * calls on an older context of the same device then fail with
 * UNISON_E_INVALID ("superseded").  Work of two such contexts that overlaps
 * on one GPU races; a fresh unison_run (without UNISON_RUN_CONTINUE) starts
 * every simulation from an empty pool whatever the array held.
 * Errors: UNISON_E_INVALID (null out, invalid dims), UNISON_E_CAPACITY
 * (unison_workspace_size(d) exceeds UNISON_STATIC_WORKSPACE_BYTES; nothing
 * is created), UNISON_E_HIP (no current device, or the array's address could
 * not be taken).  unison_last_error(NULL) gives the message of this thread's
 * latest failed create call. */
int unison_create_static(unison_ctx** out, const unison_dims* d, void* hip_stream);

void unison_destroy(unison_ctx* ctx);
const char* unison_last_error(const unison_ctx* ctx);
const char* unison_strerror(int code);
int unison_set_stream(unison_ctx* ctx, void* hip_stream);

/* Session traces. */
typedef struct {
  uint32_t n_traces;
  uint32_t pad0;
  const uint64_t* ev_offset;   /* HOST [n_traces+1]: trace i = events [off[i], off[i+1]) */
  const uint64_t* sess_offset; /* HOST [n_traces+1]: trace i's sessions in sess_kvb */
  const uint64_t* ev_t_ns;     /* DEVICE */
  const uint32_t* ev_sid;      /* DEVICE */
  const uint32_t* ev_info;     /* DEVICE */
  const uint32_t* ev_len;      /* DEVICE */
  const uint64_t* ev_next_ns;  /* DEVICE */
  const uint32_t* sess_kvb;    /* DEVICE */
  const uint32_t* ev_tool;     /* DEVICE, or NULL: every gap is tool class 0 */
} unison_trace_batch;

/* Registers the traces (the arrays stay borrowed) and checks the event format
 * of each once, on a host copy of its events (session id in range, kind <=
 * DONE, times non-decreasing, every session's turns in order, prefixes
 * non-decreasing, gap onsets' tool classes below UNISON_ETA_CLASSES): a
 * simulation then stops at its trace's first malformed event and reports it
 * through counters.error.  Synchronises the stream.
 * Errors: UNISON_E_INVALID (count differs from the dims, offsets not
 * monotone), UNISON_E_CAPACITY (a trace has more sessions than
 * dims.max_sessions), UNISON_E_HIP. */
int unison_load_traces(unison_ctx* ctx, const unison_trace_batch* tb);

/* eq. (hazard): counts d(t) = #{T = t+1} and n(t) = #{T > t}, t = 0..50, over
 * a population of session turn counts.  turns: DEVICE [n]; d_out, n_out:
 * DEVICE [51].  Asynchronous on `hip_stream`. */
int unison_hazard_counts(void* hip_stream, const uint32_t* turns, uint32_t n, uint32_t* d_out,
                         uint32_t* n_out);

/* Installs hazard table `lut` from its counts: h(t) = d(t)/n(t) (0 where
 * n(t) = 0).  d, n: DEVICE [51], copied on the context's stream. */
int unison_set_hazard(unison_ctx* ctx, uint32_t lut, const uint32_t* d, const uint32_t* n);

/* The ETA baseline's table fitted on a trace: for each tool class c, the
 * mean (floor, integer ns) of next ARRIVE time - GAP_START time over the
 * trace's gap onsets of class c that have a next arrival; 0 for a class
 * without any.  Events: DEVICE arrays of n_events entries (ev_tool may be
 * NULL: all class 0); mean_out: DEVICE [UNISON_ETA_CLASSES].  Classes at or
 * above UNISON_ETA_CLASSES are skipped.  Asynchronous on `hip_stream`. */
int unison_eta_fit(void* hip_stream, uint64_t n_events, const uint64_t* ev_t_ns,
                   const uint32_t* ev_info, const uint32_t* ev_tool, const uint64_t* ev_next_ns,
                   uint64_t* mean_out);

/* Installs the ETA table of trace `trace`: the expected wait (ns) of each of
 * the UNISON_ETA_CLASSES tool classes.  A simulation of that trace under
 * UNISON_POLICY_ETA keys a session at its gap onset by the predicted return
 * onset + mean[class] (saturating); a completed session never returns.
 * mean: DEVICE, copied on the context's stream.  Errors: UNISON_E_INVALID. */
int unison_set_eta(unison_ctx* ctx, uint32_t trace, const uint64_t* mean);

/* Copies n_sims parameter rows (HOST) into the workspace.  Errors:
 * UNISON_E_INVALID for an out-of-range field (policy, lut, trace, b_h, b_g,
 * tau, n_slots, dma bandwidth, negative or NaN penalty, hazard_online,
 * dual_sync, or a dual row when dims.views is 0). */
int unison_set_params(unison_ctx* ctx, const unison_sim_params* params);

/* Runs every simulation over at most `max_events` further events of its
 * trace (UINT64_MAX: to the end).  Without UNISON_RUN_CONTINUE each
 * simulation starts from an empty pool; with it, each simulation resumes
 * under the parameter row and policy it ran with (state a policy never
 * reads, such as the gap EMA of LRU or timeout without TIDE, is not kept).
 * policy_override is a UNISON_POLICY_* value applied to all simulations, or
 * UNISON_POLICY_PARAMS.  A batch with a dual-design row runs on the copies'
 * kernel (variant 11).  Tables above the LDS-resident size run, while no
 * simulation can hold more than 4,096 residents (min(N_sess, sessions)), on
 * one wavefront per simulation with the residents in 24-byte LDS slots
 * (variant 14); otherwise on workgroup kernels that keep one bit of LDS per
 * session (the residency bits their scans visit): 128 KiB at
 * UNISON_MAX_SESSIONS; the LDS left holds up to 8 resident-cache slots of
 * 28 B per thread.  Asynchronous.
 * Errors: UNISON_E_NOT_READY (also: an ETA simulation whose trace has no ETA
 * table), UNISON_E_INVALID (also: a register-table
 * variant forced on a batch with a dual-design row), UNISON_E_CAPACITY (the
 * largest trace exceeds the chosen kernel variant, e.g. on a device with
 * less LDS per workgroup than the bits need). */
int unison_run(unison_ctx* ctx, uint32_t policy_override, uint32_t flags, uint64_t max_events);

/* Copies counters of simulations [first, first+n) to HOST `dst`; synchronises
 * the stream.  Returns UNISON_E_BAD_TRACE if any of them recorded an error
 * (the counters are still copied). */
int unison_read_counters(unison_ctx* ctx, unison_counters* dst, uint32_t first, uint32_t n);

/* DEVICE pointer to the counters array [n_sims] (valid until destroy). */
int unison_counters_device(unison_ctx* ctx, const unison_counters** out);

/* Copies simulation `sim`'s decision records of the last runs (in decision
 * order, at most dims.log_cap kept) to HOST `dst` (cap entries); *n_total is
 * the number of records produced, which may exceed what was kept.
 * Synchronises the stream. */
int unison_read_log(unison_ctx* ctx, uint32_t sim, unison_record* dst, uint32_t cap,
                    uint64_t* n_total);

/* ------------------------------------------------ ranking fidelity (C ABI
 * without a context; all arrays DEVICE; asynchronous on `hip_stream`). */

/* Replays each session's gap history through both register-file EMAs:
 * eq. (ema) in fp32 microseconds and eq. (gapq) + eq. (ema-int) in integers.
 * gaps_ns [n][max_hist] (row i uses its first n_hist[i] entries). */
int unison_ema_replay(void* hip_stream, uint32_t n, uint32_t max_hist, const uint64_t* gaps_ns,
                      const uint8_t* n_hist, uint32_t b_g, uint64_t tau_ns, float* g_out,
                      uint64_t* gq_out);

/* eq. (surv) + eq. (esp) in fp32: out[i] = +inf if done[i], else
 * g/sigma + (1 - sigma) P with sigma = max(0.01, 1 - h(min(turn, 50))) and
 * h = d/n from the counts lut_d, lut_n [51]. */
int unison_score_fp32(void* hip_stream, uint32_t n, const uint8_t* turn, const float* g,
                      const uint8_t* done, const uint32_t* lut_d, const uint32_t* lut_n,
                      float penalty_us, float* out);

/* eq. (hq), eq. (survq), eq. (t1), eq. (t2), eq. (scoreq) with b_s = 64:
 * out[i] = 2^64-1 if done[i], else sat64(T1 + floor((Lambda - sigma_q) P_Z /
 * Lambda)), Lambda = 2^b_h - 1, with T1 = floor(gq Lambda / sigma_q) for
 * recip_bits = 0 (exact divider), else T1 = floor(gq Lambda r / 2^W) with
 * r = floor(2^W / sigma_q + 1/2) and W = recip_bits <= 32 (reciprocal
 * table). */
int unison_score_fixed(void* hip_stream, uint32_t n, const uint8_t* turn, const uint64_t* gq,
                       const uint8_t* done, const uint32_t* lut_d, const uint32_t* lut_n,
                       uint32_t b_h, uint64_t p_z, uint32_t recip_bits, uint64_t* out);

/* Kendall tau-b pair counts per snapshot (Sec. VI-F): counts[s][5] =
 * {concordant, discordant, tied in x only, tied in y only, tied in both}
 * over pairs i < j of snapshot s, and top1[s] = 1 when argmax x and argmax y
 * (ties to the earlier position) coincide, else 0.  x, y: DEVICE [n_x].
 * Snapshot s holds x[idx[s][j]], y[idx[s][j]] for j < n_per (idx NULL: rows
 * s*n_per .. s*n_per+n_per-1, which must lie below n_x).  An index >= n_x
 * is not read: the snapshot's top1 is then 255 and its counts are void.
 * x holds scores, never NaN (a NaN has no rank; its snapshot's counts are
 * unspecified).  2 <= n_per <= 4096; from 256 entries on the counts come
 * from sorting the snapshot in LDS (O(n log^2 n)), below it pair by pair. */
int unison_kendall(void* hip_stream, uint32_t n_snap, uint32_t n_per, uint64_t n_x, const float* x,
                   const uint64_t* y, const uint32_t* idx, uint64_t* counts, uint8_t* top1);

/* Copies the hazard counts d(t), n(t), t = 0..50, that simulation `sim`'s
 * table held at the end of the latest run to HOST d_out[51], n_out[51]: its
 * fixed table's, or what its online table (hazard_online = 1) has counted.
 * Synchronises the context's stream.  Errors: UNISON_E_INVALID (sim out of
 * range, null pointer), UNISON_E_NOT_READY (no run yet). */
int unison_read_hazard(unison_ctx* ctx, uint32_t sim, uint32_t* d_out, uint32_t* n_out);

/* Test hook: pins the simulation kernel variant (-1 = chosen by the largest
 * trace and the largest resident count; register tables of lanes x sessions
 * per lane 0: 16 x 1, 1: 64 x 1, 2: 64 x 4, 4: 4 x 4, 5: 8 x 2, 7: 16 x 4,
 * 8: 32 x 8 (6 is retired); one workgroup per simulation with the table 3:
 * streamed from the workspace by 256 threads, 10: by 512 threads, 9: held in
 * LDS (256 threads), 12: held in LDS by one wavefront, 11: streamed by 512
 * threads with the dual design's copies -- the only variant for a batch with
 * a dual-design row; one wavefront per simulation with 13: the table in LDS
 * and the residents in 1 to 8 vector-register slots per lane (at most 512
 * residents), 14: the table in the workspace and the residents in LDS slots
 * (at most 4,096 residents)).  A variant too small for the traces or their
 * resident counts, or an unknown id, makes unison_run return
 * UNISON_E_CAPACITY. */
int unison_debug_force_variant(unison_ctx* ctx, int variant);

/* Test hook: at most `slots` resident-cache slots per thread for the streamed
 * table kernels (variants 3 and 10), so tests can drive threads past their
 * slots; -1 restores the automatic count (up to 8, as the LDS left by the
 * residency bits allows).  The results never depend on it.  Errors:
 * UNISON_E_INVALID (null context, slots < -1). */
int unison_debug_cache_slots(unison_ctx* ctx, int slots);

/* Test hook, host only (no GPU work): the barrier plan of the sorted Kendall
 * path for a snapshot padded to n_pad entries (a power of two, 256..4096).
 * step 0: bitonic pass of stage a (= k) and stride b (= j); step 1: merge
 * level that merges runs of a entries (a >= 8: shorter runs are merged in
 * registers).  Bitonic passes run in groups of up to three in registers, one
 * LDS load before a group's first pass and one store after its last.
 * Returns 1 when the kernel places a workgroup barrier after that step, 0
 * when none (the next pass of the group runs in registers) or only the
 * wavefront-local fence (the step and the next touch no LDS entry another
 * wavefront touches), or UNISON_E_INVALID for a step the kernel does not
 * take. */
int unison_debug_kendall_barrier(uint32_t n_pad, uint32_t step, uint32_t a, uint32_t b);

uint32_t unison_version(void);

#ifdef __cplusplus
}
#endif
#endif /* UNISON_H */
