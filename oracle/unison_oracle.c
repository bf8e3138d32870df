/*
 * unison_oracle.c -- TEST INFRASTRUCTURE, not part of the product.
 *
 * A plain, slow, single-threaded CPU reference ("the oracle") for the UNISON
 * residency policy: SPEAR eviction scoring (Sec. III-B), TIDE idle-window
 * tiering (Sec. III-C), the joint event loop (Algorithm 1), the fixed-point
 * image of the score (Sec. IV-C) and the ranking-fidelity statistics
 * (Sec. VI-F).  Only the test-suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no source
 * with the HIP implementation; the two meet only in the binary trace format.
 *
 * Every step is written the obvious way: one loop over the events of one
 * simulation, a full linear scan of the session table for every argmax or
 * argmin, and the TIDE pass as a literal while-loop.  Nothing is cached,
 * blocked or reordered.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no FMA contraction, IEEE float division, round-to-nearest-even).
 *
 * ---------------------------------------------------------------------------
 * Readings of points the paper leaves open (both implementations follow them)
 * ---------------------------------------------------------------------------
 *  time      Trace times are integer nanoseconds.  The tool gap of eq. (gap)
 *            is a_{s,k} - c_{s,k-1}: the ARRIVE time minus the time of the
 *            session's previous GAP_START, both taken from the trace.
 *  events    ARRIVE (turn k starts; a gap_end when k >= 1), GAP_START (turn
 *            k ended and another follows) and DONE (the final turn ended).
 *            The trace fixes their order; the simulator consumes it as given.
 *  table     A session enters the register file at its first ARRIVE and
 *            stays while it is not completed or while it still holds KV.
 *            The per-event scan covers every table entry (the hardware scans
 *            the whole register file, eq. (scan)).  Victims and migrants are
 *            the residents that are not being served (an ARRIVE pins its
 *            session until its GAP_START/DONE).
 *  EMA       g = 0 and g_q = 0 before the first gap.  Float path, in us:
 *            x = (float)min(gap_ns / 1000, 2^32 - 1) (whole microseconds);
 *            g = (3x + 7g) / 10 with every operation rounded to fp32.  Integer path eq. (gapq) and
 *            eq. (ema-int): x_q = min(gap_ns / tau, 2^b_g - 1),
 *            g_q = (3 x_q + 7 g_q) / 10, floors.
 *  hazard    t is the 0-based index of the session's latest turn.  From a
 *            population of turn counts T: n(t) = #{T > t}, d(t) = #{T = t+1}
 *            for t = 0..50; h = 0 where n(t) = 0.  Float LUT: (float)d /
 *            (float)n.  Fixed LUT eq. (hq): floor(h*Lambda + 1/2) computed
 *            exactly as (2 d Lambda + n) / (2 n).  eps = 1/100 exactly.
 *  divider   eq. (t1) divides by sigma_q with an exact divider, or (the sweep's
 *            other divider type) multiplies by a reciprocal read from a table
 *            of depth Lambda: r[s] = floor(2^W / s + 1/2) for s = 1..Lambda,
 *            W the entry's fraction bits, and T1 = floor(g_q Lambda r[sigma_q]
 *            / 2^W).  The division by the constant Lambda in eq. (t2) stays
 *            exact.
 *  score     eq. (esp) with S_max = +inf for a completed session; operation
 *            order sigma = max(0.01f, 1 - h); a = g/sigma; b = 1 - sigma;
 *            c = b*P; s = a + c.  P is in microseconds.
 *  keys      "larger key = evict first".  SPEAR: the fp32 score (or the
 *            fixed-point score).  LRU/timeout: UINT64_MAX - last event time.
 *            Belady: time of the next ARRIVE (UINT64_MAX once completed).
 *            Ties in argmax and argmin go to the smallest session id.
 *  capacity  eq. (cap) in bytes: a session holds len * kv_bytes_per_token.
 *  placement On ARRIVE the request is classified by the session's tier at
 *            arrival (SRAM hit, HBM hit, miss).  The session then holds its
 *            new length; it prefers its current tier on a hit and SRAM on a
 *            miss, else the other tier.  While it fits neither, the argmax
 *            victim over all evictable residents is evicted (Alg. 1 evicts
 *            one victim per violation; the loop repeats it).  A session that
 *            cannot fit even an empty tier, or finds nothing left to evict,
 *            is bypassed (served, not retained).
 *  TIDE      On GAP_START with the DMA engine free, Delta is the session's
 *            own gap EMA (us, truncated), budget = Delta * B in bytes
 *            (eq. (budget), eq. (budgetq)).  Loop: p = argmin over evictable
 *            HBM residents, stop if none or if p is completed.  If p fits in
 *            free SRAM and in the budget: promote it alone.  Otherwise d =
 *            argmax over evictable SRAM residents; swap when key(p) < key(d)
 *            strictly, both fit the budget and eq. (cap) holds after the
 *            swap.  The first move that is not legal ends the pass.  The DMA
 *            engine is then busy for ceil(moved * 1000 / B) ns.
 *  online    Online hazard table (the convergence study beside eq.
 *            (attainment)): the counts start at zero, and each DONE adds its
 *            session (T = its turn index + 1) to eq. (hazard) -- n(t) += 1
 *            for t < min(T, 51), d(T-1) += 1 when T - 1 <= 50 -- for the
 *            first online_sessions completions.  The update follows the DONE's
 *            register write, so that event's scan already uses the new table;
 *            every score is then re-evaluated against it.
 *  prefetch  A promotion or swap moves its session into SRAM ahead of its
 *            return; the session's next request is a prefetch hit when it
 *            finds the session in SRAM (prefetch accuracy = prefetch hits /
 *            (promotions + swaps), the ablation of scoring and tiering).
 *  dual      The dual design of eq. (rf) / eq. (stale): the eviction engine and
 *            the TIDE engine each read keys from a private copy of the
 *            register file (every field of every session), overwritten with
 *            the live file after every ARRIVE and GAP_START ("after every
 *            request and gap"), after every 8th ARRIVE, or after every
 *            GAP_START.  Which sessions are resident, in which tier, and
 *            which are pinned stays live (it is the pool's physical state).
 *            The per-event scan and the victims use the eviction copy; TIDE's
 *            p, d and key(p) < key(d) use the TIDE copy.  At each eviction and
 *            at each TIDE move the live file's choice over the same candidates
 *            is computed too: vict_diff / prom_diff count the decisions that
 *            differ.  The copies start as the empty register file.
 *  timeout   Before an event is written, every resident that has been idle
 *            longer than the TTL expires (its timer fired since the last event).
 *  ETA       The tool-type arrival-table baseline (the expected-completion
 *            estimator among the related methods): each gap onset names the
 *            tool class of the gap it opens, and a table holds one expected
 *            wait per class -- the same wait for every session that calls
 *            the tool.  By default the table is fitted on the whole trace, as
 *            the hazard table is: the mean (floor, integer ns) of the gaps of
 *            that class, a gap being the next ARRIVE's time minus the
 *            GAP_START's.  The key is the predicted return, gap start + the
 *            class's wait (saturating), larger = evict first; a completed
 *            session never returns (2^64 - 1).  Tool classes are 0..15; a
 *            gap onset naming a larger one breaks the trace format.
 *  account   eq. (hr-amat), eq. (prered): SRAM hit amat += len*kvb*t_s,
 *            ttft += len_prev*kvb*t_s + dlen*t_p, computed += dlen; HBM hit
 *            likewise with t_h; miss amat += len*t_p, ttft += len*t_p,
 *            computed += len, extra prefill += len_prev.  f64, event order.
 *  digest    Each decision (event index, op, sid a, sid b or tier) -- place,
 *            evict, expire, bypass, promote, swap -- is hashed: w0 = ev << 8 |
 *            op, w1 = a << 32 | b, h = mix(w0 ^ w1 * 0x9e3779b97f4a7c15) with
 *            mix the SplitMix64 finaliser (Steele, Lea and Flood, 2014); the
 *            hashes are summed mod 2^64, so the digest does not depend on
 *            the order in which one event's decisions are listed.  The scan
 *            result v of event e (0xFFFFFFFF when nothing is evictable) enters
 *            a second digest as (v + 1) * ((2e + 1) * 0x9e3779b97f4a7c15).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#define NONE_ID 0xFFFFFFFFu
#define LUT_LEN 51 /* t = 0..50, eq. (hazard) */
#define ETA_CLASSES 16 /* tool classes of the ETA table */

enum { K_ARRIVE = 0, K_GAP_START = 1, K_DONE = 2 };
enum { P_SPEAR = 0, P_LRU = 1, P_TIMEOUT = 2, P_BELADY = 3, P_ETA = 4 };
enum { T_NONE = 0, T_SRAM = 1, T_HBM = 2 };
enum { PH_UNSEEN = 0, PH_SERVING = 1, PH_GAP = 2, PH_DONE = 3 };
enum { OP_EVICT = 1, OP_EXPIRE = 2, OP_BYPASS = 3, OP_PROMOTE = 4, OP_SWAP = 5, OP_VICTIM = 6,
       OP_PLACE = 7 };

enum { ORC_OK = 0, ORC_E_INVALID = -1, ORC_E_BAD_TRACE = -2 };

typedef struct {
  uint32_t policy;      /* P_SPEAR .. P_ETA */
  uint32_t tide;        /* 1: run the TIDE pass on GAP_START */
  uint32_t score_mode;  /* 0: fp32 score, 1: fixed-point score (SPEAR only) */
  uint32_t lut;         /* index of the hazard count table */
  uint64_t cap_sram_B;  /* C_S in bytes */
  uint64_t cap_hbm_B;   /* C_H in bytes */
  uint64_t n_slots;     /* N_sess */
  uint64_t dma_B_per_us;/* logical DMA bandwidth B */
  uint64_t ttl_ns;      /* timeout policy TTL */
  double t_s_ns_per_B;  /* SRAM read cost */
  double t_h_ns_per_B;  /* HBM read cost */
  double t_p_ns_per_tok;/* prefill cost */
  float penalty_us;     /* P of eq. (esp) */
  uint32_t b_h;         /* hazard fraction bits */
  uint32_t b_g;         /* gap register bits */
  uint32_t hazard_online;   /* 1: the table is rebuilt from completions */
  uint32_t online_sessions; /* completions it counts at most */
  uint32_t pad0;
  uint64_t tau_ns;      /* gap time divisor */
  uint64_t p_z;         /* integer penalty P_Z */
  uint32_t dual_sync;   /* 0 unified; 1, 2, 3: dual copies (see "dual" above) */
  uint32_t recip_bits;  /* 0: exact divider in eq. (t1); W: reciprocal table (see "divider") */
} orc_params;

typedef struct {
  uint64_t requests, hit_sram, hit_hbm, miss, bypass, evict, expire, promote, swap;
  uint64_t dma_bytes, tide_passes, tokens_total, tokens_computed, extra_prefill_tok;
  uint64_t score_evals, resident_evals, digest, victim_digest, events, error;
  uint64_t prefetch_hits, vict_diff, prom_diff;
  double amat_sum_ns, ttft_sum_ns;
} orc_counters;

typedef struct {
  uint32_t ev, op, a, b;
} orc_rec;

typedef struct {
  uint64_t used_sram, used_hbm;
  uint32_t n_res, n_table;
  uint32_t victim;      /* this event's scan result: argmax evictable key */
  uint32_t tide_ran;
  uint64_t tide_budget, tide_moved;
} orc_state;

/* ---------------------------------------------------------------- helpers */

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

/* The record's two words are combined by an odd multiplier (a bijection on
 * w1) before one finaliser pass. */
static uint64_t rec_hash(uint32_t ev, uint32_t op, uint32_t a, uint32_t b) {
  uint64_t w0 = ((uint64_t)ev << 8) | (uint64_t)op;
  uint64_t w1 = ((uint64_t)a << 32) | (uint64_t)b;
  return mix64(w0 ^ (w1 * 0x9e3779b97f4a7c15ULL));
}

static uint64_t sat_u64(unsigned __int128 x) {
  return x > (unsigned __int128)UINT64_MAX ? UINT64_MAX : (uint64_t)x;
}

/* ---------------------------------------------------- hazard, eq. (hazard) */

void orc_hazard_counts(const uint32_t* T, uint32_t n_sessions, uint32_t* d_out,
                       uint32_t* n_out) {
  for (uint32_t t = 0; t < LUT_LEN; t++) {
    uint32_t d = 0, n = 0;
    for (uint32_t i = 0; i < n_sessions; i++) {
      if (T[i] > t) n++;        /* still live at turn t */
      if (T[i] == t + 1) d++;   /* its last turn is t */
    }
    d_out[t] = d;
    n_out[t] = n;
  }
}

/* float hazard h(t) = d(t)/n(t) */
void orc_lut_f32(const uint32_t* d, const uint32_t* n, float* hf) {
  for (int t = 0; t < LUT_LEN; t++)
    hf[t] = n[t] ? (float)d[t] / (float)n[t] : 0.0f;
}

/* eq. (uq) applied to h = d/n: floor(d/n * Lambda + 1/2), clipped to Lambda. */
static uint64_t quantize_ratio(uint64_t d, uint64_t n, uint64_t lambda) {
  if (n == 0) return 0;
  unsigned __int128 num = (unsigned __int128)2 * d * lambda + n;
  uint64_t q = (uint64_t)(num / ((unsigned __int128)2 * n));
  return q > lambda ? lambda : q;
}

void orc_lut_q(const uint32_t* d, const uint32_t* n, uint32_t b_h, uint64_t* hq) {
  uint64_t lambda = (1ULL << b_h) - 1;
  for (int t = 0; t < LUT_LEN; t++) hq[t] = quantize_ratio(d[t], n[t], lambda);
}

/* ------------------------------------------------------ scores, eq. (esp) */

static float spear_f32(uint32_t turn, float g, int done, const float* hf, float P) {
  if (done) return INFINITY; /* S_max */
  uint32_t t = turn < 50 ? turn : 50;
  float sigma = fmaxf(0.01f, 1.0f - hf[t]); /* eq. (surv) */
  float a = g / sigma;
  float b = 1.0f - sigma;
  float c = b * P;
  return a + c;
}

/* The reciprocal table of the LUT divider: r[s] = floor(2^W / s + 1/2) for
 * s = 1..lambda, computed exactly as (2^(W+1) + s) / (2 s); r[0] unused. */
static uint64_t* recip_table(uint64_t lambda, uint32_t w) {
  uint64_t* r = (uint64_t*)calloc(lambda + 1, sizeof(uint64_t));
  if (!r) return NULL;
  for (uint64_t v = 1; v <= lambda; v++) r[v] = ((2ULL << w) + v) / (2 * v);
  return r;
}

/* eq. (hq), eq. (survq), eq. (t1), eq. (t2), eq. (scoreq) with b_s = 64; with
 * a reciprocal table (recip != NULL, w fraction bits) eq. (t1) multiplies by
 * recip[sigma_q] instead of dividing by sigma_q. */
static uint64_t spear_fixed(uint32_t turn, uint64_t gq, int done, const uint64_t* hq,
                            uint32_t b_h, uint64_t p_z, const uint64_t* recip, uint32_t w) {
  if (done) return UINT64_MAX; /* 2^b_s - 1 */
  uint64_t lambda = (1ULL << b_h) - 1;
  uint32_t t = turn < 50 ? turn : 50;
  uint64_t eps_q = (lambda + 50) / 100; /* floor(Lambda/100 + 1/2) */
  uint64_t h = hq[t];
  uint64_t sigma_q = lambda - h;
  if (sigma_q < eps_q) sigma_q = eps_q;
  unsigned __int128 t1;
  if (recip)
    t1 = ((unsigned __int128)gq * lambda * recip[sigma_q]) >> w;
  else
    t1 = ((unsigned __int128)gq * lambda) / sigma_q;
  unsigned __int128 t2 = ((unsigned __int128)(lambda - sigma_q) * p_z) / lambda;
  return sat_u64(t1 + t2);
}

void orc_score_f32(uint32_t n, const uint8_t* turn, const float* g, const uint8_t* done,
                   const float* hf, float P, float* out) {
  for (uint32_t i = 0; i < n; i++) out[i] = spear_f32(turn[i], g[i], done[i], hf, P);
}

/* The fixed-point scores of n sessions; recip_bits 0: exact divider, else the
 * reciprocal table of that many fraction bits.  b_h must be 6..32 (below 6,
 * floor(eps Lambda + 1/2) = 0 and sigma_q can be 0, where eq. (t1) is not
 * defined).  Returns ORC_OK or ORC_E_INVALID. */
int orc_score_fixed(uint32_t n, const uint8_t* turn, const uint64_t* gq,
                    const uint8_t* done, const uint64_t* hq, uint32_t b_h, uint64_t p_z,
                    uint32_t recip_bits, uint64_t* out) {
  if (b_h < 6 || b_h > 32 || recip_bits > 32) return ORC_E_INVALID;
  uint64_t* r = recip_bits ? recip_table((1ULL << b_h) - 1, recip_bits) : NULL;
  if (recip_bits && !r) return ORC_E_INVALID;
  for (uint32_t i = 0; i < n; i++)
    out[i] = spear_fixed(turn[i], gq[i], done[i], hq, b_h, p_z, r, recip_bits);
  free(r);
  return ORC_OK;
}

/* ----------------------------------------------------------- EMA updates */

/* The gap sample is taken in whole microseconds (the tau = 10^3 resolution of
 * eq. (lock)), clipped to 2^32 - 1 like the 32-bit gap register, so that the
 * fp32 and the integer register see the same sample. */
static uint32_t gap_us(uint64_t gap_ns) {
  uint64_t us = gap_ns / 1000;
  return us > 0xFFFFFFFFULL ? 0xFFFFFFFFu : (uint32_t)us;
}

static float ema_f32(float g, uint64_t gap_ns) {
  float x = (float)gap_us(gap_ns);
  float a = 3.0f * x;
  float b = 7.0f * g;
  return (a + b) / 10.0f; /* eq. (ema) */
}

static uint64_t ema_int(uint64_t gq, uint64_t gap_ns, uint32_t b_g, uint64_t tau) {
  uint64_t cap = b_g >= 64 ? UINT64_MAX : ((1ULL << b_g) - 1);
  uint64_t x = gap_ns / tau; /* eq. (gapq) */
  if (x > cap) x = cap;
  unsigned __int128 s = (unsigned __int128)3 * x + (unsigned __int128)7 * gq;
  return (uint64_t)(s / 10); /* eq. (ema-int) */
}

/* Replays a gap history per session through both EMAs. gaps is [n][max_hist]. */
void orc_ema_replay(uint32_t n, uint32_t max_hist, const uint64_t* gaps_ns,
                    const uint8_t* n_hist, uint32_t b_g, uint64_t tau, float* g_out,
                    uint64_t* gq_out) {
  for (uint32_t i = 0; i < n; i++) {
    float g = 0.0f;
    uint64_t gq = 0;
    for (uint32_t k = 0; k < n_hist[i] && k < max_hist; k++) {
      g = ema_f32(g, gaps_ns[(uint64_t)i * max_hist + k]);
      gq = ema_int(gq, gaps_ns[(uint64_t)i * max_hist + k], b_g, tau);
    }
    g_out[i] = g;
    gq_out[i] = gq;
  }
}

/* ------------------------------------------------------- the ETA table */

/* Mean wait per tool class over a trace's gaps (see "ETA" above): for every
 * GAP_START with a next arrival, gap = next - t joins its class's sum; mean =
 * floor(sum / count), 0 for a class without gaps. */
void orc_eta_fit(uint64_t n_events, const uint64_t* ev_t, const uint32_t* ev_info,
                 const uint32_t* ev_tool, const uint64_t* ev_next, uint64_t* mean_out) {
  unsigned __int128 sum[ETA_CLASSES];
  uint64_t cnt[ETA_CLASSES];
  for (int c = 0; c < ETA_CLASSES; c++) { sum[c] = 0; cnt[c] = 0; }
  for (uint64_t e = 0; e < n_events; e++) {
    if ((ev_info[e] >> 24) != K_GAP_START || ev_next[e] == UINT64_MAX) continue;
    uint32_t c = ev_tool ? ev_tool[e] : 0;
    if (c >= ETA_CLASSES || ev_next[e] < ev_t[e]) continue;
    sum[c] += ev_next[e] - ev_t[e];
    cnt[c]++;
  }
  for (int c = 0; c < ETA_CLASSES; c++)
    mean_out[c] = cnt[c] ? sat_u64(sum[c] / cnt[c]) : 0;
}

/* --------------------------------------------- Kendall tau-b pair counts */

/* counts = {concordant, discordant, tied in x only, tied in y only, tied in
 * both} over all pairs i < j of each snapshot; top1[s] = 1 when the argmax of
 * x and the argmax of y (ties to the earlier position) coincide.  idx maps
 * snapshot positions to entries of x and y; NULL means contiguous rows. */
void orc_kendall(uint32_t n_snap, uint32_t n_per, const float* x, const uint64_t* y,
                 const uint32_t* idx, uint64_t* counts, uint8_t* top1) {
  for (uint32_t s = 0; s < n_snap; s++) {
    uint64_t c = 0, d = 0, tx = 0, ty = 0, txy = 0;
    uint32_t bx = 0, by = 0;
    for (uint32_t i = 0; i < n_per; i++) {
      uint64_t ei = idx ? idx[(uint64_t)s * n_per + i] : (uint64_t)s * n_per + i;
      float xi = x[ei];
      uint64_t yi = y[ei];
      uint64_t eb = idx ? idx[(uint64_t)s * n_per + bx] : (uint64_t)s * n_per + bx;
      uint64_t ec = idx ? idx[(uint64_t)s * n_per + by] : (uint64_t)s * n_per + by;
      if (xi > x[eb]) bx = i;
      if (yi > y[ec]) by = i;
      for (uint32_t j = i + 1; j < n_per; j++) {
        uint64_t ej = idx ? idx[(uint64_t)s * n_per + j] : (uint64_t)s * n_per + j;
        int sx = (xi > x[ej]) - (xi < x[ej]);
        int sy = (yi > y[ej]) - (yi < y[ej]);
        if (sx == 0 && sy == 0) txy++;
        else if (sx == 0) tx++;
        else if (sy == 0) ty++;
        else if (sx == sy) c++;
        else d++;
      }
    }
    counts[(uint64_t)s * 5 + 0] = c;
    counts[(uint64_t)s * 5 + 1] = d;
    counts[(uint64_t)s * 5 + 2] = tx;
    counts[(uint64_t)s * 5 + 3] = ty;
    counts[(uint64_t)s * 5 + 4] = txy;
    top1[s] = (uint8_t)(bx == by);
  }
}

/* ------------------------------------------------- the event simulation */

typedef struct {
  uint32_t phase, tier, turn, len;
  uint32_t prefetched; /* TIDE moved it into SRAM since its last request */
  float g;
  uint64_t gq, last_ns, next_ns;
} sess_t;

typedef struct {
  const orc_params* p;
  const uint64_t* eta;  /* the ETA table, ETA_CLASSES waits in ns */
  uint64_t* recip;      /* the LUT divider's reciprocal table, or NULL (exact divider) */
  sess_t* s;
  sess_t* view[2];  /* dual design: the eviction engine's and TIDE's copies */
  int keysrc;       /* where keys are read: -1 the live file, 0 or 1 a copy */
  const uint32_t* kvb;
  uint32_t n_sess;
  float hf[LUT_LEN];
  uint64_t hq[LUT_LEN];
  uint32_t hd[LUT_LEN], hn[LUT_LEN]; /* the counts the table is built from */
  uint64_t used[3]; /* indexed by tier */
  uint64_t n_res, n_table;
  uint64_t dma_free_at;
  orc_counters* c;
  orc_rec* log;
  uint32_t log_cap, log_len;
  uint32_t ev;
} sim_t;

static void emit(sim_t* m, uint32_t op, uint32_t a, uint32_t b) {
  m->c->digest += rec_hash(m->ev, op, a, b);
  if (m->log && m->log_len < m->log_cap) {
    orc_rec r = {m->ev, op, a, b};
    m->log[m->log_len] = r;
  }
  if (m->log) m->log_len++;
}

static int evictable(const sess_t* e) { return e->tier != T_NONE && e->phase != PH_SERVING; }

static uint64_t size_of(const sim_t* m, uint32_t i) {
  return (uint64_t)m->s[i].len * (uint64_t)m->kvb[i];
}

/* "larger = evict first" key of one table entry */
static uint64_t key_of(const sim_t* m, uint32_t i) {
  const sess_t* e = m->keysrc < 0 ? &m->s[i] : &m->view[m->keysrc][i];
  switch (m->p->policy) {
    case P_SPEAR:
      if (m->p->score_mode == 1)
        return spear_fixed(e->turn, e->gq, e->phase == PH_DONE, m->hq, m->p->b_h, m->p->p_z,
                           m->recip, m->p->recip_bits);
      else {
        float f = spear_f32(e->turn, e->g, e->phase == PH_DONE, m->hf, m->p->penalty_us);
        uint32_t bits;
        memcpy(&bits, &f, 4); /* non-negative floats order like their bit patterns */
        return bits;
      }
    case P_LRU:
    case P_TIMEOUT:
      return UINT64_MAX - e->last_ns;
    default: /* Belady: the next arrival; ETA: the predicted one */
      return e->next_ns;
  }
}

static uint64_t done_key(const sim_t* m) {
  if (m->p->policy == P_SPEAR) return m->p->score_mode == 1 ? UINT64_MAX : 0x7F800000u;
  if (m->p->policy == P_BELADY || m->p->policy == P_ETA) return UINT64_MAX;
  return 0; /* recency keys have no completion value */
}

/* argmax over evictable residents in tier `tier` (T_NONE = any tier) */
static uint32_t argmax_key(const sim_t* m, uint32_t tier) {
  uint32_t best = NONE_ID;
  uint64_t bk = 0;
  for (uint32_t i = 0; i < m->n_sess; i++) {
    if (!evictable(&m->s[i])) continue;
    if (tier != T_NONE && m->s[i].tier != tier) continue;
    uint64_t k = key_of(m, i);
    if (best == NONE_ID || k > bk) { best = i; bk = k; }
  }
  return best;
}

static uint32_t argmin_key(const sim_t* m, uint32_t tier) {
  uint32_t best = NONE_ID;
  uint64_t bk = 0;
  for (uint32_t i = 0; i < m->n_sess; i++) {
    if (!evictable(&m->s[i])) continue;
    if (tier != T_NONE && m->s[i].tier != tier) continue;
    uint64_t k = key_of(m, i);
    if (best == NONE_ID || k < bk) { best = i; bk = k; }
  }
  return best;
}

static void release(sim_t* m, uint32_t i) {
  m->used[m->s[i].tier] -= size_of(m, i);
  m->s[i].tier = T_NONE;
  m->n_res--;
  if (m->s[i].phase == PH_DONE) m->n_table--; /* a completed session leaves the table */
}

static void put(sim_t* m, uint32_t i, uint32_t tier) {
  m->s[i].tier = tier;
  m->used[tier] += size_of(m, i);
  m->n_res++;
}

static int fits(const sim_t* m, uint32_t tier, uint64_t size) {
  uint64_t cap = tier == T_SRAM ? m->p->cap_sram_B : m->p->cap_hbm_B;
  return m->used[tier] + size <= cap && m->n_res + 1 <= m->p->n_slots;
}

/* Algorithm 1, capacity branch: place the arriving session, evicting the
 * argmax victim while eq. (cap) would be violated. */
static void place(sim_t* m, uint32_t sid, uint32_t pref) {
  uint64_t size = size_of(m, sid);
  uint32_t other = pref == T_SRAM ? T_HBM : T_SRAM;
  if (size > m->p->cap_sram_B && size > m->p->cap_hbm_B) {
    emit(m, OP_BYPASS, sid, NONE_ID);
    m->c->bypass++;
    return;
  }
  for (;;) {
    if (fits(m, pref, size)) { put(m, sid, pref); emit(m, OP_PLACE, sid, pref); return; }
    if (fits(m, other, size)) { put(m, sid, other); emit(m, OP_PLACE, sid, other); return; }
    uint32_t v = argmax_key(m, T_NONE);
    if (m->view[0] && v != NONE_ID) {
      int src = m->keysrc;
      m->keysrc = -1;
      if (argmax_key(m, T_NONE) != v) m->c->vict_diff++; /* eq. (stale) */
      m->keysrc = src;
    }
    if (v == NONE_ID) {
      emit(m, OP_BYPASS, sid, NONE_ID);
      m->c->bypass++;
      return;
    }
    emit(m, OP_EVICT, v, NONE_ID);
    m->c->evict++;
    release(m, v);
  }
}

/* Algorithm 1, tiering branch: eq. (budget), eq. (promote), eq. (demote). */
static void tide(sim_t* m, uint32_t sid, uint64_t now, orc_state* st) {
  const orc_params* p = m->p;
  uint64_t delta_us;
  if (p->policy == P_SPEAR && p->score_mode == 1)
    delta_us = sat_u64(((unsigned __int128)m->s[sid].gq * p->tau_ns) / 1000);
  else
    delta_us = (uint64_t)m->s[sid].g;
  uint64_t budget = sat_u64((unsigned __int128)delta_us * p->dma_B_per_us);
  uint64_t left = budget, moved = 0;
  uint64_t inf = done_key(m);
  int has_inf = p->policy == P_SPEAR || p->policy == P_BELADY || p->policy == P_ETA;
  m->c->tide_passes++;
  int src = m->keysrc;
  m->keysrc = m->view[1] ? 1 : -1;
  uint32_t live_p = NONE_ID;
  for (;;) {
    uint32_t pid = argmin_key(m, T_HBM);
    if (pid == NONE_ID) break;
    if (m->view[1]) {
      m->keysrc = -1;
      live_p = argmin_key(m, T_HBM);
      m->keysrc = 1;
    }
    uint64_t kp = key_of(m, pid);
    if (has_inf && kp == inf) break;
    uint64_t sp = size_of(m, pid);
    if (m->used[T_SRAM] + sp <= p->cap_sram_B && sp <= left) {
      m->used[T_HBM] -= sp;
      m->used[T_SRAM] += sp;
      m->s[pid].tier = T_SRAM;
      m->s[pid].prefetched = 1;
      left -= sp;
      moved += sp;
      emit(m, OP_PROMOTE, pid, NONE_ID);
      m->c->promote++;
      if (m->view[1] && live_p != pid) m->c->prom_diff++;
      continue;
    }
    uint32_t did = argmax_key(m, T_SRAM);
    if (did == NONE_ID) break;
    uint64_t kd = key_of(m, did);
    uint64_t sd = size_of(m, did);
    int legal = kp < kd && sp <= left && sd <= left - sp &&
                m->used[T_SRAM] - sd + sp <= p->cap_sram_B &&
                m->used[T_HBM] - sp + sd <= p->cap_hbm_B;
    if (!legal) break;
    m->used[T_SRAM] = m->used[T_SRAM] - sd + sp;
    m->used[T_HBM] = m->used[T_HBM] - sp + sd;
    m->s[pid].tier = T_SRAM;
    m->s[pid].prefetched = 1;
    m->s[did].tier = T_HBM;
    left -= sp + sd;
    moved += sp + sd;
    emit(m, OP_SWAP, pid, did);
    m->c->swap++;
    if (m->view[1] && live_p != pid) m->c->prom_diff++;
  }
  m->keysrc = src;
  if (moved) {
    unsigned __int128 ns = ((unsigned __int128)moved * 1000 + p->dma_B_per_us - 1) / p->dma_B_per_us;
    m->dma_free_at = sat_u64((unsigned __int128)now + ns);
  }
  m->c->dma_bytes += moved;
  if (st) { st->tide_ran = 1; st->tide_budget = budget; st->tide_moved = moved; }
}

/*
 * Runs one simulation over one trace.
 *   ev_*       the trace's events (already in order), n_events long
 *   kvb        bytes per token of each of the trace's n_sess sessions
 *   lut_d/n    the hazard counts d(t), n(t) of this simulation's table (not
 *              read when p->hazard_online: that table starts empty)
 *   max_events stop after this many events (UINT64_MAX = all)
 *   log/states optional outputs (NULL to skip); states has one entry per event
 *   counts_out optional: the table's counts at the end, d[51] then n[51]
 *   elapsed_ns wall time of the event loop alone (optional)
 *   ev_tool    tool class of each event (read at gap onsets; NULL: all 0)
 *   eta_mean   the ETA table (ETA_CLASSES waits, ns); needed by the ETA policy
 * Returns ORC_OK, ORC_E_INVALID or ORC_E_BAD_TRACE (counters.error = event+1).
 */
int orc_run(const orc_params* p, uint64_t n_events, const uint64_t* ev_t,
            const uint32_t* ev_sid, const uint32_t* ev_info, const uint32_t* ev_len,
            const uint64_t* ev_next, uint32_t n_sess, const uint32_t* kvb,
            const uint32_t* lut_d, const uint32_t* lut_n, uint64_t max_events,
            orc_counters* out, orc_rec* log, uint32_t log_cap, uint32_t* log_len,
            orc_state* states, uint32_t* counts_out, uint64_t* elapsed_ns,
            const uint32_t* ev_tool, const uint64_t* eta_mean) {
  if (!p || !out || p->policy > P_ETA || (p->policy == P_ETA && !eta_mean) ||
      p->dma_B_per_us == 0 || p->n_slots == 0 ||
      p->tau_ns == 0 || p->b_h < 6 || p->b_h > 32 || p->b_g < 1 || p->b_g > 64 || p->dual_sync > 3 ||
      p->recip_bits > 32 ||
      !(p->penalty_us >= 0.0f))
    return ORC_E_INVALID;
  memset(out, 0, sizeof *out);
  sim_t m;
  memset(&m, 0, sizeof m);
  m.p = p;
  m.eta = eta_mean;
  if (p->policy == P_SPEAR && p->score_mode == 1 && p->recip_bits) {
    m.recip = recip_table((1ULL << p->b_h) - 1, p->recip_bits);
    if (!m.recip) return ORC_E_INVALID;
  }
  m.kvb = kvb;
  m.n_sess = n_sess;
  m.c = out;
  m.log = log;
  m.log_cap = log_cap;
  m.s = (sess_t*)calloc(n_sess ? n_sess : 1, sizeof(sess_t));
  if (!m.s) return ORC_E_INVALID;
  for (uint32_t i = 0; i < n_sess; i++) m.s[i].next_ns = UINT64_MAX; /* no next arrival yet */
  m.keysrc = -1;
  if (p->dual_sync) {
    for (int k = 0; k < 2; k++) {
      m.view[k] = (sess_t*)calloc(n_sess ? n_sess : 1, sizeof(sess_t));
      if (!m.view[k]) { free(m.s); free(m.view[0]); free(m.recip); return ORC_E_INVALID; }
      memcpy(m.view[k], m.s, (size_t)n_sess * sizeof(sess_t)); /* the empty register file */
    }
  }
  for (int t = 0; t < LUT_LEN; t++) {
    m.hd[t] = p->hazard_online ? 0 : lut_d[t];
    m.hn[t] = p->hazard_online ? 0 : lut_n[t];
  }
  orc_lut_f32(m.hd, m.hn, m.hf);
  orc_lut_q(m.hd, m.hn, p->b_h, m.hq);
  uint32_t online_seen = 0;
  int rc = ORC_OK;
  uint64_t n_run = n_events < max_events ? n_events : max_events;
  struct timespec t0, t1;
  clock_gettime(CLOCK_MONOTONIC, &t0);
  uint64_t prev_t = 0;
  for (uint64_t e = 0; e < n_run; e++) {
    m.ev = (uint32_t)e;
    uint64_t now = ev_t[e];
    uint32_t sid = ev_sid[e];
    uint32_t kind = ev_info[e] >> 24;
    uint32_t turn = ev_info[e] & 0xFFFFFFu;
    orc_state* st = states ? &states[e] : NULL;
    if (st) memset(st, 0, sizeof *st);
    uint32_t tool = ev_tool ? ev_tool[e] : 0;
    if (sid >= n_sess || now < prev_t || kind > K_DONE || (kind == K_GAP_START && tool >= ETA_CLASSES)) {
      rc = ORC_E_BAD_TRACE; out->error = e + 1; break;
    }
    prev_t = now;
    sess_t* x = &m.s[sid];

    /* timeout policy: the TTL timers that fired since the previous event
     * expire idle residents (the arriving session included), in ascending id */
    if (p->policy == P_TIMEOUT) {
      for (uint32_t i = 0; i < n_sess; i++) {
        if (evictable(&m.s[i]) && now - m.s[i].last_ns > p->ttl_ns) {
          emit(&m, OP_EXPIRE, i, NONE_ID);
          out->expire++;
          release(&m, i);
        }
      }
    }

    /* Alg. 1: write e into R; on gap_end update the EMA (eq. (gap), eq. (ema)) */
    uint32_t len_prev = x->len;
    if (kind == K_ARRIVE) {
      if (turn == 0) {
        if (x->phase != PH_UNSEEN) { rc = ORC_E_BAD_TRACE; out->error = e + 1; break; }
        x->g = 0.0f;
        x->gq = 0;
        x->len = 0;
        len_prev = 0;
        m.n_table++;
      } else {
        if (x->phase != PH_GAP || turn != x->turn + 1 || ev_len[e] < x->len) {
          rc = ORC_E_BAD_TRACE; out->error = e + 1; break;
        }
        uint64_t gap = now - x->last_ns;
        x->g = ema_f32(x->g, gap);
        x->gq = ema_int(x->gq, gap, p->b_g, p->tau_ns);
      }
      x->turn = turn;
      x->phase = PH_SERVING;
      x->last_ns = now;
    } else {
      if (x->phase != PH_SERVING) { rc = ORC_E_BAD_TRACE; out->error = e + 1; break; }
      x->last_ns = now;
      if (kind == K_GAP_START) {
        x->phase = PH_GAP;
        /* Belady reads the true next arrival; ETA predicts it from the tool */
        x->next_ns = p->policy == P_ETA ? sat_u64((unsigned __int128)now + m.eta[tool]) : ev_next[e];
      } else {
        x->phase = PH_DONE;
        x->next_ns = UINT64_MAX;
        if (p->hazard_online && online_seen < p->online_sessions) {
          /* the completed session joins the counts of eq. (hazard) */
          uint32_t T = x->turn + 1;
          for (uint32_t t = 0; t < LUT_LEN && t < T; t++) m.hn[t]++;
          if (T - 1 < LUT_LEN) m.hd[T - 1]++;
          online_seen++;
          orc_lut_f32(m.hd, m.hn, m.hf);
          orc_lut_q(m.hd, m.hn, p->b_h, m.hq);
        }
      }
    }

    /* the per-event scan of the register file (eq. (pipe)): every table entry
     * is scored; its result is this event's victim index */
    out->score_evals += m.n_table;
    out->resident_evals += m.n_res;
    m.keysrc = m.view[0] ? 0 : -1;
    uint32_t v0 = argmax_key(&m, T_NONE);
    /* odd weight per event: a different victim at any one event changes the sum */
    out->victim_digest += ((uint64_t)v0 + 1) * ((2 * (uint64_t)m.ev + 1) * 0x9e3779b97f4a7c15ULL);

    if (kind == K_ARRIVE) {
      /* eq. (hr-amat), eq. (prered), eq. (reuse) */
      uint64_t len = ev_len[e];
      uint64_t dlen = len - len_prev;
      uint64_t kb = kvb[sid];
      out->requests++;
      out->tokens_total += len;
      uint32_t tier0 = x->tier;
      if (tier0 == T_SRAM || tier0 == T_HBM) {
        double t_mem = tier0 == T_SRAM ? p->t_s_ns_per_B : p->t_h_ns_per_B;
        if (tier0 == T_SRAM) out->hit_sram++; else out->hit_hbm++;
        if (tier0 == T_SRAM && x->prefetched) out->prefetch_hits++;
        double a = (double)(len * kb) * t_mem;
        double b = (double)(len_prev * kb) * t_mem;
        double c = (double)dlen * p->t_p_ns_per_tok;
        out->amat_sum_ns += a;
        out->ttft_sum_ns += b + c;
        out->tokens_computed += dlen;
        release(&m, sid);
      } else {
        out->miss++;
        double a = (double)len * p->t_p_ns_per_tok;
        out->amat_sum_ns += a;
        out->ttft_sum_ns += a;
        out->tokens_computed += len;
        out->extra_prefill_tok += len_prev;
      }
      x->prefetched = 0;
      x->len = (uint32_t)len;
      place(&m, sid, tier0 == T_HBM ? T_HBM : T_SRAM);
    } else if (kind == K_GAP_START) {
      if (p->tide && now >= m.dma_free_at) tide(&m, sid, now, st);
    } else {
      if (x->tier == T_NONE) m.n_table--;
    }

    if (m.view[0]) {
      int sync = (p->dual_sync == 1 && kind != K_DONE) ||
                 (p->dual_sync == 2 && kind == K_ARRIVE && out->requests % 8 == 0) ||
                 (p->dual_sync == 3 && kind == K_GAP_START);
      if (sync)
        for (int k = 0; k < 2; k++) memcpy(m.view[k], m.s, (size_t)n_sess * sizeof(sess_t));
    }
    if (st) {
      st->used_sram = m.used[T_SRAM];
      st->used_hbm = m.used[T_HBM];
      st->n_res = (uint32_t)m.n_res;
      st->n_table = (uint32_t)m.n_table;
      st->victim = v0;
    }
    out->events++;
  }
  clock_gettime(CLOCK_MONOTONIC, &t1);
  if (elapsed_ns)
    *elapsed_ns = (uint64_t)(t1.tv_sec - t0.tv_sec) * 1000000000ULL + (uint64_t)(t1.tv_nsec - t0.tv_nsec);
  if (log_len) *log_len = m.log_len;
  if (counts_out)
    for (int t = 0; t < LUT_LEN; t++) {
      counts_out[t] = m.hd[t];
      counts_out[LUT_LEN + t] = m.hn[t];
    }
  free(m.s);
  free(m.view[0]);
  free(m.view[1]);
  free(m.recip);
  return rc;
}

/*
 * Runs n_rows simulations one after another, each exactly as orc_run does
 * (no decision log, no per-event states): a driver over orc_run for batches.
 * The traces are concatenated: trace k holds events [ev_off[k], ev_off[k+1])
 * of the ev_* arrays and sessions [ss_off[k], ss_off[k+1]) of kvb.  Row i
 * replays trace row_trace[i] with the hazard counts lut_d/lut_n + 51 *
 * row_lut[i] and writes out[i]; elapsed_ns (optional) receives the summed
 * event-loop time.  ev_tool is concatenated like the events; eta holds the
 * ETA table of each trace (ETA_CLASSES waits per trace).  Every row runs;
 * the first non-zero orc_run code is returned.
 */
int orc_run_batch(const orc_params* rows, uint32_t n_rows, const uint32_t* row_trace,
                  const uint32_t* row_lut, const uint64_t* ev_off, const uint64_t* ss_off,
                  const uint64_t* ev_t, const uint32_t* ev_sid, const uint32_t* ev_info,
                  const uint32_t* ev_len, const uint64_t* ev_next, const uint32_t* kvb,
                  const uint32_t* lut_d, const uint32_t* lut_n, uint64_t max_events,
                  orc_counters* out, uint64_t* elapsed_ns, const uint32_t* ev_tool,
                  const uint64_t* eta) {
  int rc_all = ORC_OK;
  uint64_t total = 0;
  for (uint32_t i = 0; i < n_rows; i++) {
    uint32_t k = row_trace[i];
    uint64_t e0 = ev_off[k], n_ev = ev_off[k + 1] - e0, s0 = ss_off[k];
    uint64_t ns = 0;
    int rc = orc_run(&rows[i], n_ev, ev_t + e0, ev_sid + e0, ev_info + e0, ev_len + e0,
                     ev_next + e0, (uint32_t)(ss_off[k + 1] - s0), kvb + s0,
                     lut_d + (uint64_t)LUT_LEN * row_lut[i], lut_n + (uint64_t)LUT_LEN * row_lut[i],
                     max_events, &out[i], NULL, 0, NULL, NULL, NULL, &ns, ev_tool + e0,
                     eta + (uint64_t)ETA_CLASSES * k);
    total += ns;
    if (rc != ORC_OK && rc_all == ORC_OK) rc_all = rc;
  }
  if (elapsed_ns) *elapsed_ns = total;
  return rc_all;
}

/* Layout version of the structs above. */
uint32_t orc_version(void) { return 1; }
