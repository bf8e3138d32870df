// sim.hip -- the batched UNISON event simulation on gfx950.
//
// One simulation replays one trace through Algorithm 1: per event it writes
// the register file (eq. (gap), eq. (ema)), scores every table entry (the
// register-file scan of eq. (pipe)), evicts the argmax victim while
// eq. (cap) is violated, and on a gap onset with a free DMA engine runs the
// TIDE pass (eq. (budget), eq. (promote), eq. (demote)).  Accounting follows
// eq. (hr-amat) and eq. (prered).
//
// The event loop of a simulation is sequential; parallelism comes from
// running many simulations at once and from the scan inside each event.
// Two table layouts share one event engine:
//   RegTable<G, EPL>  a group of G lanes (a quarter, half or whole wave) per
//                     simulation; each lane owns EPL sessions (sid = j*G +
//                     lane) and keeps their register-file entries in VGPRs.
//                     Scores are computed per entry and reduced with
//                     cross-lane shuffles inside the group: no LDS traffic
//                     and no barriers for the table.
//   MemTable<BLOCK>   one workgroup per simulation; the table lives in the
//                     workspace (HBM / L2 / MALL) and each event streams the
//                     populated window of it with coalesced 8-byte loads;
//                     block reductions go through LDS.
// All per-simulation scalars (capacities in use, DMA state, counters) are
// replicated in every lane of the group and updated identically, so control
// flow is uniform within a group.
#include <hip/hip_runtime.h>

#include "unison_device.h"

#pragma clang fp contract(off)

namespace unison {

struct Cand {
  uint64_t key;
  uint32_t sid;
};

__device__ __forceinline__ bool max_better(uint64_t ka, uint32_t sa, uint64_t kb, uint32_t sb) {
  return ka > kb || (ka == kb && sa < sb);
}
__device__ __forceinline__ bool min_better(uint64_t ka, uint32_t sa, uint64_t kb, uint32_t sb) {
  return ka < kb || (ka == kb && sa < sb);
}
__device__ __forceinline__ Cand cand_none_max() { return Cand{0ull, kNone}; }
__device__ __forceinline__ Cand cand_none_min() { return Cand{~0ull, kNone}; }

// Butterfly reduction over aligned groups of W lanes; every lane of the
// group ends with the same winner (ties to the smaller session id).
template <int W, bool MAX>
__device__ __forceinline__ Cand reduce_group(Cand c) {
#pragma unroll
  for (int m = 1; m < W; m <<= 1) {
    uint64_t ok = __shfl_xor(c.key, m, W);
    uint32_t os = __shfl_xor(c.sid, m, W);
    bool take = MAX ? max_better(ok, os, c.key, c.sid) : min_better(ok, os, c.key, c.sid);
    c.key = take ? ok : c.key;
    c.sid = take ? os : c.sid;
  }
  return c;
}

template <int W>
__device__ __forceinline__ uint64_t reduce_sum_group(uint64_t v) {
#pragma unroll
  for (int m = 1; m < W; m <<= 1) v += __shfl_xor(v, m, W);
  return v;
}

struct Entry {
  uint32_t meta;
  float g;
  uint64_t gq;
  uint32_t len;
  uint32_t kvb;
  uint64_t last;
  uint64_t next;
};

// What a key needs besides the entry: policy, hazard table, penalty.
struct KeyCtx {
  uint32_t pol;
  uint32_t smode;
  const float* hf;      // LDS [52]
  const uint32_t* hq;   // LDS [52]
  float P;
  uint32_t lambda;
  uint64_t p_z;
};

// "Larger key = evict first".  SPEAR: the score (eq. (esp) or eq. (scoreq));
// completed sessions take S_max.  LRU / timeout: older last event first.
// Belady: later next arrival first.
__device__ __forceinline__ uint64_t key_of(const KeyCtx& K, uint32_t meta, float g, uint64_t gq,
                                           uint64_t last, uint64_t next) {
  if (K.pol == kSpear) {
    uint32_t t = meta_turn(meta);
    t = t < 50u ? t : 50u;
    bool done = meta_phase(meta) == kDoneP;
    if (K.smode) {
      uint64_t s = spear_fixed(K.hq[t], gq, K.lambda, K.p_z);
      return done ? ~0ull : s;
    }
    float s = spear_f32(K.hf[t], g, K.P);
    return done ? 0x7F800000ull : (uint64_t)__float_as_uint(s);
  }
  if (K.pol == kBelady) return next;
  return ~0ull - last;
}

// ------------------------------------------------------------------ tables

template <int G, int EPL>
struct RegTable {
  uint32_t lane;
  uint32_t meta[EPL];
  float g[EPL];
  uint64_t gq[EPL];
  uint32_t len[EPL];
  uint32_t kvb[EPL];
  uint64_t last[EPL];
  uint64_t next[EPL];
  uint64_t key[EPL];

  __device__ __forceinline__ uint32_t sid_of(int j) const { return (uint32_t)j * G + lane; }

  template <class T>
  __device__ __forceinline__ T pick(const T (&a)[EPL], uint32_t js) const {
    T v = a[0];
#pragma unroll
    for (int j = 1; j < EPL; ++j) v = (js == (uint32_t)j) ? a[j] : v;
    return v;
  }

  __device__ __forceinline__ void event_begin() {}
  __device__ __forceinline__ void grow(uint32_t) {}

  __device__ __forceinline__ Entry read(uint32_t sid) const {
    uint32_t owner = sid % G, js = sid / G;
    Entry e;
    e.meta = __shfl(pick(meta, js), owner, G);
    e.g = __shfl(pick(g, js), owner, G);
    e.gq = __shfl(pick(gq, js), owner, G);
    e.len = __shfl(pick(len, js), owner, G);
    e.kvb = __shfl(pick(kvb, js), owner, G);
    e.last = __shfl(pick(last, js), owner, G);
    e.next = __shfl(pick(next, js), owner, G);
    return e;
  }
  // size in bytes and meta of one entry
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    uint32_t owner = sid % G, js = sid / G;
    uint32_t l = __shfl(pick(len, js), owner, G);
    uint32_t k = __shfl(pick(kvb, js), owner, G);
    m = __shfl(pick(meta, js), owner, G);
    size = (uint64_t)l * k;
  }

  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    uint32_t owner = sid % G, js = sid / G;
    bool mine = lane == owner;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      bool w = mine && js == (uint32_t)j;
      meta[j] = w ? e.meta : meta[j];
      g[j] = w ? e.g : g[j];
      gq[j] = w ? e.gq : gq[j];
      len[j] = w ? e.len : len[j];
      last[j] = w ? e.last : last[j];
      next[j] = w ? e.next : next[j];
    }
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) {
    uint32_t owner = sid % G, js = sid / G;
    bool mine = lane == owner;
#pragma unroll
    for (int j = 0; j < EPL; ++j) meta[j] = (mine && js == (uint32_t)j) ? m : meta[j];
  }

  // The per-event scan: every entry's key, kept for this event's reductions.
  __device__ __forceinline__ void scan(const KeyCtx& K) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) key[j] = key_of(K, meta[j], g[j], gq[j], last[j], next[j]);
  }

  // argmax / argmin of the keys over evictable entries in `tier` (0 = any).
  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx&) const {
    Cand c = MAX ? cand_none_max() : cand_none_min();
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      bool ok = evictable(meta[j]) && (tier == 0 || meta_tier(meta[j]) == tier);
      uint32_t s = sid_of(j);
      bool take = ok && (MAX ? max_better(key[j], s, c.key, c.sid) : min_better(key[j], s, c.key, c.sid));
      c.key = take ? key[j] : c.key;
      c.sid = take ? s : c.sid;
    }
    return reduce_group<G, MAX>(c);
  }
  __device__ __forceinline__ Cand argmax_first(uint32_t tier, const KeyCtx& K) const {
    return select<true>(tier, K);
  }

  // Smallest evictable session idle for longer than ttl (timeout policy).
  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) const {
    Cand c = cand_none_min();
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      bool ok = evictable(meta[j]) && now - last[j] > ttl;
      uint32_t s = sid_of(j);
      bool take = ok && s < c.sid;
      c.sid = take ? s : c.sid;
      c.key = take ? 0ull : c.key;
    }
    return reduce_group<G, false>(c).sid;
  }
};

// Table in the workspace, one workgroup per simulation.
template <int BLOCK>
struct MemTable {
  static constexpr int NW = BLOCK / 64;
  uint64_t* mg;
  uint64_t* gq;
  uint32_t* len;
  uint64_t* last;
  uint64_t* next;
  const uint32_t* kvb;
  uint32_t tid;
  uint32_t hi;        // entries [0, hi) can be in the table
  uint32_t parity;
  Cand* red;          // LDS [2][NW]

  __device__ __forceinline__ void event_begin() { __syncthreads(); }
  __device__ __forceinline__ void grow(uint32_t h) { hi = h; }

  // Uniform reads end with a barrier: every wave has read the entry before
  // any wave goes on to overwrite it.
  __device__ __forceinline__ Entry read(uint32_t sid) const {
    Entry e;
    uint64_t x = mg[sid];
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = gq[sid];
    e.len = len[sid];
    e.kvb = kvb[sid];
    e.last = last[sid];
    e.next = next[sid];
    __syncthreads();
    return e;
  }
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    m = (uint32_t)mg[sid];
    size = (uint64_t)len[sid] * kvb[sid];
    __syncthreads();
  }
  // Every thread stores the same values, so each thread's later loads see
  // them; reads end with a barrier and each event starts with one, so no wave
  // writes an entry that another wave has still to read.
  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    mg[sid] = (uint64_t)e.meta | ((uint64_t)__float_as_uint(e.g) << 32);
    gq[sid] = e.gq;
    len[sid] = e.len;
    last[sid] = e.last;
    next[sid] = e.next;
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) {
    uint64_t x = mg[sid];
    mg[sid] = (x & 0xFFFFFFFF00000000ull) | m;
  }

  __device__ __forceinline__ void scan(const KeyCtx&) {}

  template <bool MAX>
  __device__ __forceinline__ Cand block_reduce(Cand c) {
    c = reduce_group<64, MAX>(c);
    Cand* buf = red + parity * NW;
    parity ^= 1u;
    if ((tid & 63u) == 0) buf[tid >> 6] = c;
    __syncthreads();
    Cand r = buf[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      Cand o = buf[w];
      bool take = MAX ? max_better(o.key, o.sid, r.key, r.sid) : min_better(o.key, o.sid, r.key, r.sid);
      r = take ? o : r;
    }
    return r;
  }

  // Streams the window and reduces the keys of evictable entries in `tier`.
  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx& K) {
    Cand c = MAX ? cand_none_max() : cand_none_min();
    const bool need_gq = K.pol == kSpear && K.smode;
    for (uint32_t i = tid; i < hi; i += BLOCK) {
      uint64_t x = mg[i];
      uint32_t m = (uint32_t)x;
      float gv = __uint_as_float((uint32_t)(x >> 32));
      uint64_t k;
      if (K.pol == kSpear && !need_gq) {
        k = key_of(K, m, gv, 0, 0, 0);
      } else {
        k = key_of(K, m, gv, need_gq ? gq[i] : 0ull, K.pol != kBelady ? last[i] : 0ull,
                   K.pol == kBelady ? next[i] : 0ull);
      }
      bool ok = evictable(m) && (tier == 0 || meta_tier(m) == tier);
      bool take = ok && (MAX ? max_better(k, i, c.key, c.sid) : min_better(k, i, c.key, c.sid));
      c.key = take ? k : c.key;
      c.sid = take ? i : c.sid;
    }
    return block_reduce<MAX>(c);
  }
  // The first reduction of an event is the full-table scan.
  __device__ __forceinline__ Cand argmax_first(uint32_t tier, const KeyCtx& K) {
    return select<true>(tier, K);
  }

  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) {
    Cand c = cand_none_min();
    for (uint32_t i = tid; i < hi; i += BLOCK) {
      uint32_t m = (uint32_t)mg[i];
      if (evictable(m) && now - last[i] > ttl && i < c.sid) {
        c.sid = i;
        c.key = 0;
      }
    }
    return block_reduce<false>(c).sid;
  }
};

// ------------------------------------------------------------- the engine

struct Scalars {
  uint64_t used_s, used_h, dma_free_at, prev_t, log_len;
  uint32_t n_res, n_table, hi;
};

struct LogSink {
  unison_record* rec;  // this simulation's records, or null
  uint32_t cap;
  bool lead;           // the one lane that stores records
};

__device__ __forceinline__ void emit(unison_counters& C, Scalars& S, const LogSink& L, uint32_t ev,
                                     uint32_t op, uint32_t a, uint32_t b) {
  C.digest += rec_hash(ev, op, a, b);
  if (L.rec) {
    if (L.lead && S.log_len < L.cap) {
      unison_record r;
      r.ev = ev;
      r.op = op;
      r.a = a;
      r.b = b;
      L.rec[S.log_len] = r;
    }
    S.log_len++;
  }
}

struct TraceView {
  const uint64_t* t;
  const uint32_t* sid;
  const uint32_t* info;
  const uint32_t* len;
  const uint64_t* next;
  uint64_t n_ev;
  uint32_t n_sess;
};

template <class Tab>
__device__ __forceinline__ void release(Tab& T, Scalars& S, uint32_t sid) {
  uint64_t size;
  uint32_t m;
  T.read_size(sid, size, m);
  if (meta_tier(m) == kTierSram) S.used_s -= size; else S.used_h -= size;
  S.n_res--;
  if (meta_phase(m) == kDoneP) S.n_table--;   // a completed session leaves the table
  T.set_meta(sid, with_tier(m, kTierNone));
}

// Algorithm 1 over events [S.next, end) of one simulation.
template <class Tab>
__device__ void run_events(Tab& T, const unison_sim_params& P, const KeyCtx& K, const TraceView& tr,
                           Scalars& S, unison_counters& C, const LogSink& L, uint64_t& next_event,
                           uint64_t max_events) {
  const uint32_t pol = K.pol;
  const bool has_inf = pol == kSpear || pol == kBelady;
  const uint64_t inf_key = (pol == kSpear && !K.smode) ? 0x7F800000ull : ~0ull;
  uint64_t e = next_event;
  uint64_t end = tr.n_ev - e < max_events ? tr.n_ev : e + max_events;
  for (; e < end; ++e) {
    T.event_begin();
    const uint64_t now = tr.t[e];
    const uint32_t sid = tr.sid[e];
    const uint32_t info = tr.info[e];
    const uint32_t kind = info >> 24, turn = info & 0xFFFFFFu;
    const uint32_t ev = (uint32_t)e;
    if (sid >= tr.n_sess || now < S.prev_t || kind > kDone) {
      C.error = e + 1;
      break;
    }
    S.prev_t = now;

    // timeout policy: TTL timers that fired since the previous event
    if (pol == kTimeout) {
      for (;;) {
        uint32_t v = T.first_idle(now, P.ttl_ns);
        if (v == kNone) break;
        emit(C, S, L, ev, kOpExpire, v, kNone);
        C.expire++;
        release(T, S, v);
      }
    }

    // Alg. 1: write e into R; on gap_end update the EMA
    Entry x = T.read(sid);
    const uint32_t ph = meta_phase(x.meta), tier0 = meta_tier(x.meta);
    uint32_t len_prev = x.len;
    bool bad;
    if (kind == kArrive) {
      if (turn == 0) {
        bad = ph != kUnseen;
        x.g = 0.0f;
        x.gq = 0;
        x.len = 0;
        len_prev = 0;
      } else {
        bad = ph != kGap || turn != meta_turn(x.meta) + 1 || tr.len[e] < x.len;
        uint64_t gap = now - x.last;  // eq. (gap)
        x.g = ema_f32(x.g, gap);
        x.gq = ema_int(x.gq, gap, P.b_g, P.tau_ns);
      }
      x.meta = make_meta(kServing, tier0, turn);
    } else {
      bad = ph != kServing;
      x.meta = make_meta(kind == kGapStart ? kGap : kDoneP, tier0, meta_turn(x.meta));
      x.next = kind == kGapStart ? tr.next[e] : ~0ull;
    }
    if (bad) {
      C.error = e + 1;
      break;
    }
    x.last = now;
    if (kind == kArrive && turn == 0) {
      S.n_table++;
      if (sid + 1 > S.hi) S.hi = sid + 1;
      T.grow(S.hi);
    }
    T.write(sid, x);

    // the register-file scan: every table entry is scored; its argmax over
    // evictable residents is this event's victim index
    C.score_evals += S.n_table;
    C.resident_evals += S.n_res;
    T.scan(K);
    const Cand v0 = T.argmax_first(0, K);
    C.victim_digest += rec_hash(ev, kOpVictim, v0.sid, kNone);

    if (kind == kArrive) {
      // eq. (hr-amat), eq. (prered), eq. (reuse)
      const uint64_t ln = tr.len[e];
      const uint64_t dlen = ln - len_prev;
      const uint64_t kb = x.kvb;
      C.requests++;
      C.tokens_total += ln;
      if (tier0 != kTierNone) {
        const double t_mem = tier0 == kTierSram ? P.t_s_ns_per_B : P.t_h_ns_per_B;
        if (tier0 == kTierSram) C.hit_sram++; else C.hit_hbm++;
        const double a = (double)(ln * kb) * t_mem;
        const double b = (double)((uint64_t)len_prev * kb) * t_mem;
        const double c = (double)dlen * P.t_p_ns_per_tok;
        C.amat_sum_ns += a;
        C.ttft_sum_ns += b + c;
        C.tokens_computed += dlen;
        const uint64_t old = (uint64_t)len_prev * kb;
        if (tier0 == kTierSram) S.used_s -= old; else S.used_h -= old;
        S.n_res--;
      } else {
        C.miss++;
        const double a = (double)ln * P.t_p_ns_per_tok;
        C.amat_sum_ns += a;
        C.ttft_sum_ns += a;
        C.tokens_computed += ln;
        C.extra_prefill_tok += len_prev;
      }
      x.len = (uint32_t)ln;
      x.meta = with_tier(x.meta, kTierNone);
      T.write(sid, x);

      // Alg. 1 capacity branch: evict the argmax victim until the session fits
      const uint64_t size = ln * kb;
      const uint32_t pref = tier0 == kTierHbm ? kTierHbm : kTierSram;
      const uint32_t other = pref == kTierSram ? kTierHbm : kTierSram;
      if (size > P.cap_sram_B && size > P.cap_hbm_B) {
        emit(C, S, L, ev, kOpBypass, sid, kNone);
        C.bypass++;
      } else {
        bool first = true;
        for (;;) {
          const bool slot = (uint64_t)S.n_res + 1 <= P.n_slots;
          const bool fit_s = slot && S.used_s + size <= P.cap_sram_B;
          const bool fit_h = slot && S.used_h + size <= P.cap_hbm_B;
          const bool fit_p = pref == kTierSram ? fit_s : fit_h;
          const bool fit_o = pref == kTierSram ? fit_h : fit_s;
          if (fit_p || fit_o) {
            const uint32_t t = fit_p ? pref : other;
            if (t == kTierSram) S.used_s += size; else S.used_h += size;
            S.n_res++;
            T.set_meta(sid, with_tier(x.meta, t));
            emit(C, S, L, ev, kOpPlace, sid, t);
            break;
          }
          // the event's own scan result is the first victim: the arriving
          // session was never evictable, so releasing it changed nothing
          const Cand v = first ? v0 : T.template select<true>(0, K);
          first = false;
          if (v.sid == kNone) {
            emit(C, S, L, ev, kOpBypass, sid, kNone);
            C.bypass++;
            break;
          }
          emit(C, S, L, ev, kOpEvict, v.sid, kNone);
          C.evict++;
          release(T, S, v.sid);
        }
      }
    } else if (kind == kGapStart) {
      if (P.tide && now >= S.dma_free_at) {
        // eq. (budget) / eq. (budgetq): Delta is the session's gap EMA in us
        uint64_t delta_us;
        if (pol == kSpear && K.smode) {
          unsigned __int128 d = ((unsigned __int128)x.gq * P.tau_ns) / 1000u;
          delta_us = d > (unsigned __int128)~0ull ? ~0ull : (uint64_t)d;
        } else {
          delta_us = (uint64_t)x.g;
        }
        const uint64_t budget = sat_mul(delta_us, P.dma_B_per_us);
        uint64_t left = budget, moved = 0;
        C.tide_passes++;
        for (;;) {
          const Cand p = T.template select<false>(kTierHbm, K);  // eq. (promote)
          if (p.sid == kNone) break;
          if (has_inf && p.key == inf_key) break;
          uint64_t sp;
          uint32_t mp;
          T.read_size(p.sid, sp, mp);
          if (S.used_s + sp <= P.cap_sram_B && sp <= left) {
            S.used_h -= sp;
            S.used_s += sp;
            T.set_meta(p.sid, with_tier(mp, kTierSram));
            left -= sp;
            moved += sp;
            emit(C, S, L, ev, kOpPromote, p.sid, kNone);
            C.promote++;
            continue;
          }
          const Cand d = T.template select<true>(kTierSram, K);  // eq. (demote)
          if (d.sid == kNone) break;
          uint64_t sd;
          uint32_t md;
          T.read_size(d.sid, sd, md);
          const bool legal = p.key < d.key && sp <= left && sd <= left - sp &&
                             S.used_s - sd + sp <= P.cap_sram_B && S.used_h - sp + sd <= P.cap_hbm_B;
          if (!legal) break;
          S.used_s = S.used_s - sd + sp;
          S.used_h = S.used_h - sp + sd;
          T.set_meta(p.sid, with_tier(mp, kTierSram));
          T.set_meta(d.sid, with_tier(md, kTierHbm));
          left -= sp + sd;
          moved += sp + sd;
          emit(C, S, L, ev, kOpSwap, p.sid, d.sid);
          C.swap++;
        }
        if (moved) {
          // DMA busy for ceil(moved * 1000 / B) ns
          unsigned __int128 ns = ((unsigned __int128)moved * 1000u + P.dma_B_per_us - 1u) / P.dma_B_per_us;
          unsigned __int128 fin = (unsigned __int128)now + ns;
          S.dma_free_at = fin > (unsigned __int128)~0ull ? ~0ull : (uint64_t)fin;
        }
        C.dma_bytes += moved;
      }
    } else {
      if (tier0 == kTierNone) S.n_table--;
    }
    C.events++;
  }
  next_event = e;
}

// Hazard tables of one simulation into LDS (h as fp32 and as UQ0.b_h).
__device__ __forceinline__ void load_lut(const uint32_t* d, const uint32_t* n, uint32_t lambda,
                                         float* hf, uint32_t* hq, uint32_t lane, uint32_t width) {
  for (uint32_t t = lane; t < kLut; t += width) {
    hf[t] = hazard_f32(d[t], n[t]);
    hq[t] = hazard_q(d[t], n[t], lambda);
  }
}

__device__ __forceinline__ void load_scalars(const SimState& st, Scalars& S) {
  S.used_s = st.used_s;
  S.used_h = st.used_h;
  S.dma_free_at = st.dma_free_at;
  S.prev_t = st.prev_t;
  S.log_len = st.log_len;
  S.n_res = st.n_res;
  S.n_table = st.n_table;
  S.hi = st.hi;
}

__device__ __forceinline__ void store_scalars(SimState& st, const Scalars& S, uint64_t next_event) {
  st.next_event = next_event;
  st.used_s = S.used_s;
  st.used_h = S.used_h;
  st.dma_free_at = S.dma_free_at;
  st.prev_t = S.prev_t;
  st.log_len = S.log_len;
  st.n_res = S.n_res;
  st.n_table = S.n_table;
  st.hi = S.hi;
}

__device__ __forceinline__ uint32_t sim_policy(const SimArgs& a, const unison_sim_params& P) {
  return a.policy_override == UNISON_POLICY_PARAMS ? P.policy : a.policy_override;
}

// --------------------------------------------------------------- kernels

template <int G, int EPL>
__global__ __launch_bounds__(256) void sim_regs_kernel(SimArgs a) {
  constexpr int GROUPS = 256 / G;
  __shared__ float s_hf[GROUPS][52];
  __shared__ uint32_t s_hq[GROUPS][52];
  const uint32_t gtid = blockIdx.x * 256u + threadIdx.x;
  const uint32_t sim = gtid / G;
  const uint32_t lane = gtid % G;
  const uint32_t grp = threadIdx.x / G;
  const bool live = sim < a.n_sims;
  const uint32_t simc = live ? sim : 0u;
  const unison_sim_params P = a.params[simc];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  load_lut(a.lut_d + (size_t)P.lut * kLut, a.lut_n + (size_t)P.lut * kLut, lambda, s_hf[grp],
           s_hq[grp], lane, G);
  __syncthreads();
  if (!live) return;

  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb, ee - eb,
               n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  RegTable<G, EPL> T;
  T.lane = lane;
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const uint32_t s = (uint32_t)j * G + lane;
    const bool in = s < n_sess;
    T.kvb[j] = in ? a.sess_kvb[sb + s] : 0u;
    if (cont && in) {
      const uint64_t x = a.t_mg[tb + s];
      T.meta[j] = (uint32_t)x;
      T.g[j] = __uint_as_float((uint32_t)(x >> 32));
      T.gq[j] = a.t_gq[tb + s];
      T.len[j] = a.t_len[tb + s];
      T.last[j] = a.t_last[tb + s];
      T.next[j] = a.t_next[tb + s];
    } else {
      T.meta[j] = 0;
      T.g[j] = 0.0f;
      T.gq[j] = 0;
      T.len[j] = 0;
      T.last[j] = 0;
      T.next[j] = ~0ull;
    }
    T.key[j] = 0;
  }

  Scalars S;
  unison_counters C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = a.counters[sim];
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{0, 0, 0, 0, 0, 0, 0, 0};
    C = unison_counters{};
  }
  KeyCtx K{sim_policy(a, P), P.score_mode, s_hf[grp], s_hq[grp], P.penalty_us, lambda, P.p_z};
  LogSink L{(a.flags & UNISON_RUN_LOG) && a.log_cap ? a.log + (size_t)sim * a.log_cap : nullptr,
            a.log_cap, lane == 0};
  if (C.error == 0) {
    if (n_sess > (uint32_t)(G * EPL)) {
      C.error = ~0ull;  // the launcher picks a variant that holds the trace
    } else {
      run_events(T, P, K, tr, S, C, L, next_event, a.max_events);
    }
  }

#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const uint32_t s = (uint32_t)j * G + lane;
    if (s < n_sess) {
      a.t_mg[tb + s] = (uint64_t)T.meta[j] | ((uint64_t)__float_as_uint(T.g[j]) << 32);
      a.t_gq[tb + s] = T.gq[j];
      a.t_len[tb + s] = T.len[j];
      a.t_last[tb + s] = T.last[j];
      a.t_next[tb + s] = T.next[j];
    }
  }
  if (lane == 0) {
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = C;
  }
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void sim_block_kernel(SimArgs a) {
  __shared__ float s_hf[52];
  __shared__ uint32_t s_hq[52];
  __shared__ Cand s_red[2 * (BLOCK / 64)];
  const uint32_t sim = blockIdx.x;
  const uint32_t tid = threadIdx.x;
  const unison_sim_params P = a.params[sim];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  load_lut(a.lut_d + (size_t)P.lut * kLut, a.lut_n + (size_t)P.lut * kLut, lambda, s_hf, s_hq, tid,
           BLOCK);

  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb, ee - eb,
               n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  MemTable<BLOCK> T;
  T.mg = a.t_mg + tb;
  T.gq = a.t_gq + tb;
  T.len = a.t_len + tb;
  T.last = a.t_last + tb;
  T.next = a.t_next + tb;
  T.kvb = a.sess_kvb + sb;
  T.tid = tid;
  T.parity = 0;
  T.red = s_red;
  if (!cont) {
    for (uint32_t i = tid; i < n_sess; i += BLOCK) {
      T.mg[i] = 0;
      T.gq[i] = 0;
      T.len[i] = 0;
      T.last[i] = 0;
      T.next[i] = ~0ull;
    }
  }
  __syncthreads();

  Scalars S;
  unison_counters C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = a.counters[sim];
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{0, 0, 0, 0, 0, 0, 0, 0};
    C = unison_counters{};
  }
  if (S.hi > n_sess) S.hi = n_sess;  // never scan past the trace's sessions
  T.hi = S.hi;
  KeyCtx K{sim_policy(a, P), P.score_mode, s_hf, s_hq, P.penalty_us, lambda, P.p_z};
  LogSink L{(a.flags & UNISON_RUN_LOG) && a.log_cap ? a.log + (size_t)sim * a.log_cap : nullptr,
            a.log_cap, tid == 0};
  if (C.error == 0) run_events(T, P, K, tr, S, C, L, next_event, a.max_events);
  __syncthreads();
  if (tid == 0) {
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = C;
  }
}

// eq. (hazard) counts over a population of turn counts.
__global__ __launch_bounds__(256) void hazard_counts_kernel(const uint32_t* turns, uint32_t n,
                                                            uint32_t* d_out, uint32_t* n_out) {
  __shared__ uint32_t s_end[kLut + 1];   // #{T = t+1} for t < 51, and #{T > 51}
  for (uint32_t t = threadIdx.x; t <= kLut; t += 256) s_end[t] = 0;
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < n; i += 256) {
    uint32_t T = turns[i];
    if (T >= 1) atomicAdd(&s_end[T - 1 < kLut ? T - 1 : kLut], 1u);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // n(t) = #{T > t} = sessions ending at t or later
    uint32_t alive = s_end[kLut];
    for (int t = (int)kLut - 1; t >= 0; --t) {
      alive += s_end[t];
      n_out[t] = alive;
      d_out[t] = s_end[t];
    }
  }
}

}  // namespace unison

// ------------------------------------------------------------ launchers

namespace unison {

hipError_t launch_sim(const SimArgs& a, uint32_t max_sess_in_batch, hipStream_t stream, int force_variant) {
  // Variant by the largest trace: register tables while a group can hold
  // every session, the streamed table beyond.
  int v = force_variant;
  if (v < 0) {
    if (max_sess_in_batch <= 16) v = 0;
    else if (max_sess_in_batch <= 64) v = 1;
    else if (max_sess_in_batch <= 256) v = 2;
    else v = 3;
  }
  const uint32_t n = a.n_sims;
  switch (v) {
    case 0: hipLaunchKernelGGL((sim_regs_kernel<16, 1>), dim3((n * 16 + 255) / 256), dim3(256), 0, stream, a); break;
    case 1: hipLaunchKernelGGL((sim_regs_kernel<64, 1>), dim3((n * 64 + 255) / 256), dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL((sim_regs_kernel<64, 4>), dim3((n * 64 + 255) / 256), dim3(256), 0, stream, a); break;
    case 4: hipLaunchKernelGGL((sim_regs_kernel<4, 4>), dim3((n * 4 + 255) / 256), dim3(256), 0, stream, a); break;
    case 5: hipLaunchKernelGGL((sim_regs_kernel<8, 2>), dim3((n * 8 + 255) / 256), dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL((sim_block_kernel<256>), dim3(n), dim3(256), 0, stream, a); break;
  }
  return hipGetLastError();
}

uint32_t sim_variant_capacity(int v) {
  switch (v) {
    case 0: return 16;
    case 1: return 64;
    case 2: return 256;
    case 4: return 16;
    case 5: return 16;
    default: return UNISON_MAX_SESSIONS;
  }
}

hipError_t launch_hazard_counts(const uint32_t* turns, uint32_t n, uint32_t* d, uint32_t* nn,
                                hipStream_t stream) {
  hipLaunchKernelGGL(hazard_counts_kernel, dim3(1), dim3(256), 0, stream, turns, n, d, nn);
  return hipGetLastError();
}

}  // namespace unison
