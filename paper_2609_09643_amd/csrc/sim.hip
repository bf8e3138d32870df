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
//   RegTable<G, EPL>  a group of G lanes (4 to 64) per simulation; each lane
//                     owns EPL sessions (sid = j*G + lane) and keeps their
//                     register-file entries in VGPRs.  Keys are computed per
//                     entry and reduced with DPP butterflies inside the
//                     group (quad_perm, row_half_mirror, row_mirror, then
//                     ds_swizzle / bpermute across rows): no LDS traffic and
//                     no barriers for the table.
//   MemTable<BLOCK>   one workgroup per simulation; the table lives in the
//                     workspace (HBM / L2 / MALL) and each event streams the
//                     populated window of it with coalesced 8-byte loads;
//                     block reductions go through LDS.
// The engine is instantiated per policy and score mode, so each simulation
// keeps only the register-file fields its keys read.  All per-simulation
// scalars are replicated in every lane of the group and updated identically,
// so control flow is uniform within a group.
#include <hip/hip_runtime.h>

#include "unison_device.h"

#pragma clang fp contract(off)

namespace unison {

// ------------------------------------------------------- cross-lane moves

// Every pattern used here reads a lane of the same row, so no lane needs a
// fallback value (mov_dpp leaves the destination's old value unspecified).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}

// Partner value for butterfly step M.  Before step M every aligned block of
// M lanes holds one value; the partner lane lies in the sibling block.
template <int M>
__device__ __forceinline__ uint32_t xchg(uint32_t v) {
  if constexpr (M == 1) return dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  else if constexpr (M == 2) return dpp<0x4E>(v);  // quad_perm [2,3,0,1]
  else if constexpr (M == 4) return dpp<0x141>(v);  // row_half_mirror
  else if constexpr (M == 8) return dpp<0x140>(v);  // row_mirror
  else if constexpr (M == 16) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);  // xor 16
  else return (uint32_t)__shfl_xor((int)v, 32);
}

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

// Max (MAX) or min of a 32-bit value over each aligned group of W lanes;
// every lane of the group ends with it.
template <int W, int M, bool MAX>
__device__ __forceinline__ uint32_t group_ext32(uint32_t v) {
  if constexpr (M < W) {
    const uint32_t o = xchg<M>(v);
    return group_ext32<W, M * 2, MAX>(MAX ? (o > v ? o : v) : (o < v ? o : v));
  } else {
    return v;
  }
}

// Max (MAX) or min of a packed 64-bit value over each aligned group of W
// lanes, as two 32-bit words, most significant first: the group's best high
// word, then the best low word among the lanes that hold it (the others enter
// the empty value).  Each word's step is one max or min with a lane permute,
// which the compiler folds into one DPP instruction, where a 64-bit step
// needs two permutes, a compare and two selects.
template <int W, bool MAX>
__device__ __forceinline__ uint64_t reduce_words(uint64_t c) {
  const uint32_t hi = (uint32_t)(c >> 32);
  const uint32_t h = group_ext32<W, 1, MAX>(hi);
  const uint32_t lo = hi == h ? (uint32_t)c : (MAX ? 0u : ~0u);
  return ((uint64_t)h << 32) | group_ext32<W, 1, MAX>(lo);
}

template <int W, int M>
__device__ __forceinline__ uint32_t reduce_min32(uint32_t c) {
  if constexpr (M < W) {
    const uint32_t o = xchg<M>(c);
    return reduce_min32<W, M * 2>(o < c ? o : c);
  } else {
    return c;
  }
}

// Every lane of an aligned group of W lanes ends with the winner (ties to
// the smaller session id): the key's two words, most significant first, then
// the smallest id among the lanes still tied, each over the lanes that hold
// the best word so far (the others enter the empty value).
template <int W, bool MAX>
__device__ __forceinline__ Cand reduce_group(Cand c) {
  const uint32_t empty = MAX ? 0u : ~0u;
  const uint32_t khi = (uint32_t)(c.key >> 32), klo = (uint32_t)c.key;
  const uint32_t h = group_ext32<W, 1, MAX>(khi);
  const bool tied = khi == h;
  const uint32_t l = group_ext32<W, 1, MAX>(tied ? klo : empty);
  const uint32_t s = group_ext32<W, 1, false>(tied && klo == l ? c.sid : ~0u);
  return Cand{((uint64_t)h << 32) | l, s};
}

// Whole-wavefront max (MAX) or min of a 32-bit value, uniform: a DPP
// butterfly inside each row of 16 lanes, then the four row results compared
// in scalar registers (no cross-row permute through the LDS crossbar).
template <bool MAX>
__device__ __forceinline__ uint32_t ext32(uint32_t a, uint32_t b) {
  return MAX ? (a > b ? a : b) : (a < b ? a : b);
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_ext32(uint32_t v) {
  v = ext32<MAX>(v, xchg<1>(v));
  v = ext32<MAX>(v, xchg<2>(v));
  v = ext32<MAX>(v, xchg<4>(v));
  v = ext32<MAX>(v, xchg<8>(v));
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
  const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
  return ext32<MAX>(ext32<MAX>(r0, r1), ext32<MAX>(r2, r3));
}
// One phase of a lexicographic wavefront reduction over N words per lane:
// the best word M among the active ones; with NARROW, a word stays active
// only where it equals M, so the next phase breaks the ties.
template <bool MAX, bool NARROW, int N>
__device__ __forceinline__ uint32_t lex_phase(const uint32_t (&w)[N], bool (&act)[N]) {
  uint32_t v = MAX ? 0u : ~0u;
#pragma unroll
  for (int k = 0; k < N; ++k) v = act[k] ? ext32<MAX>(v, w[k]) : v;
  const uint32_t m = wave_ext32<MAX>(v);
  if constexpr (NARROW) {
#pragma unroll
    for (int k = 0; k < N; ++k) act[k] = act[k] && w[k] == m;
  }
  return m;
}

// Sum mod 2^64 over the wavefront; every lane ends with it.
__device__ __forceinline__ uint64_t wave_sum64_step(uint64_t v, uint32_t lo, uint32_t hi) {
  return v + (((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ uint64_t wave_sum64(uint64_t v) {
  v = wave_sum64_step(v, xchg<1>((uint32_t)v), xchg<1>((uint32_t)(v >> 32)));
  v = wave_sum64_step(v, xchg<2>((uint32_t)v), xchg<2>((uint32_t)(v >> 32)));
  v = wave_sum64_step(v, xchg<4>((uint32_t)v), xchg<4>((uint32_t)(v >> 32)));
  v = wave_sum64_step(v, xchg<8>((uint32_t)v), xchg<8>((uint32_t)(v >> 32)));
  v = wave_sum64_step(v, xchg<16>((uint32_t)v), xchg<16>((uint32_t)(v >> 32)));
  v = wave_sum64_step(v, xchg<32>((uint32_t)v), xchg<32>((uint32_t)(v >> 32)));
  return v;
}

// Pins a value to a vector register.  A workgroup-per-simulation kernel keeps
// its long-lived per-simulation state (pool usage, counters) there: held in
// scalar registers it would exceed them and spill on every event.
__device__ __forceinline__ uint32_t in_vgpr(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ uint64_t in_vgpr(uint64_t v) {
  return ((uint64_t)in_vgpr((uint32_t)(v >> 32)) << 32) | in_vgpr((uint32_t)v);
}
__device__ __forceinline__ double in_vgpr(double v) {
  return __longlong_as_double((long long)in_vgpr((uint64_t)__double_as_longlong(v)));
}

__device__ __forceinline__ uint32_t uni32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}
__device__ __forceinline__ uint64_t uni64(uint64_t v) {
  return ((uint64_t)uni32((uint32_t)(v >> 32)) << 32) | uni32((uint32_t)v);
}
// A condition every lane of the wavefront evaluates alike (UNI), as a scalar
// branch condition: values pinned to vector registers would otherwise make
// the compiler treat the branch as divergent (exec masking, merges of every
// live value at the join).
template <bool UNI>
__device__ __forceinline__ bool uc(bool c) {
  if constexpr (UNI) return __builtin_amdgcn_ballot_w64(c) != 0ull;
  else return c;
}

// ------------------------------------------------------------ keys

template <uint32_t POL, uint32_t SMODE>
struct Pol {
  static constexpr bool spear = POL == kSpear;
  static constexpr bool fixed = spear && SMODE == 1;
  static constexpr bool belady = POL == kBelady;
  static constexpr bool eta = POL == kEta;
  // the key is the session's next arrival: true (Belady) or predicted (ETA)
  static constexpr bool nextkey = belady || eta;
  static constexpr bool timeout = POL == kTimeout;
  static constexpr bool recency = POL == kLru || POL == kTimeout;
  static constexpr bool has_inf = spear || nextkey;
  static constexpr uint64_t inf_key = (spear && !fixed) ? 0x7F800000ull : ~0ull;
};

// The simulation's hazard table lives in LDS: its counts d(t), n(t) of
// eq. (hazard) and both derived forms, h as fp32 and h_q (eq. (hq)).  An
// online table (online_cap > 0) grows by one session at each of the first
// online_cap completions.
struct KeyCtx {
  float* hf;            // LDS [52]
  uint32_t* hq;         // LDS [52]
  uint32_t* hd;         // LDS [52]
  uint32_t* hn;         // LDS [52]
  float P;
  uint32_t lambda;
  uint64_t p_z;
  bool pack44;          // times fit 44 bits and ids 20 bits: recency / Belady keys pack
  uint32_t online_cap;  // completions an online table still may count; 0: fixed table
  const uint64_t* eta;  // the trace's ETA table: expected wait per tool class, ns (global)
  uint32_t recip_bits;  // eq. (t1) by a reciprocal of this many fraction bits; 0: exact
};

// Adds a completed session of Tn turns to the counts (n(t) += 1 for t < Tn,
// d(Tn - 1) += 1) and rebuilds the entries it changed; t is split over
// `width` cooperating lanes starting at `lane`.
__device__ __forceinline__ void hazard_add_counts(const KeyCtx& K, uint32_t Tn, uint32_t lane,
                                                  uint32_t width) {
  for (uint32_t t = lane; t < kLut; t += width) {
    const uint32_t dn = t < Tn ? 1u : 0u;
    const uint32_t dd = t + 1u == Tn ? 1u : 0u;
    if (dn | dd) {
      const uint32_t d = K.hd[t] + dd;
      const uint32_t n = K.hn[t] + dn;
      K.hd[t] = d;
      K.hn[t] = n;
      K.hf[t] = hazard_f32(d, n);
      K.hq[t] = hazard_q(d, n, K.lambda);
    }
  }
}

// The hazard entry eq. (hazard) / eq. (hq) of a session at turn index t
// (clamped to 50): fp32 bits of h for the fp32 score, h_q for the integer one.
template <uint32_t POL, uint32_t SMODE>
__device__ __forceinline__ uint32_t hazard_of(const KeyCtx& K, uint32_t meta) {
  using PT = Pol<POL, SMODE>;
  if constexpr (PT::spear) {
    uint32_t t = meta_turn(meta);
    t = t < 50u ? t : 50u;
    return PT::fixed ? K.hq[t] : __float_as_uint(K.hf[t]);
  } else {
    return 0u;
  }
}

// "Larger key = evict first".  SPEAR: the score (eq. (esp) or eq. (scoreq))
// from the entry's hazard value hz (hazard_of); completed sessions take
// S_max.  LRU / timeout: older last event first.  Belady: later next arrival
// first.
template <uint32_t POL, uint32_t SMODE>
__device__ __forceinline__ uint64_t key_of(const KeyCtx& K, uint32_t meta, uint32_t hz, float g,
                                           uint64_t gq, uint64_t last, uint64_t next) {
  using PT = Pol<POL, SMODE>;
  if constexpr (PT::spear) {
    const bool done = meta_phase(meta) == kDoneP;
    if constexpr (PT::fixed) {
      const uint64_t s = spear_fixed(hz, gq, K.lambda, K.p_z, K.recip_bits);
      return done ? ~0ull : s;
    } else {
      const float s = spear_f32(__uint_as_float(hz), g, K.P);
      return done ? 0x7F800000ull : (uint64_t)__float_as_uint(s);
    }
  } else if constexpr (PT::nextkey) {
    return next;
  } else {
    return ~0ull - last;
  }
}

// A session's timer has fired (now - last > ttl) exactly when last lies below
// this threshold: last never exceeds now, and nothing fires while now <= ttl.
__device__ __forceinline__ uint64_t idle_threshold(uint64_t now, uint64_t ttl) {
  return now > ttl ? now - ttl : 0ull;
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

struct TraceView {
  const uint64_t* t;
  const uint32_t* sid;
  const uint32_t* info;
  const uint32_t* len;
  const uint64_t* next;
  const uint32_t* tool;  // or null: every gap is tool class 0
  uint64_t n_ev;
  uint32_t n_sess;
};

struct Ev {
  uint64_t t;
  uint32_t sid, info, len, tool;
  uint64_t next;
};

// The event record; the next arrival only where the key reads it (Belady),
// the tool class only where it predicts one (ETA).
template <bool NEXT, bool TOOL>
__device__ __forceinline__ Ev load_ev(const TraceView& tr, uint64_t e) {
  Ev v;
  v.t = tr.t[e];
  v.sid = tr.sid[e];
  v.info = tr.info[e];
  v.len = tr.len[e];
  v.next = NEXT ? tr.next[e] : ~0ull;
  v.tool = (TOOL && tr.tool) ? tr.tool[e] : 0u;
  return v;
}

// Event records one event ahead: the next record's loads are in flight while
// the current event is processed.
template <bool NEXT, bool TOOL>
struct AheadReader {
  const TraceView& tr;
  uint64_t end;
  Ev cur;
  __device__ __forceinline__ AheadReader(const TraceView& t, uint64_t e, uint64_t end_, void*)
      : tr(t), end(end_), cur(load_ev<NEXT, TOOL>(t, e)) {}
  __device__ __forceinline__ Ev take(uint64_t e) {
    const Ev c = cur;
    cur = load_ev<NEXT, TOOL>(tr, e + 1 < end ? e + 1 : e);
    return c;
  }
};

// Event records 64 at a time for a lone wavefront: lane l holds event base + l
// of the current window and of the next, whose loads are issued a whole
// window ahead; an event's fields are read out of its lane.
template <bool NEXT, bool TOOL>
struct WindowReader {
  const TraceView& tr;
  uint64_t end, base;
  uint32_t lane;
  uint64_t ct, cn, nt, nn;
  uint32_t csid, cinfo, clen, ctool, nsid, ninfo, nlen, ntool;
  __device__ __forceinline__ void load(uint64_t b, uint64_t& t, uint32_t& sid, uint32_t& info,
                                       uint32_t& len, uint64_t& nx, uint32_t& tool) const {
    const uint64_t e = b + lane;
    const bool ok = e < end;
    const uint64_t i = ok ? e : (end ? end - 1 : 0);
    t = tr.t[i];
    sid = tr.sid[i];
    info = tr.info[i];
    len = tr.len[i];
    nx = NEXT ? tr.next[i] : ~0ull;
    tool = (TOOL && tr.tool) ? tr.tool[i] : 0u;
  }
  __device__ __forceinline__ WindowReader(const TraceView& t, uint64_t e, uint64_t end_, void*)
      : tr(t), end(end_), base(e), lane(threadIdx.x & 63u) {
    load(base, ct, csid, cinfo, clen, cn, ctool);
    load(base + 64, nt, nsid, ninfo, nlen, nn, ntool);
  }
  __device__ __forceinline__ static uint64_t lane64(uint64_t v, int k) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), k) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, k);
  }
  // Session id of event e, the event after the one take() returned last (at
  // the end of the trace, the last event's: the window repeats it).
  __device__ __forceinline__ uint32_t peek_sid(uint64_t e) const {
    const uint64_t k = e - base;
    return k < 64 ? (uint32_t)__builtin_amdgcn_readlane((int)csid, (int)k)
                  : (uint32_t)__builtin_amdgcn_readlane((int)nsid, (int)(k - 64));
  }
  __device__ __forceinline__ Ev take(uint64_t e) {
    if (e - base >= 64) {
      ct = nt; csid = nsid; cinfo = ninfo; clen = nlen; cn = nn; ctool = ntool;
      base += 64;
      load(base + 64, nt, nsid, ninfo, nlen, nn, ntool);
    }
    const int k = (int)(e - base);
    Ev v;
    v.t = lane64(ct, k);
    v.sid = (uint32_t)__builtin_amdgcn_readlane((int)csid, k);
    v.info = (uint32_t)__builtin_amdgcn_readlane((int)cinfo, k);
    v.len = (uint32_t)__builtin_amdgcn_readlane((int)clen, k);
    v.next = NEXT ? lane64(cn, k) : ~0ull;
    v.tool = TOOL ? (uint32_t)__builtin_amdgcn_readlane((int)ctool, k) : 0u;
    return v;
  }
};

// Events through a window in LDS (one wavefront): events [base, base + 128)
// of the trace, reloaded 64 further on every 64 events, so that the event
// after the current one is always there.  An event is read back from LDS as
// uniform values; the window's registers hold no load in flight across
// events (a load still in flight across the loop would be waited for at
// every event, with every table store the wavefront issued).
template <bool NEXT, bool TOOL>
struct LdsWindowReader {
  static constexpr uint32_t kWin = 128;
  static constexpr uint32_t kBytes = kWin * (2 * sizeof(uint64_t) + 4 * sizeof(uint32_t));
  const TraceView& tr;
  uint64_t end, base;
  uint32_t lane;
  uint64_t* wt;
  uint64_t* wn;
  uint32_t* wsid;
  uint32_t* winfo;
  uint32_t* wlen;
  uint32_t* wtool;
  __device__ __forceinline__ void fill() {
#pragma unroll
    for (uint32_t h = 0; h < kWin; h += 64) {
      const uint64_t e = base + h + lane;
      const uint64_t i = e < end ? e : end - 1;  // end > 0: a reader exists only for events
      const uint64_t t = tr.t[i];
      const uint32_t sid = tr.sid[i], info = tr.info[i], len = tr.len[i];
      const uint64_t nx = NEXT ? tr.next[i] : ~0ull;
      const uint32_t tool = (TOOL && tr.tool) ? tr.tool[i] : 0u;
      wt[h + lane] = t;
      wn[h + lane] = nx;
      wsid[h + lane] = sid;
      winfo[h + lane] = info;
      wlen[h + lane] = len;
      wtool[h + lane] = tool;
    }
  }
  __device__ __forceinline__ LdsWindowReader(const TraceView& t, uint64_t e, uint64_t end_, void* w)
      : tr(t), end(end_), base(e), lane(threadIdx.x & 63u) {
    wt = reinterpret_cast<uint64_t*>(w);
    wn = wt + kWin;
    wsid = reinterpret_cast<uint32_t*>(wn + kWin);
    winfo = wsid + kWin;
    wlen = winfo + kWin;
    wtool = wlen + kWin;
    fill();
  }
  // Session id of event e, the event after the one take() returned last.
  __device__ __forceinline__ uint32_t peek_sid(uint64_t e) const {
    return uni32(wsid[(uint32_t)(e - base)]);
  }
  __device__ __forceinline__ Ev take(uint64_t e) {
    if (e - base >= 64) {
      base += 64;
      fill();
    }
    const uint32_t k = (uint32_t)(e - base);
    Ev v;
    v.t = uni64(wt[k]);
    v.sid = uni32(wsid[k]);
    v.info = uni32(winfo[k]);
    v.len = uni32(wlen[k]);
    v.next = NEXT ? uni64(wn[k]) : ~0ull;
    v.tool = TOOL ? uni32(wtool[k]) : 0u;
    return v;
  }
};

// ------------------------------------------------------------ tables

// Most resident-cache slots per thread of the streamed-table kernels.
constexpr uint32_t kCacheSlotsMax = 8;

template <int G, int EPL, uint32_t POL, uint32_t SMODE>
struct RegTable {
  using PT = Pol<POL, SMODE>;
  static constexpr bool kViews = false;  // no dual-design copies
  // Gap onsets reduce their scan victim and TIDE's candidates separately:
  // fusing the three reductions made this kernel slower (0.518 vs 0.498 ms).
  static constexpr bool kFuseGap = false;
  // TIDE's demotion candidate is reduced only when the pass needs it.
  static constexpr bool kDeferD = true;
  static constexpr bool kLaneDigest = false;
  static constexpr bool kPrefetch = false;
  __device__ __forceinline__ void* window() const { return nullptr; }
  struct Pf {};
  __device__ __forceinline__ Pf prefetch_issue(uint32_t) { return Pf{}; }
  __device__ __forceinline__ void prefetch_land(const Pf&) {}
  template <bool N, bool T>
  using Reader = AheadReader<N, T>;
  uint32_t lane;
  uint32_t meta[EPL];
  float g[EPL];
  uint64_t gq[EPL];
  uint32_t len[EPL];
  uint32_t kvb[EPL];
  uint64_t last[EPL];
  uint64_t next[EPL];
  // Each entry's key in the form its reductions compare (packed_key).  A key
  // reads only its own entry's fields and the hazard table, so it is
  // recomputed for the event's entry at each scan, and for all entries when
  // the hazard table changes.
  uint64_t pk[EPL];
  uint32_t hz[EPL];   // hazard value at the entry's turn (hazard_of), set when the turn changes

  __device__ __forceinline__ uint32_t sid_of(int j) const { return (uint32_t)j * G + lane; }

  template <class T>
  __device__ __forceinline__ T pick(const T (&a)[EPL], uint32_t js) const {
    T v = a[0];
#pragma unroll
    for (int j = 1; j < EPL; ++j) v = (js == (uint32_t)j) ? a[j] : v;
    return v;
  }
  template <class T>
  __device__ __forceinline__ T bcast(const T (&a)[EPL], uint32_t sid) const {
    return __shfl(pick(a, sid / G), sid % G, G);
  }

  __device__ __forceinline__ void event_begin() {}
  __device__ __forceinline__ void grow(uint32_t) {}

  __device__ __forceinline__ Entry read(uint32_t sid) const {
    Entry e;
    e.meta = bcast(meta, sid);
    e.g = bcast(g, sid);
    e.gq = PT::fixed ? bcast(gq, sid) : 0ull;
    e.len = bcast(len, sid);
    e.kvb = bcast(kvb, sid);
    e.last = bcast(last, sid);
    e.next = PT::nextkey ? bcast(next, sid) : ~0ull;
    return e;
  }
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    const uint32_t l = bcast(len, sid);
    const uint32_t k = bcast(kvb, sid);
    m = bcast(meta, sid);
    size = (uint64_t)l * k;
  }
  // The fields a gap onset or completion reads: meta and the gap EMAs.
  __device__ __forceinline__ void read_end(uint32_t sid, Entry& e) const {
    e.meta = bcast(meta, sid);
    e.g = bcast(g, sid);
    e.gq = PT::fixed ? bcast(gq, sid) : 0ull;
  }
  // A gap onset or completion: the new meta x.meta (its EMAs x.g, x.gq are
  // unchanged), the event time t and, at a gap onset, the next arrival nx.
  __device__ __forceinline__ void write_end(uint32_t sid, const Entry& x, uint64_t t, uint64_t nx) {
    const uint32_t m = x.meta;
    const uint32_t js = sid / G;
    const bool mine = lane == sid % G;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool w = mine && js == (uint32_t)j;
      meta[j] = w ? m : meta[j];
      last[j] = w ? t : last[j];
      if constexpr (PT::nextkey) next[j] = w ? nx : next[j];
    }
  }

  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    const uint32_t js = sid / G;
    const bool mine = lane == sid % G;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool w = mine && js == (uint32_t)j;
      meta[j] = w ? e.meta : meta[j];
      g[j] = w ? e.g : g[j];
      if constexpr (PT::fixed) gq[j] = w ? e.gq : gq[j];
      len[j] = w ? e.len : len[j];
      last[j] = w ? e.last : last[j];
      if constexpr (PT::nextkey) next[j] = w ? e.next : next[j];
    }
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) {
    const uint32_t js = sid / G;
    const bool mine = lane == sid % G;
#pragma unroll
    for (int j = 0; j < EPL; ++j) meta[j] = (mine && js == (uint32_t)j) ? m : meta[j];
  }
  // A new turn index: look its hazard up once instead of at every scan.
  __device__ __forceinline__ void set_turn(uint32_t sid, uint32_t m, const KeyCtx& K) {
    if constexpr (PT::spear) {
      const uint32_t h = hazard_of<POL, SMODE>(K, m);
      const uint32_t js = sid / G;
      const bool mine = lane == sid % G;
#pragma unroll
      for (int j = 0; j < EPL; ++j) hz[j] = (mine && js == (uint32_t)j) ? h : hz[j];
    }
  }
  __device__ __forceinline__ void set_len_meta(uint32_t sid, uint32_t l, uint32_t m) {
    const uint32_t js = sid / G;
    const bool mine = lane == sid % G;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool w = mine && js == (uint32_t)j;
      meta[j] = w ? m : meta[j];
      len[j] = w ? l : len[j];
    }
  }

  // An entry's key as its reductions take it: an fp32 score in the upper
  // word (select32); a recency or next-arrival time as k44 << 20 when times
  // pack (select44); otherwise the key itself.
  __device__ __forceinline__ static uint64_t packed_key(const KeyCtx& K, uint32_t m, uint32_t h,
                                                        float gv, uint64_t gqv, uint64_t lastv,
                                                        uint64_t nextv) {
    if constexpr (PT::spear) {
      const uint64_t k = key_of<POL, SMODE>(K, m, h, gv, gqv, 0ull, 0ull);
      return PT::fixed ? k : k << 32;
    } else {
      constexpr uint64_t kCap = (1ull << 44) - 1;
      // predicted returns (ETA) may pass 2^44: they compare unpacked
      if ((PT::recency || PT::belady) && K.pack44) {
        uint64_t k44;
        if constexpr (PT::belady) k44 = nextv < kCap ? nextv : kCap;
        else k44 = kCap - lastv;
        return k44 << 20;
      }
      return key_of<POL, SMODE>(K, m, h, gv, gqv, lastv, nextv);
    }
  }
  __device__ __forceinline__ uint64_t packed_key_at(const KeyCtx& K, int j) const {
    return packed_key(K, meta[j], hz[j], g[j], PT::fixed ? gq[j] : 0ull, PT::recency ? last[j] : 0ull,
                      PT::nextkey ? next[j] : 0ull);
  }
  __device__ __forceinline__ void rescore_all(const KeyCtx& K) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) pk[j] = packed_key_at(K, j);
  }

  // The per-event scan.  Only the event's session changed a field a key
  // reads, so its key is the one to recompute; every other entry keeps its
  // key from its own latest event.
  __device__ __forceinline__ void scan(const KeyCtx& K, uint32_t sid) {
    const uint32_t js = sid / G;
    const bool mine = lane == sid % G;
    const uint64_t k = packed_key(K, pick(meta, js), pick(hz, js), pick(g, js),
                                  PT::fixed ? pick(gq, js) : 0ull, PT::recency ? pick(last, js) : 0ull,
                                  PT::nextkey ? pick(next, js) : 0ull);
#pragma unroll
    for (int j = 0; j < EPL; ++j) pk[j] = (mine && js == (uint32_t)j) ? k : pk[j];
  }

  // argmax / argmin of the keys over evictable entries in `tier` (0 = any).
  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx& K) const {
    if constexpr (PT::spear && !PT::fixed) return select32<MAX>(tier);
    if constexpr (PT::recency || PT::belady)
      if (K.pack44) return select44<MAX>(tier);
    Cand c = MAX ? cand_none_max() : cand_none_min();
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool ok = evictable(meta[j]) && (tier == 0 || meta_tier(meta[j]) == tier);
      const uint32_t s = sid_of(j);
      const bool take =
          ok && (MAX ? max_better(pk[j], s, c.key, c.sid) : min_better(pk[j], s, c.key, c.sid));
      c.key = take ? pk[j] : c.key;
      c.sid = take ? s : c.sid;
    }
    return reduce_group<G, MAX>(c);
  }
  __device__ __forceinline__ Cand argmax_first(const KeyCtx& K) const { return select<true>(0, K); }

  // 32-bit keys (fp32 scores) reduce as one packed u64: key << 32 with the
  // complement of the id for argmax (ties to the smaller id) and the id itself
  // for argmin; 0 and 2^64 - 1 are the empty values.
  template <bool MAX>
  __device__ __forceinline__ Cand select32(uint32_t tier) const {
    uint64_t c = MAX ? 0ull : ~0ull;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool ok = evictable(meta[j]) && (tier == 0 || meta_tier(meta[j]) == tier);
      const uint32_t s = sid_of(j);
      const uint64_t p = pk[j] | (MAX ? (0xFFFFFFFFu - s) : s);
      c = ok && (MAX ? p > c : p < c) ? p : c;
    }
    c = reduce_words<G, MAX>(c);
    const bool none = MAX ? c == 0ull : c == ~0ull;
    const uint32_t lo = (uint32_t)c;
    return Cand{c >> 32, none ? kNone : (MAX ? 0xFFFFFFFFu - lo : lo)};
  }

  // Recency and Belady keys are times; below 2^44 - 1 they pack with a 20-bit
  // id as k44 << 20 | id field.  Recency: k44 = 2^44 - 1 - last (the order of
  // 2^64 - 1 - last); Belady: k44 = min(next, 2^44 - 1), the cap standing for
  // "never".  The id field is 2^20 - 1 - id for argmax and id for argmin,
  // so ties go to the smaller id; ids stay below 2^20 - 1, which keeps 0 and
  // 2^64 - 1 free as the empty values.
  template <bool MAX>
  __device__ __forceinline__ Cand select44(uint32_t tier) const {
    constexpr uint64_t kCap = (1ull << 44) - 1;
    uint64_t c = MAX ? 0ull : ~0ull;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool ok = evictable(meta[j]) && (tier == 0 || meta_tier(meta[j]) == tier);
      const uint32_t s = sid_of(j);
      const uint64_t p = pk[j] | (MAX ? (0xFFFFFu - s) : s);
      c = ok && (MAX ? p > c : p < c) ? p : c;
    }
    c = reduce_words<G, MAX>(c);
    const bool none = MAX ? c == 0ull : c == ~0ull;
    const uint32_t lo = (uint32_t)c & 0xFFFFFu;
    const uint64_t k44 = c >> 20;
    uint64_t key;
    if constexpr (PT::belady) key = k44 == kCap ? ~0ull : k44;
    else key = k44 | ~kCap;
    return Cand{key, none ? kNone : (MAX ? 0xFFFFFu - lo : lo)};
  }

  // TIDE's two candidates, eq. (promote) and eq. (demote).
  __device__ __forceinline__ void select_pd(const KeyCtx& K, Cand& p, Cand& d) const {
    p = select<false>(kTierHbm, K);
    d = select<true>(kTierSram, K);
  }
  __device__ __forceinline__ Cand select_p(const KeyCtx& K) const { return select<false>(kTierHbm, K); }
  __device__ __forceinline__ Cand select_d(const KeyCtx& K) const { return select<true>(kTierSram, K); }

  // Online hazard table: does it still count completions?  Then add one and
  // refresh every entry's hazard value, so the next scan rescores them all.
  __device__ __forceinline__ bool hazard_open(const KeyCtx& K) const { return K.hn[0] < K.online_cap; }
  __device__ __forceinline__ void hazard_add(const KeyCtx& K, uint32_t Tn) {
    hazard_add_counts(K, Tn, lane, G);
#pragma unroll
    for (int j = 0; j < EPL; ++j) hz[j] = hazard_of<POL, SMODE>(K, meta[j]);
    rescore_all(K);
  }

  // Smallest evictable session idle for longer than ttl (timeout policy);
  // kNone if there is none.
  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) const {
    const uint64_t thr = idle_threshold(now, ttl);
    uint32_t c = kNone;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool ok = evictable(meta[j]) && last[j] < thr;
      const uint32_t s = sid_of(j);
      c = ok && s < c ? s : c;
    }
    // no timer fired anywhere in the wavefront: nothing to reduce
    if (__builtin_amdgcn_ballot_w64(c != kNone) == 0) return kNone;
    return reduce_min32<G, 1>(c);
  }
};

// Table in the workspace, one workgroup per simulation.  Uniform values read
// from memory or LDS go through readfirstlane so the engine's scalars live in
// SGPRs.
template <int BLOCK, uint32_t POL, uint32_t SMODE, bool VIEWS, bool CACHE>
struct MemTable {
  using PT = Pol<POL, SMODE>;
  static constexpr int NW = BLOCK / 64;
  static constexpr bool kViews = VIEWS;  // instantiated with the dual design's copies
  // A gap onset's scan and TIDE's first candidates share one pass and one
  // barrier (the dual design scans different copies for the two engines).
  static constexpr bool kFuseGap = !VIEWS;
  static constexpr bool kDeferD = false;
  static constexpr bool kLaneDigest = false;
  static constexpr bool kPrefetch = false;
  __device__ __forceinline__ void* window() const { return nullptr; }
  struct Pf {};
  __device__ __forceinline__ Pf prefetch_issue(uint32_t) { return Pf{}; }
  __device__ __forceinline__ void prefetch_land(const Pf&) {}
  template <bool N, bool T>
  using Reader = AheadReader<N, T>;
  uint64_t* mg;
  uint64_t* gq;
  uint32_t* len;
  uint64_t* last;
  uint64_t* next;
  const uint32_t* kvb;
  // The dual design (eq. (rf), eq. (stale)): the eviction engine's (copy 0)
  // and TIDE's (copy 1) copies of the key fields, [4 fields][max_sessions]
  // each.  Keys come from the copy set_src chose, or from the live table.
  // Eligibility and tiers are always live.
  uint64_t* view0;
  uint64_t* view1;
  uint32_t view_stride;  // max_sessions
  const uint64_t* kmg;   // the key fields the scans read
  const uint64_t* kgq;
  const uint64_t* klast;
  const uint64_t* knext;

  // Keys from copy c (0 or 1), or from the live table for c < 0.
  __device__ __forceinline__ void set_src(int c) {
    const uint64_t* v = c == 0 ? view0 : view1;
    const bool live = c < 0;
    kmg = live ? mg : v;
    kgq = live ? gq : v + view_stride;
    klast = live ? last : v + 2 * (size_t)view_stride;
    knext = live ? next : v + 3 * (size_t)view_stride;
  }
  uint32_t tid;
  uint32_t hi;        // entries [0, hi) can be in the table
  uint32_t parity;
  Cand* red;          // LDS [2][3][NW]: two alternating sets of up to three reductions
  // Residency bits of this thread's entries (sid = tid + k * BLOCK): bit
  // k % 32 of LDS word res[(k / 32) * BLOCK + tid].  Only the owning thread
  // reads or writes its words, so they need no barrier; the scans visit set
  // bits only, since no other entry can be a victim or a migrant.
  uint32_t* res;
  // Resident cache (CACHE: a table streamed from the workspace).  The meta /
  // gap word, the aux field (aux_table) and the key of this thread's
  // resident entries, in LDS slots o = s * BLOCK + tid, s < rc_cap, which
  // only the owning thread reads or writes.  While the thread has at most rc_cap
  // residents the slots hold all of them and its scans read no table memory;
  // with more, it reads them from the table, and it refills the slots once
  // it is back within them.
  uint64_t* rc_mg;
  uint64_t* rc_aux;
  uint64_t* rc_key;   // the entry's key, kept current with its fields and the hazard table
  uint32_t* rc_k;     // k of the entry in slot s (sid = tid + k * BLOCK)
  KeyCtx kc;          // the simulation's key context
  uint32_t rc_cap;
  uint32_t rc_used;   // bit s: slot s is taken
  uint32_t n_mine;    // residents of this thread
  uint32_t w_sid;     // the entry of the latest write(), its meta / gap word and aux field
  uint64_t w_x;
  uint64_t w_aux;

  // The one field besides meta and the gap EMA that an entry's key reads:
  // the integer gap EMA (fixed-point score), the next arrival (Belady) or
  // the last event time (LRU, timeout).
  __device__ __forceinline__ static uint64_t aux_pick(uint64_t q, uint64_t l, uint64_t n) {
    return PT::fixed ? q : PT::nextkey ? n : PT::recency ? l : 0ull;
  }
  __device__ __forceinline__ uint64_t aux_table(uint32_t i) const {
    if constexpr (PT::fixed) return gq[i];
    else if constexpr (PT::nextkey) return next[i];
    else if constexpr (PT::recency) return last[i];
    else return 0ull;
  }
  // The key of an entry with meta / gap word x and aux field aux.
  __device__ __forceinline__ uint64_t key_from(uint64_t x, uint64_t aux) const {
    const uint32_t m = (uint32_t)x;
    return key_of<POL, SMODE>(kc, m, hazard_of<POL, SMODE>(kc, m),
                              __uint_as_float((uint32_t)(x >> 32)), aux, aux, aux);
  }

  // Refills the slots from the table with every resident of this thread
  // (at most rc_cap of them).
  __device__ __forceinline__ void rc_refill() {
    uint32_t n = 0;
    const uint32_t nw = res_words();
    for (uint32_t w = 0; w < nw; ++w) {
      for (uint32_t bits = res[w * BLOCK + tid]; bits; bits &= bits - 1u) {
        const uint32_t k = w * 32u + (uint32_t)__builtin_ctz(bits);
        const uint32_t i = tid + k * BLOCK;
        const uint32_t o = n * BLOCK + tid;
        const uint64_t x = mg[i], aux = aux_table(i);
        rc_k[o] = k;
        rc_mg[o] = x;
        rc_aux[o] = aux;
        rc_key[o] = key_from(x, aux);
        ++n;
      }
    }
    rc_used = n ? (0xFFFFFFFFu >> (32u - n)) : 0u;
  }

  // Keeps the owner's residency bit, and its resident cache, in step with
  // an entry's new meta m: its whole new meta / gap word is x when has_x,
  // else m over the old gap EMA; its aux field changes to aux when has_aux.
  __device__ __forceinline__ void note(uint32_t sid, uint32_t m, uint64_t x, bool has_x,
                                       uint64_t aux, bool has_aux) {
    if ((sid & (BLOCK - 1u)) != tid) return;
    const uint32_t k = sid / BLOCK;
    uint32_t* w = res + (k >> 5) * BLOCK + tid;
    const uint32_t bit = 1u << (k & 31u);
    const bool was = (*w & bit) != 0;
    const bool now = meta_tier(m) != kTierNone;
    *w = now ? (*w | bit) : (*w & ~bit);
    if constexpr (CACHE) {
      constexpr uint64_t kGapHalf = 0xFFFFFFFF00000000ull;
      uint32_t slot = kNone;
      if (was && n_mine <= rc_cap) {
        for (uint32_t u = rc_used; u; u &= u - 1u) {
          const uint32_t t = (uint32_t)__builtin_ctz(u);
          if (rc_k[t * BLOCK + tid] == k) slot = t;
        }
      }
      if (now && !was) {
        ++n_mine;
        if (n_mine <= rc_cap) {
          // a placement follows the arriving session's write(); otherwise
          // the entry's other fields come from the table
          const bool latest = sid == w_sid;
          if (!has_x) x = ((latest ? w_x : mg[sid]) & kGapHalf) | m;
          if (!has_aux) aux = latest ? w_aux : aux_table(sid);
          slot = (uint32_t)__builtin_ctz(~rc_used);
          rc_used |= 1u << slot;
          const uint32_t o = slot * BLOCK + tid;
          rc_k[o] = k;
          rc_mg[o] = x;
          rc_aux[o] = aux;
          rc_key[o] = key_from(x, aux);
        } else {
          rc_used = 0;  // more residents than slots: the scans read the table
        }
      } else if (!now && was) {
        --n_mine;
        if (slot != kNone) rc_used &= ~(1u << slot);
        else if (n_mine == rc_cap) rc_refill();
      } else if (slot != kNone) {
        // a meta word alone changes the tier or the prefetch flag, which no
        // key reads; new EMAs or times change the key
        const uint32_t o = slot * BLOCK + tid;
        x = has_x ? x : (rc_mg[o] & kGapHalf) | m;
        rc_mg[o] = x;
        if (has_aux) rc_aux[o] = aux;
        if (has_x || has_aux) rc_key[o] = key_from(x, has_aux ? aux : rc_aux[o]);
      }
    }
  }
  // An entry's meta word alone: the low half of its meta / gap word.
  __device__ __forceinline__ void store_meta(uint32_t sid, uint32_t m) {
    reinterpret_cast<uint32_t*>(mg + sid)[0] = m;
  }
  // Words per thread that cover entries [0, hi).
  __device__ __forceinline__ uint32_t res_words() const { return (hi + 32u * BLOCK - 1u) / (32u * BLOCK); }

  __device__ __forceinline__ void event_begin() { __syncthreads(); }
  __device__ __forceinline__ void grow(uint32_t h) { hi = h; }

  // Uniform reads end with a barrier: every wave has read the entry before
  // any wave goes on to overwrite it.
  __device__ __forceinline__ Entry read(uint32_t sid) const {
    Entry e;
    const uint64_t x = uni64(mg[sid]);
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = PT::fixed ? uni64(gq[sid]) : 0ull;
    e.len = uni32(len[sid]);
    e.kvb = uni32(kvb[sid]);
    e.last = uni64(last[sid]);
    e.next = PT::nextkey ? uni64(next[sid]) : ~0ull;
    __syncthreads();
    return e;
  }
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    m = uni32((uint32_t)mg[sid]);
    size = (uint64_t)uni32(len[sid]) * uni32(kvb[sid]);
    __syncthreads();
  }
  __device__ __forceinline__ void read_end(uint32_t sid, Entry& e) const {
    const uint64_t x = uni64(mg[sid]);
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = PT::fixed ? uni64(gq[sid]) : 0ull;
    __syncthreads();
  }
  __device__ __forceinline__ void write_end(uint32_t sid, const Entry& e, uint64_t t, uint64_t nx) {
    const uint32_t m = e.meta;
    const uint64_t x = (uint64_t)m | ((uint64_t)__float_as_uint(e.g) << 32);
    // the event moves the key's time field (LRU / timeout: last; Belady: next)
    note(sid, m, x, true, aux_pick(e.gq, t, nx), true);
    w_sid = kNone;
    store_meta(sid, m);
    last[sid] = t;
    if constexpr (PT::nextkey) next[sid] = nx;
  }
  // Every thread stores the same values, so each thread's later loads see
  // them; reads end with a barrier and each event starts with one, so no wave
  // writes an entry that another wave has still to read.
  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    const uint64_t x = (uint64_t)e.meta | ((uint64_t)__float_as_uint(e.g) << 32);
    w_sid = sid;
    w_x = x;
    w_aux = aux_pick(e.gq, e.last, e.next);
    note(sid, e.meta, x, true, w_aux, true);
    mg[sid] = x;
    if constexpr (PT::fixed) gq[sid] = e.gq;
    len[sid] = e.len;
    last[sid] = e.last;
    if constexpr (PT::nextkey) next[sid] = e.next;
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) {
    note(sid, m, 0ull, false, 0ull, false);
    store_meta(sid, m);
  }
  __device__ __forceinline__ void set_len_meta(uint32_t sid, uint32_t l, uint32_t m) {
    set_meta(sid, m);
    len[sid] = l;
  }
  __device__ __forceinline__ void set_turn(uint32_t, uint32_t, const KeyCtx&) {}

  __device__ __forceinline__ void scan(const KeyCtx&, uint32_t) {}

  // The wavefront's best candidate as uniform values.  The scans visit
  // resident entries only, so most lanes usually hold none: up to 16
  // candidates are compared one lane at a time in scalar registers, more
  // go through the DPP butterfly.
  template <bool MAX>
  __device__ __forceinline__ Cand wave_best(Cand c) {
    uint64_t lanes = __builtin_amdgcn_ballot_w64(c.sid != kNone);
    if (__builtin_popcountll(lanes) > 16) {
      c = reduce_group<64, MAX>(c);
      return Cand{uni64(c.key), uni32(c.sid)};
    }
    Cand b = MAX ? cand_none_max() : cand_none_min();
    while (lanes) {
      const int l = __builtin_ctzll(lanes);
      lanes &= lanes - 1u;
      const uint32_t khi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(c.key >> 32), l);
      const uint32_t klo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)c.key, l);
      const uint32_t s = (uint32_t)__builtin_amdgcn_readlane((int)c.sid, l);
      const uint64_t k = ((uint64_t)khi << 32) | klo;
      const bool take = MAX ? max_better(k, s, b.key, b.sid) : min_better(k, s, b.key, b.sid);
      b.key = take ? k : b.key;
      b.sid = take ? s : b.sid;
    }
    return b;
  }


  // Lane l of every wavefront takes buf[l]: NW per reduction, up to three
  // reductions side by side (lanes [r NW, (r + 1) NW) for reduction r, an
  // argmax where is_max, else an argmin); a butterfly within each group of
  // NW lanes leaves its winner in all of them.
  __device__ __forceinline__ Cand gather_best(const Cand* buf, uint32_t n_red, uint32_t max_mask) const {
    const uint32_t l = tid & 63u;
    const uint32_t r = l / NW;
    const bool is_max = (max_mask >> (r < 3u ? r : 0u)) & 1u;
    Cand c = is_max ? cand_none_max() : cand_none_min();
    if (r < n_red) c = buf[l];
#pragma unroll
    for (uint32_t m = 1; m < (uint32_t)NW; m <<= 1) {
      uint32_t klo, khi, s;
      if (m == 1) {
        klo = xchg<1>((uint32_t)c.key); khi = xchg<1>((uint32_t)(c.key >> 32)); s = xchg<1>(c.sid);
      } else if (m == 2) {
        klo = xchg<2>((uint32_t)c.key); khi = xchg<2>((uint32_t)(c.key >> 32)); s = xchg<2>(c.sid);
      } else {
        klo = xchg<4>((uint32_t)c.key); khi = xchg<4>((uint32_t)(c.key >> 32)); s = xchg<4>(c.sid);
      }
      const uint64_t k = ((uint64_t)khi << 32) | klo;
      const bool take = is_max ? max_better(k, s, c.key, c.sid) : min_better(k, s, c.key, c.sid);
      c.key = take ? k : c.key;
      c.sid = take ? s : c.sid;
    }
    return c;
  }
  __device__ __forceinline__ static Cand lane_cand(const Cand& c, int lane) {
    const uint32_t khi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(c.key >> 32), lane);
    const uint32_t klo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)c.key, lane);
    const uint32_t s = (uint32_t)__builtin_amdgcn_readlane((int)c.sid, lane);
    return Cand{((uint64_t)khi << 32) | klo, s};
  }

  template <bool MAX>
  __device__ __forceinline__ Cand block_reduce(Cand c) {
    c = wave_best<MAX>(c);
    Cand* buf = red + parity * 3 * NW;
    parity ^= 1u;
    if ((tid & 63u) == 0) buf[tid >> 6] = c;
    __syncthreads();
    return lane_cand(gather_best(buf, 1, MAX ? 1u : 0u), 0);
  }

  // Two reductions (min, max) behind one barrier.
  __device__ __forceinline__ void block_reduce2(Cand& p, Cand& d) {
    p = wave_best<false>(p);
    d = wave_best<true>(d);
    Cand* buf = red + parity * 3 * NW;
    parity ^= 1u;
    if ((tid & 63u) == 0) {
      buf[tid >> 6] = p;
      buf[NW + (tid >> 6)] = d;
    }
    __syncthreads();
    const Cand g = gather_best(buf, 2, 0x2u);
    p = lane_cand(g, 0);
    d = lane_cand(g, NW);
  }

  // Three reductions (max, min, max) behind one barrier.
  __device__ __forceinline__ void block_reduce3(Cand& v, Cand& p, Cand& d) {
    v = wave_best<true>(v);
    p = wave_best<false>(p);
    d = wave_best<true>(d);
    Cand* buf = red + parity * 3 * NW;
    parity ^= 1u;
    if ((tid & 63u) == 0) {
      buf[tid >> 6] = v;
      buf[NW + (tid >> 6)] = p;
      buf[2 * NW + (tid >> 6)] = d;
    }
    __syncthreads();
    const Cand g = gather_best(buf, 3, 0x5u);
    v = lane_cand(g, 0);
    p = lane_cand(g, NW);
    d = lane_cand(g, 2 * NW);
  }

  __device__ __forceinline__ uint64_t key_at(const KeyCtx& K, uint32_t i, uint64_t x) const {
    const uint64_t* q = gq;
    const uint64_t* l = last;
    const uint64_t* n = next;
    if constexpr (VIEWS) {
      x = kmg[i];
      q = kgq;
      l = klast;
      n = knext;
    }
    const uint32_t m = (uint32_t)x;
    const float gv = __uint_as_float((uint32_t)(x >> 32));
    return key_of<POL, SMODE>(K, m, hazard_of<POL, SMODE>(K, m), gv, PT::fixed ? q[i] : 0ull,
                              PT::recency ? l[i] : 0ull, PT::nextkey ? n[i] : 0ull);
  }

  // f(i, x, aux, k) for each resident entry i of this thread: x its live
  // meta / gap word, aux its live aux field and k its key (from the copies
  // set_src chose, for the dual design), from the resident cache or the
  // table.
  template <class F>
  __device__ __forceinline__ void each_resident(const KeyCtx& K, F&& f) const {
    if constexpr (CACHE) {
      if (n_mine <= rc_cap) {
        // the next slot's loads issue before the current slot is used
        uint32_t u = rc_used;
        if (u) {
          uint32_t o = (uint32_t)__builtin_ctz(u) * BLOCK + tid;
          uint32_t ck = rc_k[o];
          uint64_t cx = rc_mg[o], ca = rc_aux[o], cv = rc_key[o];
          for (;;) {
            u &= u - 1u;
            const bool more = u != 0;
            o = more ? (uint32_t)__builtin_ctz(u) * BLOCK + tid : o;
            const uint32_t nk = rc_k[o];
            const uint64_t nx = rc_mg[o], na = rc_aux[o], nv = rc_key[o];
            f(tid + ck * BLOCK, cx, ca, cv);
            if (!more) break;
            ck = nk;
            cx = nx;
            ca = na;
            cv = nv;
          }
        }
        return;
      }
    }
    const uint32_t nw = res_words();
    for (uint32_t w = 0; w < nw; ++w) {
      for (uint32_t bits = res[w * BLOCK + tid]; bits; bits &= bits - 1u) {
        const uint32_t i = tid + (w * 32u + (uint32_t)__builtin_ctz(bits)) * BLOCK;
        const uint64_t x = mg[i], aux = aux_table(i);
        uint64_t k;
        if constexpr (VIEWS) {
          k = key_at(K, i, x);
        } else {
          const uint32_t m = (uint32_t)x;
          k = key_of<POL, SMODE>(K, m, hazard_of<POL, SMODE>(K, m),
                                 __uint_as_float((uint32_t)(x >> 32)), aux, aux, aux);
        }
        f(i, x, aux, k);
      }
    }
  }

  // Overwrites both copies with the live key fields of every entry.
  __device__ __forceinline__ void sync_views() {
    const size_t st = view_stride;
    for (uint32_t i = tid; i < hi; i += BLOCK) {
      const uint64_t m = mg[i], q = gq[i], l = last[i], n = next[i];
      view0[i] = m;
      view0[st + i] = q;
      view0[2 * st + i] = l;
      view0[3 * st + i] = n;
      view1[i] = m;
      view1[st + i] = q;
      view1[2 * st + i] = l;
      view1[3 * st + i] = n;
    }
    __syncthreads();
  }

  // Streams the window and reduces the keys of evictable entries in `tier`.
  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx& K) {
    Cand c = MAX ? cand_none_max() : cand_none_min();
    each_resident(K, [&](uint32_t i, uint64_t x, uint64_t, uint64_t k) {
      const uint32_t m = (uint32_t)x;
      const bool ok = evictable(m) && (tier == 0 || meta_tier(m) == tier);
      const bool take = ok && (MAX ? max_better(k, i, c.key, c.sid) : min_better(k, i, c.key, c.sid));
      c.key = take ? k : c.key;
      c.sid = take ? i : c.sid;
    });
    return block_reduce<MAX>(c);
  }
  // The first reduction of an event is the full-table scan.
  __device__ __forceinline__ Cand argmax_first(const KeyCtx& K) { return select<true>(0, K); }

  // TIDE's two candidates, eq. (promote) and eq. (demote), from one pass.
  __device__ __forceinline__ void select_pd(const KeyCtx& K, Cand& p, Cand& d) {
    Cand cp = cand_none_min(), cd = cand_none_max();
    each_resident(K, [&](uint32_t i, uint64_t x, uint64_t, uint64_t k) {
      const uint32_t m = (uint32_t)x;
      const bool ev = evictable(m);
      const bool in_h = ev && meta_tier(m) == kTierHbm;
      const bool in_s = ev && meta_tier(m) == kTierSram;
      const bool tp = in_h && min_better(k, i, cp.key, cp.sid);
      const bool td = in_s && max_better(k, i, cd.key, cd.sid);
      cp.key = tp ? k : cp.key;
      cp.sid = tp ? i : cp.sid;
      cd.key = td ? k : cd.key;
      cd.sid = td ? i : cd.sid;
    });
    block_reduce2(cp, cd);
    p = cp;
    d = cd;
  }
  // A gap onset's scan victim and TIDE's first candidates from one pass over
  // the residents and one barrier.
  __device__ __forceinline__ void scan3(const KeyCtx& K, Cand& v, Cand& p, Cand& d) {
    Cand cv = cand_none_max(), cp = cand_none_min(), cd = cand_none_max();
    each_resident(K, [&](uint32_t i, uint64_t x, uint64_t, uint64_t k) {
      const uint32_t m = (uint32_t)x;
      const bool ev = evictable(m);
      const bool tv = ev && max_better(k, i, cv.key, cv.sid);
      const bool tp = ev && meta_tier(m) == kTierHbm && min_better(k, i, cp.key, cp.sid);
      const bool td = ev && meta_tier(m) == kTierSram && max_better(k, i, cd.key, cd.sid);
      cv.key = tv ? k : cv.key;
      cv.sid = tv ? i : cv.sid;
      cp.key = tp ? k : cp.key;
      cp.sid = tp ? i : cp.sid;
      cd.key = td ? k : cd.key;
      cd.sid = td ? i : cd.sid;
    });
    block_reduce3(cv, cp, cd);
    v = cv;
    p = cp;
    d = cd;
  }

  // Online hazard table: both calls are made by the whole workgroup.
  __device__ __forceinline__ bool hazard_open(const KeyCtx& K) const {
    const uint32_t seen = uni32(K.hn[0]);
    __syncthreads();
    return seen < K.online_cap;
  }
  __device__ __forceinline__ void hazard_add(const KeyCtx& K, uint32_t Tn) {
    hazard_add_counts(K, Tn, tid, BLOCK);
    __syncthreads();
    if constexpr (CACHE) {
      // every cached key reads the table that just changed
      if (n_mine <= rc_cap) {
        for (uint32_t u = rc_used; u; u &= u - 1u) {
          const uint32_t o = (uint32_t)__builtin_ctz(u) * BLOCK + tid;
          rc_key[o] = key_from(rc_mg[o], rc_aux[o]);
        }
      }
    }
  }

  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) {
    const uint64_t thr = idle_threshold(now, ttl);
    Cand c = cand_none_min();
    // the timeout policy's aux field is the last event time
    each_resident(kc, [&](uint32_t i, uint64_t x, uint64_t last_t, uint64_t) {
      if (evictable((uint32_t)x) && last_t < thr && i < c.sid) {
        c.sid = i;
        c.key = 0;
      }
    });
    return block_reduce<false>(c).sid;
  }
};

// Digest terms of a table whose engine runs on one wavefront, queued one per
// lane and hashed 64 at a time.  Record j of the current batch sits in lane j
// (event, op, a, b); q_sum is the lane's sum of hashed records.  The scan
// victim of event v_e0 + j sits in lane j; v_sum is the lane's sum of weighted
// victims.
struct LaneQueue {
  uint32_t lane;
  uint32_t q_ev, q_op, q_a, q_b, q_n;
  uint64_t q_sum;
  uint32_t v_sid, v_n;
  uint64_t v_e0, v_sum;

  __device__ __forceinline__ void queue_init() {
    q_ev = q_op = q_a = q_b = 0u;
    q_n = 0u;
    q_sum = 0ull;
    v_sid = 0u;
    v_n = 0u;
    v_e0 = 0ull;
    v_sum = 0ull;
  }
  __device__ __forceinline__ void flush_records() {
    if (lane < q_n) q_sum += rec_hash(q_ev, q_op, q_a, q_b);
    q_n = 0u;
  }
  __device__ __forceinline__ void queue_record(uint32_t ev, uint32_t op, uint32_t a, uint32_t b) {
    const bool mine = lane == q_n;
    q_ev = mine ? ev : q_ev;
    q_op = mine ? op : q_op;
    q_a = mine ? a : q_a;
    q_b = mine ? b : q_b;
    if (++q_n == 64u) flush_records();
  }
  // The victim digest weighs event e's victim id + 1 by (2e + 1) * 0x9e3779b97f4a7c15.
  __device__ __forceinline__ void flush_victims() {
    if (lane < v_n) {
      const uint64_t e = v_e0 + lane;
      v_sum += ((uint64_t)v_sid + 1u) * ((2ull * e + 1ull) * 0x9e3779b97f4a7c15ull);
    }
    v_n = 0u;
  }
  // Events reach the queue in order, one victim each.
  __device__ __forceinline__ void queue_victim(uint64_t e, uint32_t sid) {
    if (v_n == 0u) v_e0 = e;
    v_sid = lane == v_n ? sid : v_sid;
    if (++v_n == 64u) flush_victims();
  }
  // Every queued term, summed over the wavefront mod 2^64: the record digest
  // and the victim digest still to add.
  __device__ __forceinline__ void drain(uint64_t& digest, uint64_t& victim_digest) {
    flush_records();
    flush_victims();
    digest = uni64(wave_sum64(q_sum));
    victim_digest = uni64(wave_sum64(v_sum));
    q_sum = 0ull;
    v_sum = 0ull;
  }

};

// Residents in registers, table in LDS, one wavefront per simulation.  Every
// session's entry stays in LDS (as in the LDS-resident MemTable), and each
// resident also occupies a VGPR slot of the wavefront -- its session id, meta,
// size and key -- kept current wherever the engine writes an entry.  Residents
// never exceed N_sess (eq. (cap)), so SPL slots per lane hold them all while
// N_sess <= 64 SPL: every scan and TIDE selection is then a reduction over the
// slots alone, with no table memory touched, and an event reads only its own
// session's entry.  The single wavefront's LDS accesses are in program order,
// so no barrier is needed anywhere.
template <int SPL, uint32_t POL, uint32_t SMODE>
struct SlotTable : LaneQueue {
  using PT = Pol<POL, SMODE>;
  static constexpr bool kViews = false;
  static constexpr bool kFuseGap = true;
  static constexpr bool kDeferD = false;
  // Digest terms are queued one per lane and hashed 64 at a time.
  static constexpr bool kLaneDigest = true;
  static constexpr bool kPrefetch = false;
  __device__ __forceinline__ void* window() const { return nullptr; }
  struct Pf {};
  __device__ __forceinline__ Pf prefetch_issue(uint32_t) { return Pf{}; }
  __device__ __forceinline__ void prefetch_land(const Pf&) {}
  template <bool N, bool T>
  using Reader = WindowReader<N, T>;  // events come 64 to a window, one per lane
  uint64_t* mg;
  uint64_t* gq;
  uint32_t* len;
  uint32_t* kvb;
  uint64_t* last;
  uint64_t* next;
  KeyCtx kc;
  uint32_t ssid[SPL];   // kNone: free
  uint32_t smeta[SPL];
  uint64_t skey[SPL];
  uint64_t ssize[SPL];
  // the entry of the latest write(): its key, KV bytes per token and length
  uint32_t w_sid;
  uint64_t w_key;
  uint32_t w_kvb, w_len;

  __device__ __forceinline__ uint64_t key_from(uint32_t m, float g, uint64_t q, uint64_t l,
                                               uint64_t n) const {
    return key_of<POL, SMODE>(kc, m, hazard_of<POL, SMODE>(kc, m), g, q, l, n);
  }
  // the key of entry i from its fields in LDS (per lane)
  __device__ __forceinline__ uint64_t key_at(uint32_t i) const {
    const uint64_t x = mg[i];
    return key_from((uint32_t)x, __uint_as_float((uint32_t)(x >> 32)), PT::fixed ? gq[i] : 0ull,
                    PT::recency ? last[i] : 0ull, PT::nextkey ? next[i] : ~0ull);
  }

  template <class T>
  __device__ __forceinline__ static T pick(const T (&a)[SPL], uint32_t j) {
    T v = a[0];
#pragma unroll
    for (int k = 1; k < SPL; ++k) v = j == (uint32_t)k ? a[k] : v;
    return v;
  }
  // The slot (j, lane l) holding sid; false if sid is not resident.
  __device__ __forceinline__ bool find(uint32_t sid, uint32_t& j, uint32_t& l) const {
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      const uint64_t b = __builtin_amdgcn_ballot_w64(ssid[k] == sid);
      if (b) {
        j = (uint32_t)k;
        l = (uint32_t)__builtin_ctzll(b);
        return true;
      }
    }
    return false;
  }
  __device__ __forceinline__ void put(uint32_t j, uint32_t l, uint32_t sid, uint32_t m,
                                      uint64_t key, uint64_t size) {
    const bool mine = lane == l;
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      const bool w = mine && j == (uint32_t)k;
      ssid[k] = w ? sid : ssid[k];
      smeta[k] = w ? m : smeta[k];
      skey[k] = w ? key : skey[k];
      ssize[k] = w ? size : ssize[k];
    }
  }
  __device__ __forceinline__ void set_slot_meta(uint32_t j, uint32_t l, uint32_t m) {
    const bool mine = lane == l;
#pragma unroll
    for (int k = 0; k < SPL; ++k) smeta[k] = (mine && j == (uint32_t)k) ? m : smeta[k];
  }
  __device__ __forceinline__ void set_slot_key(uint32_t j, uint32_t l, uint32_t m, uint64_t key) {
    const bool mine = lane == l;
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      const bool w = mine && j == (uint32_t)k;
      smeta[k] = w ? m : smeta[k];
      skey[k] = w ? key : skey[k];
    }
  }
  // A resident enters the first free slot.
  __device__ __forceinline__ void insert(uint32_t sid, uint32_t m, uint64_t key, uint64_t size) {
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      const uint64_t b = __builtin_amdgcn_ballot_w64(ssid[k] == kNone);
      if (b) {
        put((uint32_t)k, (uint32_t)__builtin_ctzll(b), sid, m, key, size);
        return;
      }
    }
  }
  // Meta word m of entry sid: LDS, and the resident set it implies.
  __device__ __forceinline__ void meta_to(uint32_t sid, uint32_t m) {
    if (lane == 0) reinterpret_cast<uint32_t*>(mg + sid)[0] = m;
    uint32_t j, l;
    const bool res = find(sid, j, l);
    const bool now = meta_tier(m) != kTierNone;
    if (res && !now) {
      put(j, l, kNone, 0u, 0ull, 0ull);
    } else if (res) {
      set_slot_meta(j, l, m);
    } else if (now) {
      uint64_t key, size;
      if (sid == w_sid) {
        key = w_key;
        size = (uint64_t)w_len * w_kvb;
      } else {
        key = uni64(key_at(sid));
        size = (uint64_t)uni32(len[sid]) * uni32(kvb[sid]);
      }
      insert(sid, m, key, size);
    }
  }

  __device__ __forceinline__ void event_begin() {}
  __device__ __forceinline__ void grow(uint32_t) {}

  __device__ __forceinline__ Entry read(uint32_t sid) const {
    Entry e;
    const uint64_t x = uni64(mg[sid]);
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = PT::fixed ? uni64(gq[sid]) : 0ull;
    e.len = uni32(len[sid]);
    e.kvb = uni32(kvb[sid]);
    e.last = uni64(last[sid]);
    e.next = PT::nextkey ? uni64(next[sid]) : ~0ull;
    return e;
  }
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    uint32_t j, l;
    if (find(sid, j, l)) {
      const uint64_t sz = pick(ssize, j);
      size = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(sz >> 32), (int)l) << 32) |
             (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)sz, (int)l);
      m = (uint32_t)__builtin_amdgcn_readlane((int)pick(smeta, j), (int)l);
    } else {
      m = uni32((uint32_t)mg[sid]);
      size = (uint64_t)uni32(len[sid]) * uni32(kvb[sid]);
    }
  }
  __device__ __forceinline__ void read_end(uint32_t sid, Entry& e) const {
    const uint64_t x = uni64(mg[sid]);
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = PT::fixed ? uni64(gq[sid]) : 0ull;
  }
  __device__ __forceinline__ void write_end(uint32_t sid, const Entry& e, uint64_t t, uint64_t nx) {
    if (lane == 0) {
      reinterpret_cast<uint32_t*>(mg + sid)[0] = e.meta;
      last[sid] = t;
      if constexpr (PT::nextkey) next[sid] = nx;
    }
    w_sid = kNone;
    uint32_t j, l;
    if (find(sid, j, l)) set_slot_key(j, l, e.meta, key_from(e.meta, e.g, e.gq, t, nx));
  }
  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    if (lane == 0) {
      mg[sid] = (uint64_t)e.meta | ((uint64_t)__float_as_uint(e.g) << 32);
      if constexpr (PT::fixed) gq[sid] = e.gq;
      len[sid] = e.len;
      last[sid] = e.last;
      if constexpr (PT::nextkey) next[sid] = e.next;
    }
    w_sid = sid;
    w_key = key_from(e.meta, e.g, e.gq, e.last, e.next);
    w_kvb = e.kvb;
    w_len = e.len;
    uint32_t j, l;
    if (find(sid, j, l)) set_slot_key(j, l, e.meta, w_key);
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) { meta_to(sid, m); }
  __device__ __forceinline__ void set_len_meta(uint32_t sid, uint32_t l, uint32_t m) {
    if (lane == 0) len[sid] = l;
    if (sid == w_sid) w_len = l;
    meta_to(sid, m);
  }
  __device__ __forceinline__ void set_turn(uint32_t, uint32_t, const KeyCtx&) {}
  __device__ __forceinline__ void scan(const KeyCtx&, uint32_t) {}

  // Candidates reduce as one 64-bit word where the key allows: an fp32 score
  // above the id (complemented for argmax, so ties go to the smaller id), or a
  // time below 2^44 above a 20-bit id; other keys reduce as (key, id) pairs.
  // 0 and 2^64 - 1 stay free as the empty values (ids stay far below 2^20 - 1:
  // the table is LDS-resident).
  static constexpr uint64_t kCap44 = (1ull << 44) - 1;
  __device__ __forceinline__ int pack_mode() const {
    if constexpr (PT::spear && !PT::fixed) return 1;
    if constexpr (PT::recency || PT::belady) return kc.pack44 ? 2 : 0;
    return 0;
  }
  template <bool MAX>
  __device__ __forceinline__ static uint64_t pack(int mode, uint64_t key, uint32_t sid) {
    if (mode == 1) return (key << 32) | (MAX ? 0xFFFFFFFFu - sid : sid);
    uint64_t k44;
    if constexpr (PT::belady) k44 = key < kCap44 ? key : kCap44;
    else k44 = key & kCap44;  // recency: key = 2^64 - 1 - last, last below 2^44 - 1
    return (k44 << 20) | (MAX ? 0xFFFFFu - sid : sid);
  }
  template <bool MAX>
  __device__ __forceinline__ static Cand unpack(int mode, uint64_t c) {
    const bool none = MAX ? c == 0ull : c == ~0ull;
    if (mode == 1) {
      const uint32_t lo = (uint32_t)c;
      return Cand{c >> 32, none ? kNone : (MAX ? 0xFFFFFFFFu - lo : lo)};
    }
    const uint32_t lo = (uint32_t)c & 0xFFFFFu;
    const uint64_t k44 = c >> 20;
    uint64_t key;
    if constexpr (PT::belady) key = k44 == kCap44 ? ~0ull : k44;
    else key = k44 | ~kCap44;
    return Cand{key, none ? kNone : (MAX ? 0xFFFFFu - lo : lo)};
  }
  __device__ __forceinline__ bool eligible(int k, uint32_t tier) const {
    const uint32_t m = smeta[k];
    return ssid[k] != kNone && meta_phase(m) != kServing && (tier == 0 || meta_tier(m) == tier);
  }

  // Up to three reductions over the slots side by side: argmax over tier ta
  // (A), argmin over tier tb (B), argmax over tier tc (C).  Each compares its
  // candidates as a string of 32-bit words, most significant first -- the
  // packed key's two halves, or a wide key's two halves and then the id -- one
  // wavefront max / min per word.  The id enters complemented for argmax, so
  // both directions break ties towards the smaller id, and an id word never
  // equals the empty value: no candidate leaves it at 0 (argmax) or at
  // 2^32 - 1 (argmin).
  template <bool A, bool B, bool C>
  __device__ __forceinline__ void reduce3(uint32_t ta, uint32_t tb, uint32_t tc, Cand& ra, Cand& rb,
                                          Cand& rc) const {
    const int mode = pack_mode();
    bool aa[SPL], ab[SPL], ac[SPL];
    uint32_t hi[SPL], lox[SPL], lon[SPL], idx[SPL], idn[SPL];
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      aa[k] = A && eligible(k, ta);
      ab[k] = B && eligible(k, tb);
      ac[k] = C && eligible(k, tc);
      const uint64_t key = skey[k];
      const uint32_t sid = ssid[k];
      idx[k] = ~sid;
      idn[k] = sid;
      if (mode == 1) {
        hi[k] = (uint32_t)key;
        lox[k] = ~sid;
        lon[k] = sid;
      } else if (mode == 2) {
        uint64_t k44;
        if constexpr (PT::belady) k44 = key < kCap44 ? key : kCap44;
        else k44 = key & kCap44;  // recency: key = 2^64 - 1 - last, last below 2^44 - 1
        hi[k] = (uint32_t)(k44 >> 12);
        const uint32_t base = (uint32_t)k44 << 20;
        lox[k] = base | (0xFFFFFu - sid);
        lon[k] = base | sid;
      } else {
        hi[k] = (uint32_t)(key >> 32);
        lox[k] = (uint32_t)key;
        lon[k] = (uint32_t)key;
      }
    }
    uint32_t a0 = 0, a1 = 0, a2 = 0, b0 = 0, b1 = 0, b2 = 0, c0 = 0, c1 = 0, c2 = 0;
    if (A) a0 = lex_phase<true, true>(hi, aa);
    if (B) b0 = lex_phase<false, true>(hi, ab);
    if (C) c0 = lex_phase<true, true>(hi, ac);
    if (mode) {
      if (A) a1 = lex_phase<true, false>(lox, aa);
      if (B) b1 = lex_phase<false, false>(lon, ab);
      if (C) c1 = lex_phase<true, false>(lox, ac);
      if (A) ra = unpack<true>(mode, ((uint64_t)a0 << 32) | a1);
      if (B) rb = unpack<false>(mode, ((uint64_t)b0 << 32) | b1);
      if (C) rc = unpack<true>(mode, ((uint64_t)c0 << 32) | c1);
      return;
    }
    if (A) a1 = lex_phase<true, true>(lox, aa);
    if (B) b1 = lex_phase<false, true>(lon, ab);
    if (C) c1 = lex_phase<true, true>(lox, ac);
    if (A) a2 = lex_phase<true, false>(idx, aa);
    if (B) b2 = lex_phase<false, false>(idn, ab);
    if (C) c2 = lex_phase<true, false>(idx, ac);
    if (A) ra = Cand{((uint64_t)a0 << 32) | a1, a2 == 0u ? kNone : ~a2};
    if (B) rb = Cand{((uint64_t)b0 << 32) | b1, b2};
    if (C) rc = Cand{((uint64_t)c0 << 32) | c1, c2 == 0u ? kNone : ~c2};
  }

  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx&) const {
    Cand r, unused;
    if constexpr (MAX) reduce3<true, false, false>(tier, 0, 0, r, unused, unused);
    else reduce3<false, true, false>(0, tier, 0, unused, r, unused);
    return r;
  }
  __device__ __forceinline__ Cand argmax_first(const KeyCtx& K) const { return select<true>(0, K); }
  __device__ __forceinline__ void select_pd(const KeyCtx&, Cand& p, Cand& d) const {
    Cand unused;
    reduce3<false, true, true>(0, kTierHbm, kTierSram, unused, p, d);
  }
  __device__ __forceinline__ void scan3(const KeyCtx&, Cand& v, Cand& p, Cand& d) const {
    reduce3<true, true, true>(0, kTierHbm, kTierSram, v, p, d);
  }

  // Online hazard table: add the completed session, then rescore every resident.
  __device__ __forceinline__ bool hazard_open(const KeyCtx& K) const {
    return uni32(K.hn[0]) < K.online_cap;
  }
  __device__ __forceinline__ void hazard_add(const KeyCtx& K, uint32_t Tn) {
    hazard_add_counts(K, Tn, lane, 64);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int k = 0; k < SPL; ++k)
      if (ssid[k] != kNone) skey[k] = key_at(ssid[k]);
    w_sid = kNone;
  }

  // Smallest evictable resident idle for longer than ttl (timeout: key = 2^64 - 1 - last).
  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) const {
    const uint64_t thr = idle_threshold(now, ttl);
    uint32_t c = kNone;
#pragma unroll
    for (int k = 0; k < SPL; ++k) {
      const bool ok = ssid[k] != kNone && meta_phase(smeta[k]) != kServing && (~0ull - skey[k]) < thr;
      c = ok && ssid[k] < c ? ssid[k] : c;
    }
    if (__builtin_amdgcn_ballot_w64(c != kNone) == 0) return kNone;
    return uni32(reduce_min32<64, 1>(c));
  }
};

// One wavefront per simulation for tables too large for LDS.  The session
// table stays in the workspace; the residents (at most 64 * rows of them,
// bounded by N_sess, eq. (cap)) sit in LDS slots: slot s holds (key, session
// id, meta) and the KV bytes, and belongs to lane s % 64; the table records
// each resident's slot.  For each of the three reductions the engine asks
// for -- argmax over every evictable resident (the scan victim), argmin over
// the evictable HBM residents and argmax over the evictable SRAM residents
// (TIDE's candidates, eq. (promote), eq. (demote)) -- each lane keeps the
// best of its own slots, kept current as slots change.  A lane whose best
// left or got worse marks that reduction dirty, and before the next one the
// whole wavefront rebuilds it from that lane's slots; so every reduction is
// one wavefront reduction over the lanes' bests, with the decisions of a
// full scan.  The next event's session entry is loaded one event ahead, and
// every write to that entry is applied to the loaded copy too.  Lane 0
// issues every table write and every uniform read takes lane 0's value, so
// the single wavefront sees its own writes in program order.
template <uint32_t POL, uint32_t SMODE>
struct WideTable : LaneQueue {
  using PT = Pol<POL, SMODE>;
  static constexpr bool kViews = false;
  static constexpr bool kFuseGap = true;
  // The gap onset's fused scan leaves TIDE's demotion candidate to the pass,
  // which selects it only if it gets that far.
  static constexpr bool kDeferD = true;
  static constexpr bool kLaneDigest = true;
  static constexpr bool kPrefetch = true;
  template <bool N, bool T>
  using Reader = LdsWindowReader<N, T>;
  void* win;          // LDS: the event window
  __device__ __forceinline__ void* window() const { return win; }
  // the session table (workspace)
  uint64_t* mg;
  uint64_t* gq;
  uint32_t* len;
  uint64_t* last;
  uint64_t* next;
  const uint32_t* kvb;
  uint32_t* slot;     // slot of each resident session
  KeyCtx kc;
  // residents (LDS), column by lane: slot s (lane s % 64, row s / 64) at
  // index (s % 64) * rows + s / 64, so that one lane's slots are contiguous.
  // A resident keeps its slot until it leaves; a new one takes a free slot of
  // the next lane round the wavefront that has one.
  uint4* rec;         // (key low, key high, session id, meta)
  uint64_t* rsize;    // KV bytes
  uint32_t rows;      // slots per lane (capacity / 64)
  uint32_t n_res;     // residents (uniform)
  uint64_t used;      // per lane: bit j set when slot j * 64 + lane holds a resident
  uint32_t cur;       // the lane the next search for a free slot starts at (uniform)
  uint32_t top;       // rows [0, top) have held residents (uniform)
  __device__ __forceinline__ uint32_t at(uint32_t s) const { return (s & 63u) * rows + (s >> 6); }
  // per-lane bests of the lane's slots: 0 argmax (any tier), 1 argmin (HBM),
  // 2 argmax (SRAM); bsid kNone: none
  uint64_t bkey[3];
  uint32_t bsid[3], bslot[3];
  uint32_t dirty;     // bit t: best t must be rebuilt from the lane's slots
  // the latest winners of each reduction, their slots and keys (uniform)
  uint32_t cw_sid[3], cw_slot[3];
  uint64_t cw_key[3];
  // the latest session first_idle returned, and its slot
  uint32_t ci_sid, ci_slot;
  // the event's session and its slot (kNone: not resident)
  uint32_t e_sid, e_slot;
  // the entry of the latest write(): the fields its key reads (the key itself
  // is computed only if the entry is placed), KV bytes per token and length
  uint32_t w_sid, w_meta;
  float w_g;
  uint64_t w_gq, w_last, w_next;
  uint32_t w_kvb, w_len;
  // The next event's entry: loaded while the current event runs, written
  // into LDS staging (with the writes made to it meanwhile, kept in patch
  // registers; pfp: which fields) once the current event is done, and read
  // from there by its event.
  uint32_t pf_sid;
  uint64_t* stage;    // LDS: mg, gq, last, next, len | kvb << 32, slot
  uint32_t pfp;
  uint64_t pp_mg, pp_gq, pp_last, pp_next;
  uint32_t pp_meta, pp_len, pp_slot;
  enum : uint32_t { kPMg = 1, kPMeta = 2, kPGq = 4, kPLen = 8, kPLast = 16, kPNext = 32, kPSlot = 64 };

  __device__ __forceinline__ uint64_t key_from(uint32_t m, float g, uint64_t q, uint64_t l,
                                               uint64_t n) const {
    return key_of<POL, SMODE>(kc, m, hazard_of<POL, SMODE>(kc, m), g, q, l, n);
  }
  // The key of entry i from its fields in the table (uniform).
  __device__ __forceinline__ uint64_t key_at(uint32_t i) const {
    const uint64_t x = uni64(mg[i]);
    return key_from((uint32_t)x, __uint_as_float((uint32_t)(x >> 32)), PT::fixed ? uni64(gq[i]) : 0ull,
                    PT::recency ? uni64(last[i]) : 0ull, PT::nextkey ? uni64(next[i]) : ~0ull);
  }
  // Opens a path that reads the table: the compiler may not hoist those
  // loads above the branch that guards them (they would then run, and be
  // waited for, on the usual path that needs no table read).
  __device__ __forceinline__ static void cold() { asm volatile("" : : : "memory"); }
  __device__ __forceinline__ static uint64_t lane64(uint64_t v, int l) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  }
  __device__ __forceinline__ static uint64_t rkey(const uint4& r) {
    return ((uint64_t)r.y << 32) | r.x;
  }
  // Whether a resident with meta m takes part in reduction t.
  template <int t>
  __device__ __forceinline__ static bool takes(uint32_t m) {
    if (meta_phase(m) == kServing) return false;
    if constexpr (t == 0) return true;
    else if constexpr (t == 1) return meta_tier(m) == kTierHbm;
    else return meta_tier(m) == kTierSram;
  }
  template <int t>
  __device__ __forceinline__ static bool better(uint64_t ka, uint32_t sa, uint64_t kb, uint32_t sb) {
    return t == 1 ? min_better(ka, sa, kb, sb) : max_better(ka, sa, kb, sb);
  }

  // Lane s % 64 takes slot s's new resident (sid, meta m, key) into best t.
  template <int t>
  __device__ __forceinline__ void note_t(bool mine, uint32_t s, uint32_t sid, uint32_t m, uint64_t key) {
    const bool clean = (dirty & (1u << t)) == 0u;
    const bool have = bsid[t] != kNone;
    const bool was = have && bslot[t] == s;
    const bool in = takes<t>(m);
    // the slot was the best: it stays so unless it left or got worse
    const bool keep = was && in && !better<t>(bkey[t], bsid[t], key, sid);
    const bool gain = !was && in && (!have || better<t>(key, sid, bkey[t], bsid[t]));
    const bool take = mine && clean && (keep || gain);
    bkey[t] = take ? key : bkey[t];
    bsid[t] = take ? sid : bsid[t];
    bslot[t] = take ? s : bslot[t];
    dirty |= (mine && clean && was && !keep) ? (1u << t) : 0u;
  }
  __device__ __forceinline__ void note(uint32_t s, uint32_t sid, uint32_t m, uint64_t key) {
    const bool mine = lane == (s & 63u);
    note_t<0>(mine, s, sid, m, key);
    note_t<1>(mine, s, sid, m, key);
    note_t<2>(mine, s, sid, m, key);
  }
  // Lane s % 64 loses slot s: a best held there must be rebuilt.
  __device__ __forceinline__ void gone(uint32_t s) {
    const bool mine = lane == (s & 63u);
#pragma unroll
    for (int t = 0; t < 3; ++t)
      dirty |= (mine && bsid[t] != kNone && bslot[t] == s) ? (1u << t) : 0u;
  }
  // Rebuilds the dirty bests.  A few dirty lanes are rebuilt one after the
  // other by the whole wavefront (one LDS read and one wavefront reduction
  // each); many (after a hazard table change) each walk their own slots.
  __device__ __forceinline__ void rescan() {
    const uint64_t dl = __builtin_amdgcn_ballot_w64(dirty != 0u);
    if (dl == 0ull) return;
    if (__builtin_popcountll(dl) <= 4) {
      for (uint64_t bits = dl; bits; bits &= bits - 1u) {
        const uint32_t l = (uint32_t)__builtin_ctzll(bits);
        const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)dirty, (int)l);
        const uint32_t s = l + 64u * lane;
        const uint64_t ul = lane64(used, (int)l);
        const bool valid = lane < top && ((ul >> lane) & 1ull);   // then lane < rows
        const uint4 rr = rec[l * rows + (valid ? lane : 0u)];
        const uint4 r = valid ? rr : make_uint4(0u, 0u, kNone, 0u);
        if (d & 1u) rebuild<0>(l, r, s, valid);
        if (d & 2u) rebuild<1>(l, r, s, valid);
        if (d & 4u) rebuild<2>(l, r, s, valid);
      }
      dirty = 0u;
      return;
    }
    const uint32_t d = dirty;
    const bool any0 = __builtin_amdgcn_ballot_w64((d & 1u) != 0u) != 0ull;
    const bool any1 = __builtin_amdgcn_ballot_w64((d & 2u) != 0u) != 0ull;
    const bool any2 = __builtin_amdgcn_ballot_w64((d & 4u) != 0u) != 0ull;
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      const bool r = (d >> t) & 1u;
      bsid[t] = r ? kNone : bsid[t];
      bkey[t] = r ? (t == 1 ? ~0ull : 0ull) : bkey[t];
    }
    for (uint32_t j0 = 0; j0 < top; j0 += 4u) {
      uint4 r[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t j = j0 + (uint32_t)k;
        r[k] = make_uint4(0u, 0u, kNone, 0u);
        if (d != 0u && j < top && ((used >> j) & 1ull)) r[k] = rec[lane * rows + j];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t sk = (j0 + (uint32_t)k) * 64u + lane;
        if (any0) rescan_one<0>(d, sk, r[k]);
        if (any1) rescan_one<1>(d, sk, r[k]);
        if (any2) rescan_one<2>(d, sk, r[k]);
      }
    }
    dirty = 0u;
  }
  template <int t>
  __device__ __forceinline__ void rescan_one(uint32_t d, uint32_t s, const uint4& r) {
    const uint64_t key = rkey(r);
    const bool take = ((d >> t) & 1u) && r.z != kNone && takes<t>(r.w) &&
                      (bsid[t] == kNone || better<t>(key, r.z, bkey[t], bsid[t]));
    bkey[t] = take ? key : bkey[t];
    bsid[t] = take ? r.z : bsid[t];
    bslot[t] = take ? s : bslot[t];
  }

  // The best of one candidate per lane (act: the lane has one) by reduction
  // t's order: its key, id and position.  The candidates compare as strings
  // of 32-bit words, as the slot table's do: an fp32 score and the id; a
  // time below 2^44 packed above a 20-bit id; else the key's two halves and
  // the id (complemented for argmax, so ties go to the smaller id).  Every
  // phase keeps only the lanes still equal, so the one lane left holds the
  // winner.
  template <int t>
  __device__ __forceinline__ Cand wave_pick(bool in, uint64_t key, uint32_t sid, uint32_t pos,
                                            uint32_t& pos_out) const {
    constexpr bool MAX = t != 1;
    pos_out = kNone;
    if (__builtin_amdgcn_ballot_w64(in) == 0ull) return MAX ? cand_none_max() : cand_none_min();
    bool act[1] = {in};
    uint32_t w0[1], w1[1], w2[1];
    if (PT::spear && !PT::fixed) {
      w0[0] = (uint32_t)key;
      w1[0] = MAX ? ~sid : sid;
      lex_phase<MAX, true>(w0, act);
      lex_phase<MAX, true>(w1, act);
    } else if ((PT::recency || PT::belady) && kc.pack44) {
      constexpr uint64_t kCap44 = (1ull << 44) - 1;
      uint64_t k44;
      if constexpr (PT::belady) k44 = key < kCap44 ? key : kCap44;
      else k44 = key & kCap44;  // recency: key = 2^64 - 1 - last, last below 2^44 - 1
      w0[0] = (uint32_t)(k44 >> 12);
      w1[0] = ((uint32_t)k44 << 20) | (MAX ? 0xFFFFFu - sid : sid);
      lex_phase<MAX, true>(w0, act);
      lex_phase<MAX, true>(w1, act);
    } else {
      w0[0] = (uint32_t)(key >> 32);
      w1[0] = (uint32_t)key;
      w2[0] = MAX ? ~sid : sid;
      lex_phase<MAX, true>(w0, act);
      lex_phase<MAX, true>(w1, act);
      lex_phase<MAX, true>(w2, act);
    }
    const uint64_t b = __builtin_amdgcn_ballot_w64(act[0]);
    Cand c = MAX ? cand_none_max() : cand_none_min();
    if (b != 0ull) {
      const int l = __builtin_ctzll(b);
      c.key = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(key >> 32), l) << 32) |
              (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)key, l);
      c.sid = (uint32_t)__builtin_amdgcn_readlane((int)sid, l);
      pos_out = (uint32_t)__builtin_amdgcn_readlane((int)pos, l);
    }
    return c;
  }
  // Reduction t over the lanes' bests: the winner, and its slot recorded.
  template <int t>
  __device__ __forceinline__ Cand reduce_t() {
    uint32_t s;
    const Cand c = wave_pick<t>(bsid[t] != kNone, bkey[t], bsid[t], bslot[t], s);
    cw_sid[t] = c.sid;
    cw_slot[t] = s;
    cw_key[t] = c.key;
    return c;
  }
  // Rebuilds lane l's best t from its slots, the whole wavefront at once:
  // lane k reads slot l + 64 k (lane l's slots sit side by side in LDS).
  template <int t>
  __device__ __forceinline__ void rebuild(uint32_t l, const uint4& r, uint32_t s, bool valid) {
    uint32_t pos;
    const bool in = valid && takes<t>(r.w);
    const Cand c = wave_pick<t>(in, rkey(r), r.z, s, pos);
    const bool mine = lane == l;
    bkey[t] = mine ? c.key : bkey[t];
    bsid[t] = mine ? c.sid : bsid[t];
    bslot[t] = mine ? pos : bslot[t];
  }
  // The slot of resident sid, kNone if sid is not resident.
  __device__ __forceinline__ uint32_t find(uint32_t sid) const {
    // Matching winners hold the same slot, so their slots combine by OR.  (A
    // select between two members would let the compiler load from a selected
    // member address, which keeps the whole table object in scratch memory.)
    const bool h0 = sid == cw_sid[0], h1 = sid == cw_sid[1], h2 = sid == cw_sid[2];
    const uint32_t c = (h0 ? cw_slot[0] : 0u) | (h1 ? cw_slot[1] : 0u) | (h2 ? cw_slot[2] : 0u);
    if (sid == e_sid) return e_slot;
    if (h0 || h1 || h2) return c;
    if (sid == ci_sid) return ci_slot;
    uint32_t s;
    if (sid == pf_sid && (pfp & kPSlot)) {
      s = pp_slot;
    } else {
      cold();
      s = uni32(slot[sid]);
    }
    // the table's slot field is current only while the session is resident
    if (s < 64u * rows && ((lane64(used, (int)(s & 63u)) >> (s >> 6)) & 1ull) &&
        uni32(rec[at(s)].z) == sid)
      return s;
    return kNone;
  }
  // Records that sid now sits in slot s (kNone: it left).
  __device__ __forceinline__ void moved_to(uint32_t sid, uint32_t s) {
    if (s != kNone && lane == 0) slot[sid] = s;
    if (sid == pf_sid && s != kNone) {
      pfp |= kPSlot;
      pp_slot = s;
    }
    if (sid == e_sid) e_slot = s;
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      cw_slot[t] = sid == cw_sid[t] ? s : cw_slot[t];
      cw_sid[t] = (sid == cw_sid[t] && s == kNone) ? kNone : cw_sid[t];
    }
    if (sid == ci_sid) ci_sid = kNone;
  }
  __device__ __forceinline__ void put(uint32_t s, uint32_t sid, uint32_t m, uint64_t key) {
    if (lane == 0) rec[at(s)] = make_uint4((uint32_t)key, (uint32_t)(key >> 32), sid, m);
    note(s, sid, m, key);
  }
  // A new resident takes the first free slot of the first lane from cur on
  // that has one (there is one: residents never exceed the slots).
  __device__ __forceinline__ void insert(uint32_t sid, uint32_t m, uint64_t key, uint64_t size) {
    const uint64_t rowmask = rows >= 64u ? ~0ull : ((1ull << rows) - 1ull);
    const uint64_t fm = __builtin_amdgcn_ballot_w64((~used & rowmask) != 0ull);
    const uint64_t rot = cur ? ((fm >> cur) | (fm << (64u - cur))) : fm;
    const uint32_t l = (cur + (uint32_t)__builtin_ctzll(rot)) & 63u;
    const uint32_t j = (uint32_t)__builtin_ctzll(~lane64(used, (int)l) & rowmask);
    const uint32_t s = j * 64u + l;
    used |= lane == l ? (1ull << j) : 0ull;
    cur = (l + 1u) & 63u;
    top = j + 1u > top ? j + 1u : top;
    ++n_res;
    if (lane == 0) rsize[at(s)] = size;
    put(s, sid, m, key);
    moved_to(sid, s);
  }
  // Resident sid leaves slot s.
  __device__ __forceinline__ void remove(uint32_t sid, uint32_t s) {
    gone(s);
    moved_to(sid, kNone);
    used &= lane == (s & 63u) ? ~(1ull << (s >> 6)) : ~0ull;
    --n_res;
  }
  // Meta word m of entry sid: the table, and the resident set it implies.
  __device__ __forceinline__ void meta_to(uint32_t sid, uint32_t m) {
    const uint32_t s = find(sid);
    if (lane == 0) reinterpret_cast<uint32_t*>(mg + sid)[0] = m;
    if (sid == pf_sid) patch_meta(m);
    const bool now = meta_tier(m) != kTierNone;
    if (s != kNone && !now) {
      remove(sid, s);
    } else if (s != kNone) {
      // a tier or flag change: the key stays (a reduction winner's is at hand)
      const bool h0 = sid == cw_sid[0], h1 = sid == cw_sid[1], h2 = sid == cw_sid[2];
      uint64_t key = (h0 ? cw_key[0] : 0ull) | (h1 ? cw_key[1] : 0ull) | (h2 ? cw_key[2] : 0ull);
      if (!(h0 || h1 || h2)) {
        const uint4 r = rec[at(s)];
        key = uni64(((uint64_t)r.y << 32) | r.x);
      }
      put(s, sid, m, key);
    } else if (now) {
      uint64_t key, size;
      if (sid == w_sid) {
        key = key_from(w_meta, w_g, w_gq, w_last, w_next);
        size = (uint64_t)w_len * w_kvb;
      } else {
        cold();
        key = key_at(sid);
        size = (uint64_t)uni32(len[sid]) * uni32(kvb[sid]);
      }
      insert(sid, m, key, size);
    }
  }

  __device__ __forceinline__ void event_begin() {}
  __device__ __forceinline__ void grow(uint32_t) {}
  __device__ __forceinline__ void patch_meta(uint32_t m) {
    if (pfp & kPMg) {
      pp_mg = (pp_mg & 0xFFFFFFFF00000000ull) | m;
    } else {
      pfp |= kPMeta;
      pp_meta = m;
    }
  }
  // The next event's entry as loaded from the table.
  struct Pf {
    uint64_t mg, gq, last, next;
    uint32_t len, kvb, slot;
  };
  __device__ __forceinline__ Pf prefetch_issue(uint32_t sid) {
    pf_sid = sid;
    pfp = 0u;
    Pf v;
    v.mg = mg[sid];
    v.gq = PT::fixed ? gq[sid] : 0ull;
    v.len = len[sid];
    v.last = last[sid];
    v.next = PT::nextkey ? next[sid] : ~0ull;
    v.kvb = kvb[sid];
    v.slot = slot[sid];
    return v;
  }
  // After the current event: the entry as loaded into the staging area.
  __device__ __forceinline__ void prefetch_land(const Pf& v) {
    if (lane == 0) {
      stage[0] = v.mg;
      stage[1] = v.gq;
      stage[2] = v.last;
      stage[3] = v.next;
      stage[4] = (uint64_t)v.len | ((uint64_t)v.kvb << 32);
      stage[5] = v.slot;
    }
  }
  // The event's session entry: when it was loaded ahead, the staged copy with
  // every write made to the entry since its load.
  __device__ __forceinline__ Entry read(uint32_t sid) {
    uint64_t x, q, la, nx, lk;
    uint32_t s;
    if (uc<true>(sid == pf_sid)) {
      x = uni64(stage[0]);
      q = uni64(stage[1]);
      la = uni64(stage[2]);
      nx = uni64(stage[3]);
      lk = uni64(stage[4]);
      s = uni32((uint32_t)stage[5]);
      if (pfp & kPMg) x = pp_mg;
      if (pfp & kPMeta) x = (x & 0xFFFFFFFF00000000ull) | pp_meta;
      if (pfp & kPGq) q = pp_gq;
      if (pfp & kPLast) la = pp_last;
      if (pfp & kPNext) nx = pp_next;
      if (pfp & kPLen) lk = (lk & 0xFFFFFFFF00000000ull) | pp_len;
      if (pfp & kPSlot) s = pp_slot;
    } else {
      // made uniform inside the branch, so that only this path waits for the loads
      cold();
      x = uni64(mg[sid]);
      q = PT::fixed ? uni64(gq[sid]) : 0ull;
      la = uni64(last[sid]);
      nx = PT::nextkey ? uni64(next[sid]) : ~0ull;
      lk = uni64((uint64_t)len[sid] | ((uint64_t)kvb[sid] << 32));
      s = uni32(slot[sid]);
    }
    pf_sid = kNone;
    Entry e;
    e.meta = (uint32_t)x;
    e.g = __uint_as_float((uint32_t)(x >> 32));
    e.gq = q;
    e.len = (uint32_t)lk;
    e.kvb = (uint32_t)(lk >> 32);
    e.last = la;
    e.next = nx;
    e_sid = sid;
    e_slot = meta_tier(e.meta) != kTierNone ? s : kNone;
    return e;
  }
  __device__ __forceinline__ void read_size(uint32_t sid, uint64_t& size, uint32_t& m) const {
    const uint32_t s = find(sid);
    if (s != kNone) {
      size = uni64(rsize[at(s)]);
      m = uni32(rec[at(s)].w);
    } else {
      cold();
      m = uni32((uint32_t)mg[sid]);
      size = (uint64_t)uni32(len[sid]) * uni32(kvb[sid]);
    }
  }
  __device__ __forceinline__ void read_end(uint32_t sid, Entry& e) {
    const Entry f = read(sid);
    e.meta = f.meta;
    e.g = f.g;
    e.gq = f.gq;
  }
  __device__ __forceinline__ void write_end(uint32_t sid, const Entry& e, uint64_t t, uint64_t nx) {
    if (lane == 0) {
      reinterpret_cast<uint32_t*>(mg + sid)[0] = e.meta;
      last[sid] = t;
      if constexpr (PT::nextkey) next[sid] = nx;
    }
    if (sid == pf_sid) {
      patch_meta(e.meta);
      pfp |= kPLast | (PT::nextkey ? kPNext : 0u);
      pp_last = t;
      pp_next = nx;
    }
    w_sid = kNone;
    const uint32_t s = find(sid);
    if (s != kNone) put(s, sid, e.meta, key_from(e.meta, e.g, e.gq, t, nx));
  }
  __device__ __forceinline__ void write(uint32_t sid, const Entry& e) {
    const uint64_t x = (uint64_t)e.meta | ((uint64_t)__float_as_uint(e.g) << 32);
    if (lane == 0) {
      mg[sid] = x;
      if constexpr (PT::fixed) gq[sid] = e.gq;
      len[sid] = e.len;
      last[sid] = e.last;
      if constexpr (PT::nextkey) next[sid] = e.next;
    }
    if (sid == pf_sid) {
      pfp = (pfp & kPSlot) | kPMg | kPGq | kPLen | kPLast | kPNext;
      pp_mg = x;
      pp_gq = e.gq;
      pp_len = e.len;
      pp_last = e.last;
      pp_next = e.next;
    }
    w_sid = sid;
    w_meta = e.meta;
    w_g = e.g;
    w_gq = e.gq;
    w_last = e.last;
    w_next = e.next;
    w_kvb = e.kvb;
    w_len = e.len;
    const uint32_t s = find(sid);
    if (s != kNone) put(s, sid, e.meta, key_from(e.meta, e.g, e.gq, e.last, e.next));
  }
  __device__ __forceinline__ void set_meta(uint32_t sid, uint32_t m) { meta_to(sid, m); }
  __device__ __forceinline__ void set_len_meta(uint32_t sid, uint32_t l, uint32_t m) {
    if (lane == 0) len[sid] = l;
    if (sid == pf_sid) {
      pfp |= kPLen;
      pp_len = l;
    }
    if (sid == w_sid) w_len = l;
    meta_to(sid, m);
  }
  __device__ __forceinline__ void set_turn(uint32_t, uint32_t, const KeyCtx&) {}
  __device__ __forceinline__ void scan(const KeyCtx&, uint32_t) {}

  template <bool MAX>
  __device__ __forceinline__ Cand select(uint32_t tier, const KeyCtx&) {
    rescan();
    if constexpr (MAX) {
      if (tier == kTierSram) return reduce_t<2>();
      return reduce_t<0>();
    } else {
      return reduce_t<1>();
    }
  }
  __device__ __forceinline__ Cand argmax_first(const KeyCtx& K) { return select<true>(0, K); }
  __device__ __forceinline__ void select_pd(const KeyCtx&, Cand& p, Cand& d) {
    rescan();
    p = reduce_t<1>();
    d = reduce_t<2>();
  }
  __device__ __forceinline__ void scan3(const KeyCtx&, Cand& v, Cand& p, Cand& d) {
    rescan();
    v = reduce_t<0>();
    p = reduce_t<1>();
    d = Cand{0ull, kNone};  // deferred: select_d
  }
  __device__ __forceinline__ Cand select_p(const KeyCtx&) {
    rescan();
    return reduce_t<1>();
  }
  __device__ __forceinline__ Cand select_d(const KeyCtx&) {
    rescan();
    return reduce_t<2>();
  }

  // Online hazard table: add the completed session, then rescore every resident.
  __device__ __forceinline__ bool hazard_open(const KeyCtx& K) const {
    return uni32(K.hn[0]) < K.online_cap;
  }
  __device__ __forceinline__ void hazard_add(const KeyCtx& K, uint32_t Tn) {
    hazard_add_counts(K, Tn, lane, 64);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // every lane rescores its own residents (their fields from the table)
    for (uint32_t j = 0; j < top; ++j) {
      if ((used >> j) & 1ull) {
        const uint32_t o = lane * rows + j;
        const uint4 r = rec[o];
        const uint64_t x = mg[r.z];
        const uint64_t key =
            key_from((uint32_t)x, __uint_as_float((uint32_t)(x >> 32)), PT::fixed ? gq[r.z] : 0ull,
                     PT::recency ? last[r.z] : 0ull, PT::nextkey ? next[r.z] : ~0ull);
        rec[o] = make_uint4((uint32_t)key, (uint32_t)(key >> 32), r.z, r.w);
      }
    }
    dirty = 7u;
    w_sid = kNone;
#pragma unroll
    for (int t = 0; t < 3; ++t) cw_sid[t] = kNone;   // their keys changed
  }

  // Smallest evictable resident idle for longer than ttl (timeout: key = 2^64 - 1 - last).
  __device__ __forceinline__ uint32_t first_idle(uint64_t now, uint64_t ttl) {
    const uint64_t thr = idle_threshold(now, ttl);
    rescan();
    // the oldest evictable resident decides whether any timer fired
    const Cand o = reduce_t<0>();
    if (o.sid == kNone || ~0ull - o.key >= thr) return kNone;
    uint32_t c = kNone, cs = kNone;
    for (uint32_t j = 0; j < top; ++j) {
      if ((used >> j) & 1ull) {
        const uint4 r = rec[lane * rows + j];
        const bool ok = meta_phase(r.w) != kServing && (~0ull - rkey(r)) < thr;
        cs = ok && r.z < c ? j * 64u + lane : cs;
        c = ok && r.z < c ? r.z : c;
      }
    }
    const uint32_t m = uni32(reduce_min32<64, 1>(c));
    if (m != kNone) {
      const uint64_t b = __builtin_amdgcn_ballot_w64(c == m);
      ci_sid = m;
      ci_slot = (uint32_t)__builtin_amdgcn_readlane((int)cs, __builtin_ctzll(b));
    }
    return m;
  }
};

// ------------------------------------------------------------- the engine

struct Scalars {
  uint64_t used_s, used_h, dma_free_at, prev_t, log_len;
  uint32_t n_res, n_table, hi;
  uint64_t hit_s_bytes, hit_h_bytes, miss_tok, prev_s_bytes, prev_h_bytes;
};

// Counters as kept during a run: event-bounded counts in 32 bits.
struct Cnt {
  uint32_t requests, hit_sram, hit_hbm, miss, bypass, evict, expire, promote, swap, tide_passes,
      events, prefetch_hits, vict_diff, prom_diff;
  uint64_t dma_bytes, tokens_total, tokens_computed, extra_prefill, score_evals, resident_evals,
      digest, victim_digest, error;
  double amat, ttft;
};

__device__ __forceinline__ Cnt cnt_from(const unison_counters& c) {
  Cnt k;
  k.requests = (uint32_t)c.requests;
  k.hit_sram = (uint32_t)c.hit_sram;
  k.hit_hbm = (uint32_t)c.hit_hbm;
  k.miss = (uint32_t)c.miss;
  k.bypass = (uint32_t)c.bypass;
  k.evict = (uint32_t)c.evict;
  k.expire = (uint32_t)c.expire;
  k.promote = (uint32_t)c.promote;
  k.swap = (uint32_t)c.swap;
  k.tide_passes = (uint32_t)c.tide_passes;
  k.events = (uint32_t)c.events;
  k.prefetch_hits = (uint32_t)c.prefetch_hits;
  k.vict_diff = (uint32_t)c.vict_diff;
  k.prom_diff = (uint32_t)c.prom_diff;
  k.dma_bytes = c.dma_bytes;
  k.tokens_total = c.tokens_total;
  k.tokens_computed = c.tokens_computed;
  k.extra_prefill = c.extra_prefill_tok;
  k.score_evals = c.score_evals;
  k.resident_evals = c.resident_evals;
  k.digest = c.digest;
  k.victim_digest = c.victim_digest;
  k.error = c.error;
  k.amat = c.amat_sum_ns;
  k.ttft = c.ttft_sum_ns;
  return k;
}

__device__ __forceinline__ unison_counters cnt_to(const Cnt& k) {
  unison_counters c;
  c.requests = k.requests;
  c.hit_sram = k.hit_sram;
  c.hit_hbm = k.hit_hbm;
  c.miss = k.miss;
  c.bypass = k.bypass;
  c.evict = k.evict;
  c.expire = k.expire;
  c.promote = k.promote;
  c.swap = k.swap;
  c.dma_bytes = k.dma_bytes;
  c.tide_passes = k.tide_passes;
  c.tokens_total = k.tokens_total;
  c.tokens_computed = k.tokens_computed;
  c.extra_prefill_tok = k.extra_prefill;
  c.score_evals = k.score_evals;
  c.resident_evals = k.resident_evals;
  c.digest = k.digest;
  c.victim_digest = k.victim_digest;
  c.events = k.events;
  c.error = k.error;
  c.prefetch_hits = k.prefetch_hits;
  c.vict_diff = k.vict_diff;
  c.prom_diff = k.prom_diff;
  c.amat_sum_ns = k.amat;
  c.ttft_sum_ns = k.ttft;
  return c;
}

__device__ __forceinline__ void pin_vgpr(Scalars& S) {
  S.used_s = in_vgpr(S.used_s);
  S.used_h = in_vgpr(S.used_h);
  S.dma_free_at = in_vgpr(S.dma_free_at);
  S.prev_t = in_vgpr(S.prev_t);
  S.log_len = in_vgpr(S.log_len);
  S.n_res = in_vgpr(S.n_res);
  S.n_table = in_vgpr(S.n_table);
  S.hi = in_vgpr(S.hi);
  S.hit_s_bytes = in_vgpr(S.hit_s_bytes);
  S.hit_h_bytes = in_vgpr(S.hit_h_bytes);
  S.miss_tok = in_vgpr(S.miss_tok);
  S.prev_s_bytes = in_vgpr(S.prev_s_bytes);
  S.prev_h_bytes = in_vgpr(S.prev_h_bytes);
}

__device__ __forceinline__ void pin_vgpr(unison_sim_params& p) {
  p.tide = in_vgpr(p.tide);
  p.cap_sram_B = in_vgpr(p.cap_sram_B);
  p.cap_hbm_B = in_vgpr(p.cap_hbm_B);
  p.n_slots = in_vgpr(p.n_slots);
  p.dma_B_per_us = in_vgpr(p.dma_B_per_us);
  p.ttl_ns = in_vgpr(p.ttl_ns);
  p.b_g = in_vgpr(p.b_g);
  p.tau_ns = in_vgpr(p.tau_ns);
}

__device__ __forceinline__ void pin_vgpr(Cnt& k) {
  k.requests = in_vgpr(k.requests);
  k.hit_sram = in_vgpr(k.hit_sram);
  k.hit_hbm = in_vgpr(k.hit_hbm);
  k.miss = in_vgpr(k.miss);
  k.bypass = in_vgpr(k.bypass);
  k.evict = in_vgpr(k.evict);
  k.expire = in_vgpr(k.expire);
  k.promote = in_vgpr(k.promote);
  k.swap = in_vgpr(k.swap);
  k.tide_passes = in_vgpr(k.tide_passes);
  k.events = in_vgpr(k.events);
  k.prefetch_hits = in_vgpr(k.prefetch_hits);
  k.vict_diff = in_vgpr(k.vict_diff);
  k.prom_diff = in_vgpr(k.prom_diff);
  k.dma_bytes = in_vgpr(k.dma_bytes);
  k.tokens_total = in_vgpr(k.tokens_total);
  k.tokens_computed = in_vgpr(k.tokens_computed);
  k.extra_prefill = in_vgpr(k.extra_prefill);
  k.score_evals = in_vgpr(k.score_evals);
  k.resident_evals = in_vgpr(k.resident_evals);
  k.digest = in_vgpr(k.digest);
  k.victim_digest = in_vgpr(k.victim_digest);
  k.error = in_vgpr(k.error);
  k.amat = in_vgpr(k.amat);
  k.ttft = in_vgpr(k.ttft);
}

struct LogSink {
  bool on;             // logging requested (a launch-wide, uniform flag)
  unison_record* rec;  // this simulation's records
  uint32_t cap;
  bool lead;           // the one lane that stores records
  bool victims;        // also record each event's scan result
};

template <class Tab>
__device__ __forceinline__ void emit(Tab& T, Cnt& C, Scalars& S, const LogSink& L, uint32_t ev,
                                     uint32_t op, uint32_t a, uint32_t b) {
  if constexpr (Tab::kLaneDigest) T.queue_record(ev, op, a, b);
  else C.digest += rec_hash(ev, op, a, b);
  if (L.on) {
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

// Events [e_io, end) of one simulation; e_io ends at end.
template <uint32_t POL, uint32_t SMODE, bool UNI, class Tab>
__device__ __forceinline__ void run_range(Tab& T, const unison_sim_params& P, const KeyCtx& K, const TraceView& tr,
                                          Scalars& S, Cnt& C, const LogSink& L, uint64_t& e_io, uint64_t end) {
  using PT = Pol<POL, SMODE>;
  uint64_t e = e_io;
  typename Tab::template Reader<PT::belady, PT::eta> rd(tr, e, end, T.window());
  // victim-digest weight of event e, (2e + 1) * 0x9e3779b97f4a7c15, stepped per event
  constexpr uint64_t kGolden = 0x9e3779b97f4a7c15ull;
  uint64_t vw = (2ull * e + 1ull) * kGolden;
  for (; e < end; ++e) {
    const Ev cur = rd.take(e);
    T.event_begin();
    const uint64_t now = UNI ? uni64(cur.t) : cur.t;
    const uint32_t sid = UNI ? uni32(cur.sid) : cur.sid;
    const uint32_t info = UNI ? uni32(cur.info) : cur.info;
    const uint32_t kind = info >> 24, turn = info & 0xFFFFFFu;
    const uint32_t cur_len = UNI ? uni32(cur.len) : cur.len;
    uint64_t cur_next = (UNI && PT::belady) ? uni64(cur.next) : cur.next;
    if constexpr (PT::eta) {
      // the predicted return: gap onset + the expected wait of the gap's tool class
      const uint32_t tool = UNI ? uni32(cur.tool) : cur.tool;
      if (kind == kGapStart) cur_next = sat_add(now, K.eta[tool < kEtaClasses ? tool : 0u]);
    }
    const uint32_t ev = (uint32_t)e;

    // timeout policy: TTL timers that fired since the previous event
    if constexpr (PT::timeout) {
      for (;;) {
        const uint32_t v = T.first_idle(now, P.ttl_ns);
        if (v == kNone) break;
        emit(T, C, S, L, ev, kOpExpire, v, kNone);
        C.expire++;
        release(T, S, v);
      }
    }

    // Alg. 1: write e into R; on gap_end update the EMA
    Entry x;
    uint32_t tier0, len_prev = 0;
    bool prefetched = false;
    if (kind == kArrive) {
      x = T.read(sid);
      tier0 = meta_tier(x.meta);
      prefetched = (x.meta & kPrefetched) != 0;
      len_prev = x.len;
      if (turn == 0) {
        x.g = 0.0f;
        x.gq = 0;
        x.len = 0;
        len_prev = 0;
      } else {
        const uint64_t gap = now - x.last;  // eq. (gap)
        // only SPEAR keys and TIDE budgets read the gap EMA
        if (PT::spear || PT::belady || uc<UNI>(P.tide != 0)) x.g = ema_f32(x.g, gap);
        if constexpr (PT::fixed) x.gq = ema_int(x.gq, gap, P.b_g, P.tau_ns);
      }
      x.meta = make_meta(kServing, tier0, turn);
      x.last = now;
      if (turn == 0) {
        S.n_table++;
        if (sid + 1 > S.hi) S.hi = sid + 1;
        T.grow(S.hi);
      }
      T.write(sid, x);
      T.set_turn(sid, x.meta, K);
    } else {
      T.read_end(sid, x);
      tier0 = meta_tier(x.meta);
      x.meta = make_meta(kind == kGapStart ? kGap : kDoneP, tier0, meta_turn(x.meta));
      T.write_end(sid, x, now, kind == kGapStart ? cur_next : ~0ull);
      // an online hazard table counts the completed session before the scan
      if (kind == kDone && K.online_cap && T.hazard_open(K)) T.hazard_add(K, meta_turn(x.meta) + 1u);
    }

    // a table that loads entries ahead: the next event's session
    // (also after the last event, where the window holds the last event's
    // session again: a load that nothing reads, but no branch to join)
    typename Tab::Pf pf{};
    if constexpr (Tab::kPrefetch) pf = T.prefetch_issue(rd.peek_sid(e + 1));

    // the register-file scan: every table entry is scored; its argmax over
    // evictable residents is this event's victim index
    C.score_evals += S.n_table;
    C.resident_evals += S.n_res;
    T.scan(K, sid);
    bool dual = false;
    if constexpr (Tab::kViews) {
      dual = P.dual_sync != 0;
      T.set_src(dual ? 0 : -1);  // the eviction engine scans its own copy
    }
    // At a gap onset of a TIDE simulation the same pass can also yield TIDE's
    // first candidates: nothing changes the table before the TIDE pass.
    Cand v0, p0, d0;
    bool have_pd = false;
    if constexpr (Tab::kFuseGap) {
      // TIDE's candidates are wanted only when the pass will run (the DMA
      // engine is idle at this gap onset)
      if (kind == kGapStart && uc<UNI>(P.tide && now >= S.dma_free_at)) {
        T.scan3(K, v0, p0, d0);
        have_pd = true;
      } else {
        v0 = T.argmax_first(K);
      }
    } else {
      v0 = T.argmax_first(K);
    }
    // odd weight per event: a different victim at any one event changes the sum
    if constexpr (Tab::kLaneDigest) {
      T.queue_victim(e, v0.sid);
    } else {
      C.victim_digest += ((uint64_t)v0.sid + 1u) * vw;
      vw += 2ull * kGolden;
    }
    if (L.victims) {
      if (L.lead && S.log_len < L.cap) L.rec[S.log_len] = unison_record{ev, kOpVictim, v0.sid, kNone};
      S.log_len++;
    }

    if (kind == kArrive) {
      // eq. (hr-amat), eq. (prered), eq. (reuse)
      const uint64_t ln = cur_len;
      const uint64_t dlen = ln - len_prev;
      const uint64_t kb = x.kvb;
      C.requests++;
      C.tokens_total += ln;
      if (tier0 != kTierNone) {
        const uint64_t now_b = ln * kb;
        const uint64_t old = (uint64_t)len_prev * kb;
        if (tier0 == kTierSram) {
          C.hit_sram++;
          C.prefetch_hits += prefetched ? 1u : 0u;
          S.hit_s_bytes += now_b;
          S.prev_s_bytes += old;
          S.used_s -= old;
        } else {
          C.hit_hbm++;
          S.hit_h_bytes += now_b;
          S.prev_h_bytes += old;
          S.used_h -= old;
        }
        C.tokens_computed += dlen;
        S.n_res--;
      } else {
        C.miss++;
        S.miss_tok += ln;
        C.tokens_computed += ln;
        C.extra_prefill += len_prev;
      }
      x.len = (uint32_t)ln;
      x.meta = with_tier(x.meta, kTierNone);
      T.set_len_meta(sid, x.len, x.meta);

      // Alg. 1 capacity branch: evict the argmax victim until the session fits
      const uint64_t size = ln * kb;
      const uint32_t pref = tier0 == kTierHbm ? kTierHbm : kTierSram;
      const uint32_t other = pref == kTierSram ? kTierHbm : kTierSram;
      if (uc<UNI>(size > P.cap_sram_B && size > P.cap_hbm_B)) {
        emit(T, C, S, L, ev, kOpBypass, sid, kNone);
        C.bypass++;
      } else {
        bool first = true;
        for (;;) {
          const bool slot = (uint64_t)S.n_res + 1 <= P.n_slots;
          const bool fit_s = slot && S.used_s + size <= P.cap_sram_B;
          const bool fit_h = slot && S.used_h + size <= P.cap_hbm_B;
          const bool fit_p = pref == kTierSram ? fit_s : fit_h;
          const bool fit_o = pref == kTierSram ? fit_h : fit_s;
          if (uc<UNI>(fit_p || fit_o)) {
            const uint32_t t = fit_p ? pref : other;
            if (t == kTierSram) S.used_s += size; else S.used_h += size;
            S.n_res++;
            T.set_meta(sid, with_tier(x.meta, t));
            emit(T, C, S, L, ev, kOpPlace, sid, t);
            break;
          }
          // the event's own scan result is the first victim: the arriving
          // session was never evictable, so releasing it changed nothing
          Cand v;
          if (first) {
            v.key = v0.key;
            v.sid = v0.sid;
          } else {
            v = T.template select<true>(0, K);
          }
          first = false;
          if constexpr (Tab::kViews) {
            if (dual && v.sid != kNone) {  // eq. (stale): would the live table agree?
              T.set_src(-1);
              const Cand vl = T.template select<true>(0, K);
              T.set_src(0);
              C.vict_diff += vl.sid != v.sid ? 1u : 0u;
            }
          }
          if (v.sid == kNone) {
            emit(T, C, S, L, ev, kOpBypass, sid, kNone);
            C.bypass++;
            break;
          }
          emit(T, C, S, L, ev, kOpEvict, v.sid, kNone);
          C.evict++;
          release(T, S, v.sid);
        }
      }
    } else if (kind == kGapStart) {
      if (uc<UNI>(P.tide && now >= S.dma_free_at)) {
        // eq. (budget) / eq. (budgetq): Delta is the session's gap EMA in us
        uint64_t delta_us;
        if constexpr (PT::fixed) {
          if (x.gq < (1ull << 32) && P.tau_ns < (1ull << 32)) {
            delta_us = (x.gq * P.tau_ns) / 1000u;
          } else {
            const unsigned __int128 d = ((unsigned __int128)x.gq * P.tau_ns) / 1000u;
            delta_us = d > (unsigned __int128)~0ull ? ~0ull : (uint64_t)d;
          }
        } else {
          delta_us = (uint64_t)x.g;
        }
        const uint64_t budget = sat_mul(delta_us, P.dma_B_per_us);
        uint64_t left = budget, moved = 0;
        C.tide_passes++;
        if constexpr (Tab::kViews) T.set_src(dual ? 1 : -1);  // TIDE decides from its own copy
        for (;;) {
            // eq. (promote), eq. (demote); a table that defers d reduces it
          // only when the pass gets past the promotion test
          Cand p, d;
          bool d_later = false;
          if (have_pd) {
            p = p0;
            d = d0;
            d_later = Tab::kDeferD;
            have_pd = false;
          } else if constexpr (Tab::kDeferD) {
            p = T.select_p(K);
            d_later = true;
          } else {
            T.select_pd(K, p, d);
          }
          if (p.sid == kNone) break;
          uint32_t live_p = p.sid;
          if constexpr (Tab::kViews) {
            if (dual) {
              T.set_src(-1);
              live_p = T.template select<false>(kTierHbm, K).sid;
              T.set_src(1);
            }
          }
          if (PT::has_inf && p.key == PT::inf_key) break;
          uint64_t sp;
          uint32_t mp;
          T.read_size(p.sid, sp, mp);
          // a promotion needs used_s + sp <= C_S, a swap used_s - sd + sp <= C_S
          // with sd <= used_s (d is in SRAM): neither is legal once sp > C_S,
          // and the pass can stop before it selects d (taken where d waits)
          if constexpr (Tab::kDeferD) {
            if (uc<UNI>(sp > P.cap_sram_B)) break;
          }
          if (uc<UNI>(S.used_s + sp <= P.cap_sram_B && sp <= left)) {
            S.used_h -= sp;
            S.used_s += sp;
            T.set_meta(p.sid, with_tier(mp, kTierSram) | kPrefetched);
            left -= sp;
            moved += sp;
            emit(T, C, S, L, ev, kOpPromote, p.sid, kNone);
            C.promote++;
            C.prom_diff += live_p != p.sid ? 1u : 0u;
            continue;
          }
          if constexpr (Tab::kDeferD) {
            if (d_later) d = T.select_d(K);
          }
          if (d.sid == kNone) break;
          uint64_t sd;
          uint32_t md;
          T.read_size(d.sid, sd, md);
          const bool legal = p.key < d.key && sp <= left && sd <= left - sp &&
                             S.used_s - sd + sp <= P.cap_sram_B && S.used_h - sp + sd <= P.cap_hbm_B;
          if (!uc<UNI>(legal)) break;
          S.used_s = S.used_s - sd + sp;
          S.used_h = S.used_h - sp + sd;
          T.set_meta(p.sid, with_tier(mp, kTierSram) | kPrefetched);
          T.set_meta(d.sid, with_tier(md, kTierHbm));
          left -= sp + sd;
          moved += sp + sd;
          emit(T, C, S, L, ev, kOpSwap, p.sid, d.sid);
          C.swap++;
          C.prom_diff += live_p != p.sid ? 1u : 0u;
        }
        if (uc<UNI>(moved != 0)) {
          // DMA busy for ceil(moved * 1000 / B) ns
          S.dma_free_at = sat_add(now, dma_ns(moved, P.dma_B_per_us));
        }
        C.dma_bytes += moved;
      }
    } else {
      if (tier0 == kTierNone) S.n_table--;
    }
    if constexpr (Tab::kViews) {
      // the copies are refreshed after every request and gap onset, every 8th
      // request, or every gap onset
      if (dual) {
        const bool sync = (P.dual_sync == UNISON_DUAL_EVERY && kind != kDone) ||
                          (P.dual_sync == UNISON_DUAL_EIGHT && kind == kArrive && C.requests % 8u == 0) ||
                          (P.dual_sync == UNISON_DUAL_GAP && kind == kGapStart);
        if (uni32(sync ? 1u : 0u)) T.sync_views();
      }
    }
    if constexpr (Tab::kPrefetch) T.prefetch_land(pf);
    C.events++;
  }
  e_io = e;
}

// Algorithm 1 over the simulation's events [next_event, next_event + max_events).
// UNI: every lane replays the same trace from the same event (one simulation
// per workgroup), so the event record is read as uniform values that live in
// SGPRs: scalar decode and scalar branches on the event kind.
// bad_at is the index of the trace's first event that breaks the event format
// (found once when the traces are loaded, ~0 if none): the run stops there and
// reports it, so the loop itself checks nothing.
template <uint32_t POL, uint32_t SMODE, bool UNI, class Tab>
__device__ __forceinline__ void run_events(Tab& T, const unison_sim_params& P, const KeyCtx& K, const TraceView& tr,
                                           Scalars& S, Cnt& C, const LogSink& L, uint64_t& next_event,
                                           uint64_t max_events, uint64_t bad_at) {
  uint64_t e = next_event;
  uint64_t end = (e >= tr.n_ev || tr.n_ev - e < max_events) ? tr.n_ev : e + max_events;
  const bool stops = bad_at < end;
  if (stops) end = bad_at;
  if (e < end) run_range<POL, SMODE, UNI>(T, P, K, tr, S, C, L, e, end);
  next_event = e;
  if (stops) C.error = bad_at + 1;
}

// The simulation's hazard table into LDS: the counts of its fixed table, or
// of its online table so far (none on a fresh run), and h in both forms.
__device__ __forceinline__ void load_hazard(const SimArgs& a, const unison_sim_params& P,
                                            uint32_t sim, const KeyCtx& K, uint32_t lane,
                                            uint32_t width) {
  const bool online = P.hazard_online != 0;
  const bool fresh = online && !(a.flags & UNISON_RUN_CONTINUE);
  const uint32_t* kd = online ? a.hcount + (size_t)sim * 2 * kLut : a.lut_d + (size_t)P.lut * kLut;
  const uint32_t* kn = online ? kd + kLut : a.lut_n + (size_t)P.lut * kLut;
  for (uint32_t t = lane; t < kLut; t += width) {
    const uint32_t d = fresh ? 0u : kd[t];
    const uint32_t n = fresh ? 0u : kn[t];
    K.hd[t] = d;
    K.hn[t] = n;
    K.hf[t] = hazard_f32(d, n);
    K.hq[t] = hazard_q(d, n, K.lambda);
  }
}

// An online table's counts at the end of the launch, for a later CONTINUE
// and for unison_read_hazard (a fixed table never changes: nothing to store).
__device__ __forceinline__ void store_hazard(const SimArgs& a, const unison_sim_params& P,
                                             uint32_t sim, const KeyCtx& K, uint32_t lane,
                                             uint32_t width) {
  if (!P.hazard_online) return;
  uint32_t* out = a.hcount + (size_t)sim * 2 * kLut;
  for (uint32_t t = lane; t < kLut; t += width) {
    out[t] = K.hd[t];
    out[kLut + t] = K.hn[t];
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
  S.hit_s_bytes = st.hit_s_bytes;
  S.hit_h_bytes = st.hit_h_bytes;
  S.miss_tok = st.miss_tok;
  S.prev_s_bytes = st.prev_s_bytes;
  S.prev_h_bytes = st.prev_h_bytes;
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
  st.hit_s_bytes = S.hit_s_bytes;
  st.hit_h_bytes = S.hit_h_bytes;
  st.miss_tok = S.miss_tok;
  st.prev_s_bytes = S.prev_s_bytes;
  st.prev_h_bytes = S.prev_h_bytes;
}

// eq. (hr-amat) sums from the exact integer totals, rounded once: the same
// quantities the per-request f64 sums approximate.
__device__ __forceinline__ void finish_costs(const Scalars& S, const unison_sim_params& P, Cnt& C) {
  const double a = (double)S.hit_s_bytes * P.t_s_ns_per_B;
  const double b = (double)S.hit_h_bytes * P.t_h_ns_per_B;
  const double c = (double)S.miss_tok * P.t_p_ns_per_tok;
  C.amat = (a + b) + c;
  const double d = (double)S.prev_s_bytes * P.t_s_ns_per_B;
  const double f = (double)S.prev_h_bytes * P.t_h_ns_per_B;
  const double h = (double)C.tokens_computed * P.t_p_ns_per_tok;
  C.ttft = (d + f) + h;
}

__device__ __forceinline__ uint32_t sim_policy(const SimArgs& a, const unison_sim_params& P) {
  return a.policy_override == UNISON_POLICY_PARAMS ? P.policy : a.policy_override;
}

// ------------------------------------------------- register-table kernels

template <int G, int EPL, uint32_t POL, uint32_t SMODE>
__device__ __forceinline__ void regs_run(const SimArgs& a, uint32_t sim, uint32_t lane,
                                      const unison_sim_params& P, const KeyCtx& K) {
  using PT = Pol<POL, SMODE>;
  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  const TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb,
                     a.ev_tool ? a.ev_tool + eb : nullptr, ee - eb, n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  RegTable<G, EPL, POL, SMODE> T;
  T.lane = lane;
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const uint32_t s = (uint32_t)j * G + lane;
    const bool in = s < n_sess;
    T.kvb[j] = in ? a.sess_kvb[sb + s] : 0u;
    const bool ld = cont && in;
    const uint64_t x = ld ? a.t_mg[tb + s] : 0ull;
    T.meta[j] = (uint32_t)x;
    T.g[j] = __uint_as_float((uint32_t)(x >> 32));
    if constexpr (PT::fixed) T.gq[j] = ld ? a.t_gq[tb + s] : 0ull;
    T.len[j] = ld ? a.t_len[tb + s] : 0u;
    T.last[j] = ld ? a.t_last[tb + s] : 0ull;
    if constexpr (PT::nextkey) T.next[j] = ld ? a.t_next[tb + s] : ~0ull;
    T.hz[j] = hazard_of<POL, SMODE>(K, T.meta[j]);
  }
  T.rescore_all(K);  // a resumed table's keys; a fresh table's are never read before its writes

  Scalars S;
  Cnt C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = cnt_from(a.counters[sim]);
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{};
    C = cnt_from(unison_counters{});
  }
  const bool log_on = (a.flags & UNISON_RUN_LOG) && a.log_cap;
  const LogSink L{log_on, log_on ? a.log + (size_t)sim * a.log_cap : nullptr, a.log_cap, lane == 0,
                  log_on && (a.flags & UNISON_RUN_LOG_VICTIM) != 0};
  if (C.error == 0) {
    if (n_sess > (uint32_t)(G * EPL) || P.dual_sync) {
      C.error = ~0ull;  // the launcher picks a variant that holds the trace (and its copies)
    } else {
      run_events<POL, SMODE, false>(T, P, K, tr, S, C, L, next_event, a.max_events,
                                    a.first_bad[P.trace]);
    }
  }

#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const uint32_t s = (uint32_t)j * G + lane;
    if (s < n_sess) {
      a.t_mg[tb + s] = (uint64_t)T.meta[j] | ((uint64_t)__float_as_uint(T.g[j]) << 32);
      if constexpr (PT::fixed) a.t_gq[tb + s] = T.gq[j];
      a.t_len[tb + s] = T.len[j];
      a.t_last[tb + s] = T.last[j];
      if constexpr (PT::nextkey) a.t_next[tb + s] = T.next[j];
    }
  }
  store_hazard(a, P, sim, K, lane, G);
  if (lane == 0) {
    finish_costs(S, P, C);
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = cnt_to(C);
  }
}

template <int G, int EPL>
__global__ __launch_bounds__(256) void sim_regs_kernel(SimArgs a) {
  constexpr int GROUPS = 256 / G;
  __shared__ float s_hf[GROUPS][52];
  __shared__ uint32_t s_hq[GROUPS][52];
  __shared__ uint32_t s_hd[GROUPS][52];
  __shared__ uint32_t s_hn[GROUPS][52];
  const uint32_t gtid = blockIdx.x * 256u + threadIdx.x;
  const uint32_t slot = gtid / G;
  const uint32_t sim = a.slot_sim ? (slot < a.n_slots ? a.slot_sim[slot] : kNone) : slot;
  const uint32_t lane = gtid % G;
  const uint32_t grp = threadIdx.x / G;
  const bool live = sim < a.n_sims;
  const uint32_t simc = live ? sim : 0u;
  const unison_sim_params P = a.params[simc];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  const KeyCtx K{s_hf[grp], s_hq[grp], s_hd[grp], s_hn[grp], P.penalty_us, lambda, P.p_z,
                 a.time44 != 0, P.hazard_online ? P.online_sessions : 0u,
                 a.eta + (size_t)P.trace * kEtaClasses, P.recip_bits};
  load_hazard(a, P, simc, K, lane, G);
  __syncthreads();
  if (!live) return;
  switch (sim_policy(a, P)) {
    case kSpear:
      if (P.score_mode) regs_run<G, EPL, kSpear, 1>(a, sim, lane, P, K);
      else regs_run<G, EPL, kSpear, 0>(a, sim, lane, P, K);
      break;
    case kLru: regs_run<G, EPL, kLru, 0>(a, sim, lane, P, K); break;
    case kTimeout: regs_run<G, EPL, kTimeout, 0>(a, sim, lane, P, K); break;
    case kBelady: regs_run<G, EPL, kBelady, 0>(a, sim, lane, P, K); break;
    default: regs_run<G, EPL, kEta, 0>(a, sim, lane, P, K); break;
  }
}

// ------------------------------------------------- streamed-table kernel

// One workgroup per simulation.  IN_LDS keeps the table in LDS for the whole
// run (copied from and back to the workspace); otherwise it is streamed from
// the workspace in place.
template <int BLOCK, uint32_t POL, uint32_t SMODE, bool IN_LDS, bool VIEWS>
__device__ __forceinline__ void block_run(const SimArgs& a, uint32_t sim, const unison_sim_params& P,
                                          const KeyCtx& K, Cand* s_red, uint64_t* s_tab) {
  const uint32_t tid = threadIdx.x;
  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  const TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb,
                     a.ev_tool ? a.ev_tool + eb : nullptr, ee - eb, n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  constexpr bool kCache = !IN_LDS && !VIEWS;
  MemTable<BLOCK, POL, SMODE, VIEWS, kCache> T;
  T.tid = tid;
  T.parity = 0;
  T.red = s_red;
  T.rc_cap = 0;
  T.rc_used = 0;
  T.kc = K;
  T.n_mine = 0;
  T.w_sid = kNone;
  T.w_x = 0;
  T.w_aux = 0;
  if constexpr (IN_LDS) {
    const uint32_t n = n_sess;
    T.mg = s_tab;
    T.last = s_tab + n;
    T.gq = s_tab + 2 * (size_t)n;
    T.next = s_tab + 3 * (size_t)n;
    uint32_t* s32 = reinterpret_cast<uint32_t*>(s_tab + 4 * (size_t)n);
    T.len = s32;
    uint32_t* kv = s32 + n;
    T.kvb = kv;
    T.res = kv + n;
    for (uint32_t i = tid; i < n; i += BLOCK) {
      T.mg[i] = cont ? a.t_mg[tb + i] : 0ull;
      T.last[i] = cont ? a.t_last[tb + i] : 0ull;
      T.gq[i] = cont ? a.t_gq[tb + i] : 0ull;
      T.next[i] = cont ? a.t_next[tb + i] : ~0ull;
      T.len[i] = cont ? a.t_len[tb + i] : 0u;
      kv[i] = a.sess_kvb[sb + i];
    }
  } else {
    T.mg = a.t_mg + tb;
    T.gq = a.t_gq + tb;
    T.len = a.t_len + tb;
    T.last = a.t_last + tb;
    T.next = a.t_next + tb;
    T.kvb = a.sess_kvb + sb;
    T.res = reinterpret_cast<uint32_t*>(s_tab);
    if constexpr (kCache) {
      // the resident cache's slots follow the residency bits
      const uint32_t cap = a.rc_slots;
      T.rc_cap = cap;
      T.rc_mg = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(s_tab) + a.rc_off);
      T.rc_aux = T.rc_mg + (size_t)cap * BLOCK;
      T.rc_key = T.rc_aux + (size_t)cap * BLOCK;
      T.rc_k = reinterpret_cast<uint32_t*>(T.rc_key + (size_t)cap * BLOCK);
    }
    if (!cont) {
      for (uint32_t i = tid; i < n_sess; i += BLOCK) {
        T.mg[i] = 0;
        T.gq[i] = 0;
        T.len[i] = 0;
        T.last[i] = 0;
        T.next[i] = ~0ull;
      }
    }
  }
  // the dual design's copies, [2][4 fields][max_sessions] per simulation; a
  // fresh run starts them as the empty register file
  const size_t st = a.max_sessions;
  T.view_stride = a.max_sessions;
  T.view0 = a.views ? a.views + (size_t)sim * 8 * st : nullptr;
  T.view1 = a.views ? T.view0 + 4 * st : nullptr;
  T.set_src(-1);
  if (VIEWS && P.dual_sync && a.views && !cont) {
    for (uint32_t i = tid; i < n_sess; i += BLOCK) {
      T.view0[i] = 0;
      T.view0[st + i] = 0;
      T.view0[2 * st + i] = 0;
      T.view0[3 * st + i] = ~0ull;
      T.view1[i] = 0;
      T.view1[st + i] = 0;
      T.view1[2 * st + i] = 0;
      T.view1[3 * st + i] = ~0ull;
    }
  }
  __syncthreads();
  // each thread's residency bits, from the table it resumes (empty if fresh)
  for (uint32_t w = 0; w * 32u * BLOCK < n_sess; ++w) {
    uint32_t bits = 0;
    for (uint32_t b = 0; b < 32u; ++b) {
      const uint32_t i = tid + (w * 32u + b) * BLOCK;
      if (cont && i < n_sess && meta_tier((uint32_t)T.mg[i]) != kTierNone) bits |= 1u << b;
    }
    T.res[w * BLOCK + tid] = bits;
    T.n_mine += (uint32_t)__builtin_popcount(bits);
  }

  Scalars S;
  Cnt C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = cnt_from(a.counters[sim]);
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{};
    C = cnt_from(unison_counters{});
  }
  if (S.hi > n_sess) S.hi = n_sess;  // never scan past the trace's sessions
  T.hi = S.hi;
  if constexpr (kCache) {
    if (T.n_mine && T.n_mine <= T.rc_cap) T.rc_refill();  // a resumed table's residents
  }
  if (P.dual_sync && !(VIEWS && a.views)) C.error = ~0ull;  // the launcher picks the copies' kernel
  pin_vgpr(S);
  pin_vgpr(C);
  const bool log_on = (a.flags & UNISON_RUN_LOG) && a.log_cap;
  const LogSink L{log_on, log_on ? a.log + (size_t)sim * a.log_cap : nullptr, a.log_cap, tid == 0,
                  log_on && (a.flags & UNISON_RUN_LOG_VICTIM) != 0};
  if (C.error == 0) {
    unison_sim_params Pv = P;
    pin_vgpr(Pv);
    run_events<POL, SMODE, true>(T, Pv, K, tr, S, C, L, next_event, a.max_events,
                                 a.first_bad[P.trace]);
  }
  __syncthreads();
  if constexpr (IN_LDS) {
    for (uint32_t i = tid; i < n_sess; i += BLOCK) {
      a.t_mg[tb + i] = T.mg[i];
      a.t_last[tb + i] = T.last[i];
      a.t_gq[tb + i] = T.gq[i];
      a.t_next[tb + i] = T.next[i];
      a.t_len[tb + i] = T.len[i];
    }
  }
  store_hazard(a, P, sim, K, tid, BLOCK);
  if (tid == 0) {
    finish_costs(S, P, C);
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = cnt_to(C);
  }
}

template <int BLOCK, bool IN_LDS, bool VIEWS>
__global__ __launch_bounds__(BLOCK) void sim_block_kernel(SimArgs a) {
  __shared__ float s_hf[52];
  __shared__ uint32_t s_hq[52];
  __shared__ uint32_t s_hd[52];
  __shared__ uint32_t s_hn[52];
  __shared__ Cand s_red[2 * 3 * (BLOCK / 64)];
  extern __shared__ uint64_t s_tab[];
  const uint32_t sim = blockIdx.x;
  const unison_sim_params P = a.params[sim];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  const KeyCtx K{s_hf, s_hq, s_hd, s_hn, P.penalty_us, lambda, P.p_z, a.time44 != 0,
                 P.hazard_online ? P.online_sessions : 0u, a.eta + (size_t)P.trace * kEtaClasses,
                 P.recip_bits};
  load_hazard(a, P, sim, K, threadIdx.x, BLOCK);
  __syncthreads();
  switch (sim_policy(a, P)) {
    case kSpear:
      if (P.score_mode) block_run<BLOCK, kSpear, 1, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab);
      else block_run<BLOCK, kSpear, 0, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab);
      break;
    case kLru: block_run<BLOCK, kLru, 0, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab); break;
    case kTimeout: block_run<BLOCK, kTimeout, 0, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab); break;
    case kBelady: block_run<BLOCK, kBelady, 0, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab); break;
    default: block_run<BLOCK, kEta, 0, IN_LDS, VIEWS>(a, sim, P, K, s_red, s_tab); break;
  }
}

// ------------------------------------------------- slot-table kernel

// One wavefront per simulation: the table in LDS, the residents in SPL VGPR
// slots per lane (SlotTable), events 64 to a window.
template <int SPL, uint32_t POL, uint32_t SMODE>
__device__ __forceinline__ void slot_run(const SimArgs& a, uint32_t sim, const unison_sim_params& P,
                                         const KeyCtx& K, uint64_t* s_tab) {
  const uint32_t lane = threadIdx.x;
  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  const TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb,
                     a.ev_tool ? a.ev_tool + eb : nullptr, ee - eb, n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  SlotTable<SPL, POL, SMODE> T;
  const uint32_t n = n_sess;
  T.mg = s_tab;
  T.last = s_tab + n;
  T.gq = s_tab + 2 * (size_t)n;
  T.next = s_tab + 3 * (size_t)n;
  uint32_t* s32 = reinterpret_cast<uint32_t*>(s_tab + 4 * (size_t)n);
  T.len = s32;
  T.kvb = s32 + n;
  T.lane = lane;
  T.kc = K;
  T.w_sid = kNone;
  T.w_key = 0;
  T.w_kvb = 0;
  T.w_len = 0;
  T.queue_init();
#pragma unroll
  for (int k = 0; k < SPL; ++k) {
    T.ssid[k] = kNone;
    T.smeta[k] = 0;
    T.skey[k] = 0;
    T.ssize[k] = 0;
  }
  for (uint32_t i = lane; i < n; i += 64) {
    T.mg[i] = cont ? a.t_mg[tb + i] : 0ull;
    T.last[i] = cont ? a.t_last[tb + i] : 0ull;
    T.gq[i] = cont ? a.t_gq[tb + i] : 0ull;
    T.next[i] = cont ? a.t_next[tb + i] : ~0ull;
    T.len[i] = cont ? a.t_len[tb + i] : 0u;
    T.kvb[i] = a.sess_kvb[sb + i];
  }
  __syncthreads();
  // a resumed table's residents take slots
  if (cont) {
    for (uint32_t base = 0; base < n; base += 64) {
      const uint32_t i = base + lane;
      const uint32_t ic = i < n ? i : 0u;  // lanes past the table read entry 0
      const bool res = i < n && meta_tier((uint32_t)T.mg[ic]) != kTierNone;
      const uint64_t key = T.key_at(ic);
      const uint64_t size = (uint64_t)T.len[ic] * T.kvb[ic];
      const uint32_t m = (uint32_t)T.mg[ic];
      for (uint64_t bits = __builtin_amdgcn_ballot_w64(res); bits; bits &= bits - 1u) {
        const int l = __builtin_ctzll(bits);
        T.insert(base + (uint32_t)l, (uint32_t)__builtin_amdgcn_readlane((int)m, l),
                 WindowReader<false, false>::lane64(key, l), WindowReader<false, false>::lane64(size, l));
      }
    }
  }

  Scalars S;
  Cnt C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = cnt_from(a.counters[sim]);
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{};
    C = cnt_from(unison_counters{});
  }
  if (S.hi > n_sess) S.hi = n_sess;
  // residents never exceed min(N_sess, sessions): the launcher picks a kernel that holds them
  const uint64_t max_res = P.n_slots < n_sess ? P.n_slots : n_sess;
  if (P.dual_sync || max_res > 64u * SPL) C.error = ~0ull;
  pin_vgpr(S);
  pin_vgpr(C);
  const bool log_on = (a.flags & UNISON_RUN_LOG) && a.log_cap;
  const LogSink L{log_on, log_on ? a.log + (size_t)sim * a.log_cap : nullptr, a.log_cap, lane == 0,
                  log_on && (a.flags & UNISON_RUN_LOG_VICTIM) != 0};
  if (C.error == 0) {
    unison_sim_params Pv = P;
    pin_vgpr(Pv);
    run_events<POL, SMODE, true>(T, Pv, K, tr, S, C, L, next_event, a.max_events,
                                 a.first_bad[P.trace]);
    uint64_t dg, vd;
    T.drain(dg, vd);
    C.digest += dg;
    C.victim_digest += vd;
  }
  __syncthreads();
  for (uint32_t i = lane; i < n; i += 64) {
    a.t_mg[tb + i] = T.mg[i];
    a.t_last[tb + i] = T.last[i];
    a.t_gq[tb + i] = T.gq[i];
    a.t_next[tb + i] = T.next[i];
    a.t_len[tb + i] = T.len[i];
  }
  store_hazard(a, P, sim, K, lane, 64);
  if (lane == 0) {
    finish_costs(S, P, C);
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = cnt_to(C);
  }
}

template <int SPL>
__global__ __launch_bounds__(64) void sim_slot_kernel(SimArgs a) {
  __shared__ float s_hf[52];
  __shared__ uint32_t s_hq[52];
  __shared__ uint32_t s_hd[52];
  __shared__ uint32_t s_hn[52];
  extern __shared__ uint64_t s_tab[];
  const uint32_t sim = blockIdx.x;
  const unison_sim_params P = a.params[sim];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  const KeyCtx K{s_hf, s_hq, s_hd, s_hn, P.penalty_us, lambda, P.p_z, a.time44 != 0,
                 P.hazard_online ? P.online_sessions : 0u, a.eta + (size_t)P.trace * kEtaClasses,
                 P.recip_bits};
  load_hazard(a, P, sim, K, threadIdx.x, 64);
  __syncthreads();
  switch (sim_policy(a, P)) {
    case kSpear:
      if (P.score_mode) slot_run<SPL, kSpear, 1>(a, sim, P, K, s_tab);
      else slot_run<SPL, kSpear, 0>(a, sim, P, K, s_tab);
      break;
    case kLru: slot_run<SPL, kLru, 0>(a, sim, P, K, s_tab); break;
    case kTimeout: slot_run<SPL, kTimeout, 0>(a, sim, P, K, s_tab); break;
    case kBelady: slot_run<SPL, kBelady, 0>(a, sim, P, K, s_tab); break;
    default: slot_run<SPL, kEta, 0>(a, sim, P, K, s_tab); break;
  }
}

// ------------------------------------------------- wide-table kernel

// One wavefront per simulation: the table in the workspace, the residents in
// LDS slots (WideTable), events 64 to a window.  LDS: cap slots of 24 bytes.
constexpr uint32_t kWideSlotBytes = sizeof(uint4) + sizeof(uint64_t);
constexpr uint32_t kWideStageBytes = 6 * sizeof(uint64_t) + LdsWindowReader<true, true>::kBytes;

template <uint32_t POL, uint32_t SMODE>
__device__ __forceinline__ void wide_run(const SimArgs& a, uint32_t sim, const unison_sim_params& P,
                                         const KeyCtx& K, uint64_t* s_tab, uint32_t cap) {
  const uint32_t lane = threadIdx.x;
  const uint64_t eb = a.ev_off[P.trace], ee = a.ev_off[P.trace + 1];
  const uint64_t sb = a.sess_off[P.trace];
  const uint32_t n_sess = (uint32_t)(a.sess_off[P.trace + 1] - sb);
  const TraceView tr{a.ev_t + eb, a.ev_sid + eb, a.ev_info + eb, a.ev_len + eb, a.ev_next + eb,
                     a.ev_tool ? a.ev_tool + eb : nullptr, ee - eb, n_sess};
  const size_t tb = (size_t)sim * a.max_sessions;
  const bool cont = (a.flags & UNISON_RUN_CONTINUE) != 0;

  WideTable<POL, SMODE> T;
  T.mg = a.t_mg + tb;
  T.gq = a.t_gq + tb;
  T.len = a.t_len + tb;
  T.last = a.t_last + tb;
  T.next = a.t_next + tb;
  T.kvb = a.sess_kvb + sb;
  T.slot = a.t_slot + tb;
  T.kc = K;
  T.rec = reinterpret_cast<uint4*>(s_tab);
  T.rsize = reinterpret_cast<uint64_t*>(T.rec + cap);
  T.rows = cap / 64u;
  T.lane = lane;
  T.n_res = 0;
  T.used = 0;
  T.cur = 0;
  T.top = 0;
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    T.bkey[t] = t == 1 ? ~0ull : 0ull;
    T.bsid[t] = kNone;
    T.bslot[t] = 0;
    T.cw_sid[t] = kNone;
    T.cw_slot[t] = kNone;
    T.cw_key[t] = 0;
  }
  T.ci_sid = kNone;
  T.ci_slot = kNone;
  T.dirty = 0;
  T.e_sid = kNone;
  T.e_slot = kNone;
  T.w_sid = kNone;
  T.w_meta = 0;
  T.w_g = 0.0f;
  T.w_gq = T.w_last = T.w_next = 0;
  T.w_kvb = 0;
  T.w_len = 0;
  T.pf_sid = kNone;
  T.stage = T.rsize + cap;
  T.win = T.stage + 6;
  T.pfp = 0;
  T.pp_mg = T.pp_gq = T.pp_last = T.pp_next = 0;
  T.pp_meta = T.pp_len = T.pp_slot = 0;
  T.queue_init();

  Scalars S;
  Cnt C;
  uint64_t next_event = 0;
  if (cont) {
    load_scalars(a.state[sim], S);
    C = cnt_from(a.counters[sim]);
    next_event = a.state[sim].next_event;
  } else {
    S = Scalars{};
    C = cnt_from(unison_counters{});
  }
  if (S.hi > n_sess) S.hi = n_sess;
  // residents never exceed min(N_sess, sessions): the launcher picks a kernel that holds them
  const uint64_t max_res = P.n_slots < n_sess ? P.n_slots : n_sess;
  if (P.dual_sync || max_res > cap) C.error = ~0ull;

  if (!cont) {
    for (uint32_t i = lane; i < n_sess; i += 64) {
      T.mg[i] = 0;
      T.gq[i] = 0;
      T.len[i] = 0;
      T.last[i] = 0;
      T.next[i] = ~0ull;
    }
  }
  __syncthreads();
  // a resumed table's residents take slots, in session order
  if (cont && C.error == 0) {
    for (uint32_t base = 0; base < n_sess; base += 64) {
      const uint32_t i = base + lane;
      const uint32_t ic = i < n_sess ? i : 0u;  // lanes past the table read entry 0
      const uint64_t x = T.mg[ic];
      const bool res = i < n_sess && meta_tier((uint32_t)x) != kTierNone;
      for (uint64_t bits = __builtin_amdgcn_ballot_w64(res); bits; bits &= bits - 1u) {
        const uint32_t sid = base + (uint32_t)__builtin_ctzll(bits);
        if (T.n_res >= cap) {
          C.error = ~0ull;
          break;
        }
        const uint32_t m = uni32((uint32_t)T.mg[sid]);
        T.insert(sid, m, T.key_at(sid), (uint64_t)uni32(T.len[sid]) * uni32(T.kvb[sid]));
      }
    }
    __syncthreads();
  }
  pin_vgpr(S);
  pin_vgpr(C);
  const bool log_on = (a.flags & UNISON_RUN_LOG) && a.log_cap;
  const LogSink L{log_on, log_on ? a.log + (size_t)sim * a.log_cap : nullptr, a.log_cap, lane == 0,
                  log_on && (a.flags & UNISON_RUN_LOG_VICTIM) != 0};
  if (C.error == 0) {
    unison_sim_params Pv = P;
    pin_vgpr(Pv);
    run_events<POL, SMODE, true>(T, Pv, K, tr, S, C, L, next_event, a.max_events,
                                 a.first_bad[P.trace]);
    uint64_t dg, vd;
    T.drain(dg, vd);
    C.digest += dg;
    C.victim_digest += vd;
  }
  __syncthreads();
  store_hazard(a, P, sim, K, lane, 64);
  if (lane == 0) {
    finish_costs(S, P, C);
    store_scalars(a.state[sim], S, next_event);
    a.counters[sim] = cnt_to(C);
  }
}

__global__ __launch_bounds__(64) void sim_wide_kernel(SimArgs a, uint32_t cap) {
  __shared__ float s_hf[52];
  __shared__ uint32_t s_hq[52];
  __shared__ uint32_t s_hd[52];
  __shared__ uint32_t s_hn[52];
  extern __shared__ uint64_t s_tab[];
  const uint32_t sim = blockIdx.x;
  const unison_sim_params P = a.params[sim];
  const uint32_t lambda = (1u << P.b_h) - 1u;
  const KeyCtx K{s_hf, s_hq, s_hd, s_hn, P.penalty_us, lambda, P.p_z, a.time44 != 0,
                 P.hazard_online ? P.online_sessions : 0u, a.eta + (size_t)P.trace * kEtaClasses,
                 P.recip_bits};
  load_hazard(a, P, sim, K, threadIdx.x, 64);
  __syncthreads();
  switch (sim_policy(a, P)) {
    case kSpear:
      if (P.score_mode) wide_run<kSpear, 1>(a, sim, P, K, s_tab, cap);
      else wide_run<kSpear, 0>(a, sim, P, K, s_tab, cap);
      break;
    case kLru: wide_run<kLru, 0>(a, sim, P, K, s_tab, cap); break;
    case kTimeout: wide_run<kTimeout, 0>(a, sim, P, K, s_tab, cap); break;
    case kBelady: wide_run<kBelady, 0>(a, sim, P, K, s_tab, cap); break;
    default: wide_run<kEta, 0>(a, sim, P, K, s_tab, cap); break;
  }
}

// eq. (hazard) counts over a population of turn counts.
__global__ __launch_bounds__(256) void hazard_counts_kernel(const uint32_t* turns, uint32_t n,
                                                            uint32_t* d_out, uint32_t* n_out) {
  __shared__ uint32_t s_end[kLut + 1];   // #{T = t+1} for t < 51, and #{T > 51}
  for (uint32_t t = threadIdx.x; t <= kLut; t += 256) s_end[t] = 0;
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < n; i += 256) {
    const uint32_t T = turns[i];
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

// The ETA table fitted on one trace: per tool class, the mean (floor) of next
// arrival - gap onset over the class's gap onsets that have a next arrival.
// One workgroup; each thread sums its events per class in 128 bits.
__global__ __launch_bounds__(256) void eta_fit_kernel(uint64_t n, const uint64_t* t,
                                                      const uint32_t* info, const uint32_t* tool,
                                                      const uint64_t* next, uint64_t* mean) {
  __shared__ uint64_t s_lo[4][kEtaClasses], s_hi[4][kEtaClasses], s_cnt[4][kEtaClasses];
  uint64_t lo[kEtaClasses], hi[kEtaClasses], cnt[kEtaClasses];
#pragma unroll
  for (uint32_t c = 0; c < kEtaClasses; ++c) lo[c] = hi[c] = cnt[c] = 0;
  for (uint64_t e = threadIdx.x; e < n; e += 256) {
    const uint64_t nx = next[e];
    const uint64_t te = t[e];
    const uint32_t c = tool ? tool[e] : 0u;
    const bool ok = (info[e] >> 24) == kGapStart && nx != ~0ull && nx >= te && c < kEtaClasses;
    const uint64_t g = ok ? nx - te : 0ull;
#pragma unroll
    for (uint32_t k = 0; k < kEtaClasses; ++k) {
      const bool mine = ok && c == k;
      const uint64_t add = mine ? g : 0ull;
      const uint64_t s = lo[k] + add;
      hi[k] += s < lo[k] ? 1ull : 0ull;
      lo[k] = s;
      cnt[k] += mine ? 1ull : 0ull;
    }
  }
  // sum over the wavefront, then over the four wavefronts
#pragma unroll
  for (uint32_t k = 0; k < kEtaClasses; ++k) {
    for (int m = 1; m < 64; m <<= 1) {
      const uint64_t olo = __shfl_xor(lo[k], m), ohi = __shfl_xor(hi[k], m);
      const uint64_t s = lo[k] + olo;
      hi[k] += ohi + (s < lo[k] ? 1ull : 0ull);
      lo[k] = s;
      cnt[k] += __shfl_xor(cnt[k], m);
    }
    if ((threadIdx.x & 63u) == 0) {
      s_lo[threadIdx.x >> 6][k] = lo[k];
      s_hi[threadIdx.x >> 6][k] = hi[k];
      s_cnt[threadIdx.x >> 6][k] = cnt[k];
    }
  }
  __syncthreads();
  if (threadIdx.x < kEtaClasses) {
    const uint32_t k = threadIdx.x;
    unsigned __int128 sum = 0;
    uint64_t c = 0;
    for (int w = 0; w < 4; ++w) {
      sum += ((unsigned __int128)s_hi[w][k] << 64) | s_lo[w][k];
      c += s_cnt[w][k];
    }
    const unsigned __int128 q = c ? sum / c : 0;
    mean[k] = q > (unsigned __int128)~0ull ? ~0ull : (uint64_t)q;
  }
}

hipError_t launch_eta_fit(uint64_t n, const uint64_t* t, const uint32_t* info, const uint32_t* tool,
                          const uint64_t* next, uint64_t* mean, hipStream_t stream) {
  hipLaunchKernelGGL(eta_fit_kernel, dim3(1), dim3(256), 0, stream, n, t, info, tool, next, mean);
  return hipGetLastError();
}

// ------------------------------------------------------------ launchers

struct Variant {
  int g, epl;
};

// Register-table shapes (lanes per simulation x sessions per lane); ids 3
// and 10 stream the table with 256 and 512 threads, id 9 keeps it in LDS,
// id 11 streams it with 512 threads and also keeps the dual design's copies.
// Id 6 (64 x 24, 1,536 sessions in registers) is retired: it spilled almost
// 2 KB per lane, lost to the LDS table on its sizes, and one of its launches
// faulted the GPU on a randomised batch without a cause found.
constexpr Variant kVariants[] = {{16, 1}, {64, 1}, {64, 4}, {0, 0}, {4, 4},
                                 {8, 2},  {-1, 0}, {16, 4}, {32, 8}, {0, 1}, {0, 0}, {0, 0},
                                 {0, 1},  {0, 2},  {0, 3}};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);
constexpr int kBlock = 256;
constexpr int kLdsVariant = 9;
constexpr int kLdsWaveVariant = 12;  // the table in LDS, one wavefront per simulation
constexpr int kDualVariant = 11;  // streamed, 512 threads, with the dual design's copies
constexpr int kSlotVariant = 13;  // the table in LDS, residents in VGPR slots, one wavefront
constexpr uint64_t kSlotMaxResidents = 512;  // 8 slots per lane
constexpr int kWideVariant = 14;  // the table in the workspace, residents in LDS slots, one wavefront
constexpr uint64_t kWideMaxResidents = 4096;  // 96 KiB of slots
constexpr uint32_t kLdsBytesPerSession = 4 * 8 + 2 * 4;  // mg, last, gq, next; len, kvb

// LDS of the workgroup kernels' residency bits: one bit per session, in whole
// words per thread.
static size_t res_bytes(uint32_t n_sess, uint32_t block) {
  const size_t per_word = 32u * (size_t)block;
  return (n_sess + per_word - 1) / per_word * block * sizeof(uint32_t);
}

// Largest dynamic LDS one workgroup may take on the current device.
static uint32_t lds_limit() {
  static int cached = -1;
  if (cached < 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      v = 65536;
    cached = v;
  }
  const uint32_t static_bytes = 2048;  // hazard tables, reduction slots
  return (uint32_t)cached > static_bytes ? (uint32_t)cached - static_bytes : 0u;
}

static uint32_t block_of(int v) { return v == 10 || v == kDualVariant ? 512u : (uint32_t)kBlock; }

uint32_t sim_variant_capacity(int v) {
  if (v < 0 || v >= kNumVariants) return 0;
  const uint32_t lim = lds_limit();
  if (v == kSlotVariant) return lim / kLdsBytesPerSession;  // the table alone
  if (v == kWideVariant) return UNISON_MAX_SESSIONS;  // the table stays in the workspace
  if (v == kLdsVariant || v == kLdsWaveVariant) {
    // the table and its residency bits
    uint32_t n = lim / kLdsBytesPerSession;
    const uint32_t b = v == kLdsVariant ? (uint32_t)kBlock : 64u;
    while (n && (size_t)n * kLdsBytesPerSession + res_bytes(n, b) > lim) --n;
    return n;
  }
  if (kVariants[v].g < 0) return 0;  // retired
  if (kVariants[v].g == 0) {
    // streamed table: the residency bits are the LDS it needs
    const uint32_t b = block_of(v);
    const uint64_t n = (uint64_t)(lim / (b * sizeof(uint32_t))) * 32u * b;
    return n < UNISON_MAX_SESSIONS ? (uint32_t)n : UNISON_MAX_SESSIONS;
  }
  return (uint32_t)(kVariants[v].g * kVariants[v].epl);
}

// Lanes per simulation of a register-table variant; 0 for the workgroup kernels.
uint32_t sim_variant_lanes(int v) {
  if (v < 0 || v >= kNumVariants || kVariants[v].g <= 0) return 0;
  return (uint32_t)kVariants[v].g;
}

// Measured on 4,096-simulation batches: register tables win up to 256
// sessions (32 x 8 takes half the LDS table's time there), the LDS table up
// to its capacity (one wavefront per simulation, which needs no workgroup
// barriers: C2 163 vs 169 ms with 256 threads), then the 512-thread streamed
// table.
int sim_auto_variant(uint32_t max_sess, uint64_t max_slots) {
  if (max_sess <= 16) return 5;
  if (max_sess <= 64) return 7;
  if (max_sess <= 256) return 8;
  if (max_sess <= sim_variant_capacity(kSlotVariant) && max_slots <= 256) return kSlotVariant;
  if (max_sess <= sim_variant_capacity(kLdsWaveVariant)) return kLdsWaveVariant;
  if (max_slots <= kWideMaxResidents) return kWideVariant;
  return 10;
}

// Largest N_sess a variant holds (UNISON_MAX_SESSIONS: no limit of its own).
uint64_t sim_variant_max_slots(int v) {
  if (v == kSlotVariant) return kSlotMaxResidents;
  if (v == kWideVariant) return kWideMaxResidents;
  return UNISON_MAX_SESSIONS;
}

// Whether a variant can run simulations whose N_sess reaches max_slots.
bool sim_variant_slots_ok(int v, uint64_t max_slots) { return max_slots <= sim_variant_max_slots(v); }

// The streamed-table kernels' resident cache: slots per thread of 8 + 8 + 8
// + 4 bytes each, after the residency bits; as many as the LDS left by the bits
// allows, up to kCacheSlots, or fewer when a test pins the count.
constexpr uint32_t kCacheSlots = kCacheSlotsMax;
static size_t cache_bytes(uint32_t slots, uint32_t block) {
  return (size_t)slots * block * (3 * sizeof(uint64_t) + sizeof(uint32_t));
}
static SimArgs with_cache(const SimArgs& a, uint32_t n_sess, uint32_t block, int force_slots) {
  SimArgs b = a;
  const size_t bits = res_bytes(n_sess ? n_sess : 1, block);
  const size_t lim = lds_limit();
  uint32_t slots = 0;
  while (slots < kCacheSlots && bits + cache_bytes(slots + 1, block) <= lim) ++slots;
  if (force_slots >= 0 && (uint32_t)force_slots < slots) slots = (uint32_t)force_slots;
  b.rc_off = (uint32_t)bits;
  b.rc_slots = slots;
  return b;
}

template <int G, int EPL>
static void launch_regs(const SimArgs& a, hipStream_t stream) {
  const uint32_t groups_per_block = 256 / G;
  const uint32_t blocks = (a.n_slots + groups_per_block - 1) / groups_per_block;
  hipLaunchKernelGGL((sim_regs_kernel<G, EPL>), dim3(blocks), dim3(256), 0, stream, a);
}

template <int SPL>
static void launch_slots(const SimArgs& a, uint32_t max_sess_in_batch, hipStream_t stream) {
  const uint32_t n = max_sess_in_batch ? max_sess_in_batch : 1;
  hipLaunchKernelGGL((sim_slot_kernel<SPL>), dim3(a.n_sims), dim3(64), (size_t)n * kLdsBytesPerSession,
                     stream, a);
}

hipError_t launch_sim(const SimArgs& a, uint32_t max_sess_in_batch, uint64_t max_slots,
                      hipStream_t stream, int force_variant, int force_cache_slots) {
  const int v = force_variant >= 0 ? force_variant : sim_auto_variant(max_sess_in_batch, max_slots);
  switch (v) {
    case kSlotVariant:
      if (max_slots <= 64) launch_slots<1>(a, max_sess_in_batch, stream);
      else if (max_slots <= 128) launch_slots<2>(a, max_sess_in_batch, stream);
      else if (max_slots <= 256) launch_slots<4>(a, max_sess_in_batch, stream);
      else if (max_slots <= kSlotMaxResidents) launch_slots<8>(a, max_sess_in_batch, stream);
      else return hipErrorInvalidValue;
      break;
    case kWideVariant: {
      if (max_slots > kWideMaxResidents) return hipErrorInvalidValue;
      const uint32_t cap = (uint32_t)((max_slots ? max_slots : 1) + 63) / 64u * 64u;
      hipLaunchKernelGGL(sim_wide_kernel, dim3(a.n_sims), dim3(64),
                         (size_t)cap * kWideSlotBytes + kWideStageBytes, stream, a, cap);
      break;
    }
    case 0: launch_regs<16, 1>(a, stream); break;
    case 1: launch_regs<64, 1>(a, stream); break;
    case 2: launch_regs<64, 4>(a, stream); break;
    case 4: launch_regs<4, 4>(a, stream); break;
    case 5: launch_regs<8, 2>(a, stream); break;
    case 7: launch_regs<16, 4>(a, stream); break;
    case 8: launch_regs<32, 8>(a, stream); break;
    case kLdsVariant: {
      const uint32_t n = max_sess_in_batch ? max_sess_in_batch : 1;
      const size_t lds = (size_t)n * kLdsBytesPerSession + res_bytes(n, kBlock);
      hipLaunchKernelGGL((sim_block_kernel<kBlock, true, false>), dim3(a.n_sims), dim3(kBlock), lds, stream, a);
      break;
    }
    case kLdsWaveVariant: {
      const uint32_t n = max_sess_in_batch ? max_sess_in_batch : 1;
      const size_t lds = (size_t)n * kLdsBytesPerSession + res_bytes(n, 64);
      hipLaunchKernelGGL((sim_block_kernel<64, true, false>), dim3(a.n_sims), dim3(64), lds, stream, a);
      break;
    }
    case 10: {
      SimArgs b = with_cache(a, max_sess_in_batch, 512, force_cache_slots);
      hipLaunchKernelGGL((sim_block_kernel<512, false, false>), dim3(a.n_sims), dim3(512),
                         b.rc_off + cache_bytes(b.rc_slots, 512), stream, b);
      break;
    }
    case kDualVariant:
      hipLaunchKernelGGL((sim_block_kernel<512, false, true>), dim3(a.n_sims), dim3(512),
                         res_bytes(max_sess_in_batch, 512), stream, a);
      break;
    case 3: {
      SimArgs b = with_cache(a, max_sess_in_batch, kBlock, force_cache_slots);
      hipLaunchKernelGGL((sim_block_kernel<kBlock, false, false>), dim3(a.n_sims), dim3(kBlock),
                         b.rc_off + cache_bytes(b.rc_slots, kBlock), stream, b);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Largest event or next-arrival time over all traces ("never" excluded).
__global__ __launch_bounds__(256) void max_time_kernel(const uint64_t* t, const uint64_t* next,
                                                       uint64_t n, unsigned long long* out) {
  uint64_t m = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x; i < n; i += (uint64_t)gridDim.x * 256u) {
    const uint64_t a = t[i];
    const uint64_t b = next[i];
    m = a > m ? a : m;
    m = (b != ~0ull && b > m) ? b : m;
  }
#pragma unroll
  for (int k = 1; k < 64; k <<= 1) {
    const uint64_t o = __shfl_xor(m, k);
    m = o > m ? o : m;
  }
  if ((threadIdx.x & 63u) == 0) atomicMax(out, (unsigned long long)m);
}

hipError_t launch_max_time(const uint64_t* t, const uint64_t* next, uint64_t n, uint64_t* out,
                           hipStream_t stream) {
  hipError_t e = hipMemsetAsync(out, 0, sizeof(uint64_t), stream);
  if (e != hipSuccess || n == 0) return e;
  const uint64_t want = (n + 255) / 256;
  const uint32_t blocks = (uint32_t)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(max_time_kernel, dim3(blocks), dim3(256), 0, stream, t, next, n,
                     reinterpret_cast<unsigned long long*>(out));
  return hipGetLastError();
}

hipError_t launch_hazard_counts(const uint32_t* turns, uint32_t n, uint32_t* d, uint32_t* nn,
                                hipStream_t stream) {
  hipLaunchKernelGGL(hazard_counts_kernel, dim3(1), dim3(256), 0, stream, turns, n, d, nn);
  return hipGetLastError();
}

}  // namespace unison
