// unison_device.h -- device-side arithmetic and layouts of libunison (gfx950).
//
// The session register file of one simulation is a struct-of-arrays table
// indexed by session id.  Each entry holds:
//   mg    u64  low 32 bits: meta = phase | tier << 2 | prefetched << 4 | turn << 5
//              high 32 bits: the fp32 gap EMA g in microseconds (eq. (ema))
//   gq    u64  the integer gap EMA g_q (eq. (gapq), eq. (ema-int))
//   len   u32  resident KV length of the latest turn, tokens
//   last  u64  time of the session's latest event, ns
//   next  u64  time of its next arrival (Belady key), ns
// A scan of SPEAR keys reads only mg: 8 bytes per table entry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/unison.h"

#pragma clang fp contract(off)

namespace unison {

constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr uint32_t kLut = 51;  // t = 0..50, eq. (hazard)

enum : uint32_t { kArrive = 0, kGapStart = 1, kDone = 2 };
enum : uint32_t { kSpear = 0, kLru = 1, kTimeout = 2, kBelady = 3, kEta = 4 };
constexpr uint32_t kEtaClasses = UNISON_ETA_CLASSES;
enum : uint32_t { kTierNone = 0, kTierSram = 1, kTierHbm = 2 };
enum : uint32_t { kUnseen = 0, kServing = 1, kGap = 2, kDoneP = 3 };
enum : uint32_t { kOpEvict = 1, kOpExpire = 2, kOpBypass = 3, kOpPromote = 4, kOpSwap = 5,
                  kOpVictim = 6, kOpPlace = 7 };

__host__ __device__ __forceinline__ uint32_t meta_phase(uint32_t m) { return m & 3u; }
__host__ __device__ __forceinline__ uint32_t meta_tier(uint32_t m) { return (m >> 2) & 3u; }
// Set when TIDE moves the session into SRAM; cleared by its next request.
constexpr uint32_t kPrefetched = 1u << 4;
__host__ __device__ __forceinline__ uint32_t meta_turn(uint32_t m) { return m >> 5; }
__host__ __device__ __forceinline__ uint32_t make_meta(uint32_t ph, uint32_t tier, uint32_t turn) {
  return ph | (tier << 2) | (turn << 5);
}
__host__ __device__ __forceinline__ uint32_t with_tier(uint32_t m, uint32_t tier) {
  return (m & ~0xCu) | (tier << 2);
}
// A resident that is not being served may be evicted or migrated.
__device__ __forceinline__ bool evictable(uint32_t m) {
  return meta_tier(m) != kTierNone && meta_phase(m) != kServing;
}

// SplitMix64 finaliser (Steele, Lea and Flood, 2014).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// Hash of one decision record (event, op, a, b); digests sum these mod 2^64.
// The second word enters through an odd multiplier, then one finaliser pass.
__device__ __forceinline__ uint64_t rec_hash(uint32_t ev, uint32_t op, uint32_t a, uint32_t b) {
  const uint64_t w0 = ((uint64_t)ev << 8) | (uint64_t)op;
  const uint64_t w1 = ((uint64_t)a << 32) | (uint64_t)b;
  return mix64(w0 ^ (w1 * 0x9e3779b97f4a7c15ull));
}

__device__ __forceinline__ uint64_t sat_add(uint64_t a, uint64_t b) {
  uint64_t s = a + b;
  return s < a ? ~0ull : s;
}

// DMA busy time of `bytes` at b bytes/us: ceil(bytes * 1000 / b) ns, b > 0.
// Below 2^53 both the numerator and the divisor fit 64 bits (the quotient
// then needs no 128-bit division, which the compiler expands into a
// bit-serial loop); larger values take the 128-bit form, saturated.
__device__ __forceinline__ uint64_t dma_ns(uint64_t bytes, uint64_t b) {
  if (bytes < (1ull << 53) && b < (1ull << 53)) return (bytes * 1000u + b - 1u) / b;
  const unsigned __int128 q = ((unsigned __int128)bytes * 1000u + b - 1u) / b;
  return q > (unsigned __int128)~0ull ? ~0ull : (uint64_t)q;
}

// a * b saturated to 2^64 - 1.
__device__ __forceinline__ uint64_t sat_mul(uint64_t a, uint64_t b) {
  return __umul64hi(a, b) ? ~0ull : a * b;
}

// s / 10 rounded to nearest even, as the IEEE division gives it.  Between
// 2^-64 and 2^64 the quotient comes from one product and one residual step:
// q0 = s * 0.1f, r = s - 10 * q0 (exact in one fma), q = q0 + r * 0.1f (one
// fma) -- Markstein's correction step (P. Markstein, IBM J. Res. Dev. 34(1),
// 1990) applied to division by a divisor known in advance, the setting of
// Brisebarre, Muller and Raina (IEEE Trans. Computers 53(8), 2004).  Rather
// than rely on the theorem's hypotheses, an exhaustive comparison over every
// finite float shows this equal to the division from 2^-125 upwards; outside
// the window (zero, for one) the division itself runs.  Gap EMAs stay below
// 2^36 us.
__device__ __forceinline__ float div10(float s) {
  if (s >= 0x1p-64f && s <= 0x1p64f) {
    const float q0 = s * 0.1f;
    const float r = __builtin_fmaf(-q0, 10.0f, s);
    return __builtin_fmaf(r, 0.1f, q0);
  }
  return s / 10.0f;
}

// eq. (ema) on the fp32 register.  The sample is the gap in whole
// microseconds (the tau = 10^3 resolution of eq. (lock)), clipped to 32 bits;
// every operation is rounded to fp32.  Gaps below 2^32 ns divide in 32 bits.
__device__ __forceinline__ float ema_f32(float g, uint64_t gap_ns) {
  uint32_t us;
  if (gap_ns < (1ull << 32)) {
    us = (uint32_t)gap_ns / 1000u;
  } else {
    const uint64_t u = gap_ns / 1000u;
    us = u > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)u;
  }
  const float x = (float)us;
  const float a = 3.0f * x;
  const float b = 7.0f * g;
  return div10(a + b);
}

// eq. (gapq) then eq. (ema-int) on the integer register.
__device__ __forceinline__ uint64_t ema_int(uint64_t gq, uint64_t gap_ns, uint32_t b_g, uint64_t tau) {
  uint64_t cap = b_g >= 64 ? ~0ull : ((1ull << b_g) - 1ull);
  uint64_t x = gap_ns / tau;
  if (x > cap) x = cap;
  if (x < (1ull << 60) && gq < (1ull << 60)) return (3ull * x + 7ull * gq) / 10ull;
  unsigned __int128 s = (unsigned __int128)3 * x + (unsigned __int128)7 * gq;
  return (uint64_t)(s / 10u);
}

// Float hazard h(t) = d(t) / n(t) (eq. (hazard)); 0 where n(t) = 0.
__device__ __forceinline__ float hazard_f32(uint32_t d, uint32_t n) {
  return n ? (float)d / (float)n : 0.0f;
}

// eq. (uq) of h = d/n with Lambda = 2^b_h - 1: floor(d/n * Lambda + 1/2),
// computed exactly as (2 d Lambda + n) / (2 n) and clipped to Lambda.
__device__ __forceinline__ uint32_t hazard_q(uint32_t d, uint32_t n, uint32_t lambda) {
  if (n == 0) return 0;
  uint64_t q = (2ull * d * lambda + n) / (2ull * n);
  return q > lambda ? lambda : (uint32_t)q;
}

// eq. (surv) + eq. (esp) for a live session.
__device__ __forceinline__ float spear_f32(float h, float g, float P) {
  float sigma = fmaxf(0.01f, 1.0f - h);
  float a = g / sigma;
  float b = 1.0f - sigma;
  float c = b * P;
  return a + c;
}

// eq. (survq), eq. (t1), eq. (t2), eq. (scoreq) for a live session, b_s = 64.
// recip_bits = W > 0: eq. (t1) multiplies by the reciprocal r = floor(2^W /
// sigma_q + 1/2) -- the entry a table of depth Lambda would hold, computed
// here -- and shifts right by W.
__device__ __forceinline__ uint64_t spear_fixed(uint32_t hq, uint64_t gq, uint32_t lambda,
                                                uint64_t p_z, uint32_t recip_bits) {
  uint32_t eps_q = (lambda + 50u) / 100u;  // floor(Lambda/100 + 1/2)
  uint32_t sigma = lambda - hq;
  if (sigma < eps_q) sigma = eps_q;
  uint64_t t1, t2;
  if (recip_bits) {
    const uint64_t r = ((2ull << recip_bits) + sigma) / (2ull * sigma);
    const unsigned __int128 q = ((unsigned __int128)gq * lambda * r) >> recip_bits;
    t1 = q > (unsigned __int128)~0ull ? ~0ull : (uint64_t)q;
  } else if (gq < (1ull << 47)) {
    t1 = (gq * lambda) / sigma;
  } else {
    unsigned __int128 q = ((unsigned __int128)gq * lambda) / sigma;
    t1 = q > (unsigned __int128)~0ull ? ~0ull : (uint64_t)q;  // saturates like the sum
  }
  uint64_t m = lambda - sigma;
  if (p_z < (1ull << 47)) {
    t2 = (m * p_z) / lambda;
  } else {
    t2 = (uint64_t)(((unsigned __int128)m * p_z) / lambda);
  }
  return sat_add(t1, t2);
}

// Device copy of the workspace regions one kernel launch needs.
struct SimState {
  uint64_t next_event;   // events of the trace already processed
  uint64_t prev_t;       // time of the last processed event
  uint64_t used_s, used_h, dma_free_at;
  uint32_t n_res, n_table;
  uint64_t log_len;
  uint32_t hi;           // 1 + largest session id seen so far
  uint32_t pad;
  // exact sums behind the AMAT and TTFT counters (eq. (hr-amat)): bytes read
  // by SRAM / HBM hits, tokens of missed requests, bytes of the previous
  // prefix on SRAM / HBM hits
  uint64_t hit_s_bytes, hit_h_bytes, miss_tok, prev_s_bytes, prev_h_bytes;
};

struct SimArgs {
  const unison_sim_params* params;
  const uint64_t* ev_off;
  const uint64_t* first_bad;  // [n_traces] first malformed event of each trace, ~0 if none
  const uint64_t* sess_off;
  const uint64_t* ev_t;
  const uint32_t* ev_sid;
  const uint32_t* ev_info;
  const uint32_t* ev_len;
  const uint64_t* ev_next;
  const uint32_t* ev_tool;   // tool class per event, or null (all class 0)
  const uint64_t* eta;       // [n_traces][kEtaClasses] expected wait per tool class, ns
  const uint32_t* sess_kvb;
  const uint32_t* lut_d;   // [n_luts][51]
  const uint32_t* lut_n;
  SimState* state;
  unison_counters* counters;
  uint64_t* t_mg;          // tables [n_sims][max_sessions]
  uint64_t* t_gq;
  uint32_t* t_len;
  uint64_t* t_last;
  uint64_t* t_next;
  uint32_t* t_slot;        // wide-table kernel: the LDS slot of each resident session
  unison_record* log;
  uint32_t* hcount;        // [n_sims][2][51] hazard counts d, n at the end of a launch
  uint64_t* views;         // dual design: [n_sims][2 copies][4 fields][max_sessions], or null
  uint64_t max_events;
  uint32_t n_sims;
  uint32_t max_sessions;
  uint32_t log_cap;
  uint32_t flags;
  uint32_t policy_override;
  uint32_t time44;         // every trace time is below 2^44 - 1 ns
  uint32_t rc_off;         // streamed tables: byte offset of the resident cache in dynamic LDS
  uint32_t rc_slots;       // and its slots per thread (set by the launcher)
  const uint32_t* slot_sim;  // register tables: lane group -> simulation (0xFFFFFFFF: empty), or
                             // null for group g = simulation g
  uint32_t n_slots;        // lane groups the register-table grid covers
};

// Most lane groups of a wavefront (the 4-lane register table's 16).
constexpr uint32_t kMaxGroupsPerWave = 16;

}  // namespace unison
