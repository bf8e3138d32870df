// rank.hip -- register-file EMA replay, the two scorers and the batched
// Kendall tau-b statistics of the ranking-fidelity study (Sec. IV-C, Sec. VI-F).
//
// The scorers are elementwise and HBM-bound (one thread per session, coalesced
// loads, the hazard table in LDS).  The Kendall kernels give each snapshot one
// workgroup, which gathers its (x, y) pairs once.  Small snapshots are
// classified pair by pair (each thread owns rows i and walks j > i with all
// lanes of a wave reading the same LDS word, a broadcast); from 256 entries
// on, a bitonic sort (its passes in groups of three in registers) and a
// counting merge sort (runs of 8 inside each thread, merge path above) find
// the same counts in O(n log^2 n).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "unison_device.h"

#pragma clang fp contract(off)

namespace unison {

__global__ __launch_bounds__(256) void ema_replay_kernel(uint32_t n, uint32_t max_hist,
                                                         const uint64_t* gaps, const uint8_t* n_hist,
                                                         uint32_t b_g, uint64_t tau, float* g_out,
                                                         uint64_t* gq_out) {
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= n) return;
  const uint32_t k_end = n_hist[i] < max_hist ? n_hist[i] : max_hist;
  float g = 0.0f;
  uint64_t gq = 0;
  for (uint32_t k = 0; k < k_end; ++k) {
    const uint64_t gap = gaps[(size_t)i * max_hist + k];
    g = ema_f32(g, gap);
    gq = ema_int(gq, gap, b_g, tau);
  }
  g_out[i] = g;
  gq_out[i] = gq;
}

__global__ __launch_bounds__(256) void score_fp32_kernel(uint32_t n, const uint8_t* turn,
                                                         const float* g, const uint8_t* done,
                                                         const uint32_t* lut_d, const uint32_t* lut_n,
                                                         float P, float* out) {
  __shared__ float hf[52];
  if (threadIdx.x < kLut) hf[threadIdx.x] = hazard_f32(lut_d[threadIdx.x], lut_n[threadIdx.x]);
  __syncthreads();
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= n) return;
  const uint32_t t = turn[i] < 50u ? turn[i] : 50u;
  const float s = spear_f32(hf[t], g[i], P);
  out[i] = done[i] ? __uint_as_float(0x7F800000u) : s;
}

__global__ __launch_bounds__(256) void score_fixed_kernel(uint32_t n, const uint8_t* turn,
                                                          const uint64_t* gq, const uint8_t* done,
                                                          const uint32_t* lut_d,
                                                          const uint32_t* lut_n, uint32_t b_h,
                                                          uint64_t p_z, uint32_t recip_bits,
                                                          uint64_t* out) {
  __shared__ uint32_t hq[52];
  const uint32_t lambda = (1u << b_h) - 1u;
  if (threadIdx.x < kLut) hq[threadIdx.x] = hazard_q(lut_d[threadIdx.x], lut_n[threadIdx.x], lambda);
  __syncthreads();
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= n) return;
  const uint32_t t = turn[i] < 50u ? turn[i] : 50u;
  const uint64_t s = spear_fixed(hq[t], gq[i], lambda, p_z, recip_bits);
  out[i] = done[i] ? ~0ull : s;
}

constexpr int kKendallBlock = 256;
constexpr uint32_t kKendallMax = 4096;  // sort-based path: 18 B of LDS per entry, 72 KiB
constexpr uint32_t kKendallSortFrom = 256;  // snapshots this large or larger are sorted

__device__ __forceinline__ bool fbetter(float a, uint32_t ia, float b, uint32_t ib) {
  return a > b || (a == b && ia < ib);
}
__device__ __forceinline__ bool ubetter(uint64_t a, uint32_t ia, uint64_t b, uint32_t ib) {
  return a > b || (a == b && ia < ib);
}

__global__ __launch_bounds__(kKendallBlock) void kendall_kernel(uint32_t n_per, uint64_t n_x,
                                                                const float* x, const uint64_t* y,
                                                                const uint32_t* idx,
                                                                uint64_t* counts, uint8_t* top1) {
  extern __shared__ uint64_t s_dyn[];
  uint64_t* s_y = s_dyn;                                   // [n_per]
  float* s_x = reinterpret_cast<float*>(s_dyn + n_per);    // [n_per]
  __shared__ uint64_t s_cnt[4][kKendallBlock / 64];
  __shared__ float s_bx[kKendallBlock / 64];
  __shared__ uint32_t s_bxi[kKendallBlock / 64], s_byi[kKendallBlock / 64];
  __shared__ uint64_t s_by[kKendallBlock / 64];
  __shared__ uint32_t s_bad;
  const uint32_t snap = blockIdx.x;
  const uint32_t tid = threadIdx.x;
  const size_t base = (size_t)snap * n_per;

  // gather the snapshot into LDS and find both argmaxes
  if (tid == 0) s_bad = 0;
  __syncthreads();
  float bx = 0.0f;
  uint32_t bxi = kNone, byi = kNone;
  uint64_t by = 0;
  for (uint32_t i = tid; i < n_per; i += kKendallBlock) {
    size_t e = idx ? (size_t)idx[base + i] : base + i;
    if (e >= n_x) {  // an index outside x / y: flag the snapshot, read entry 0
      s_bad = 1;
      e = 0;
    }
    const float xv = x[e];
    const uint64_t yv = y[e];
    s_x[i] = xv;
    s_y[i] = yv;
    if (bxi == kNone || fbetter(xv, i, bx, bxi)) { bx = xv; bxi = i; }
    if (byi == kNone || ubetter(yv, i, by, byi)) { by = yv; byi = i; }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const float ox = __shfl_xor(bx, m);
    const uint32_t oxi = __shfl_xor(bxi, m);
    const uint64_t oy = __shfl_xor(by, m);
    const uint32_t oyi = __shfl_xor(byi, m);
    if (oxi != kNone && (bxi == kNone || fbetter(ox, oxi, bx, bxi))) { bx = ox; bxi = oxi; }
    if (oyi != kNone && (byi == kNone || ubetter(oy, oyi, by, byi))) { by = oy; byi = oyi; }
  }
  if ((tid & 63u) == 0) {
    s_bx[tid >> 6] = bx;
    s_bxi[tid >> 6] = bxi;
    s_by[tid >> 6] = by;
    s_byi[tid >> 6] = byi;
  }
  __syncthreads();

  // pair classification: discordant, tied in x only, tied in y only, both
  uint32_t nd = 0, ntx = 0, nty = 0, nb = 0;
  const uint32_t wave0 = tid & ~63u;
  for (uint32_t r = 0; r * kKendallBlock < n_per; ++r) {
    const uint32_t i = r * kKendallBlock + tid;
    const uint32_t first = r * kKendallBlock + wave0;  // smallest row of this wave
    if (first >= n_per) break;
    const bool row = i < n_per;
    const float xa = s_x[row ? i : 0];
    const uint64_t ya = s_y[row ? i : 0];
    for (uint32_t j = first + 1; j < n_per; ++j) {
      const float xb = s_x[j];
      const uint64_t yb = s_y[j];
      const bool on = row && j > i;
      const bool tx = xa == xb;
      const bool ty = ya == yb;
      const bool gx = xa > xb;
      const bool gy = ya > yb;
      nb += (on && tx && ty) ? 1u : 0u;
      ntx += (on && tx && !ty) ? 1u : 0u;
      nty += (on && !tx && ty) ? 1u : 0u;
      nd += (on && !tx && !ty && gx != gy) ? 1u : 0u;
    }
  }
  uint64_t v[4] = {nd, ntx, nty, nb};
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v[c] += __shfl_xor(v[c], m);
    if ((tid & 63u) == 0) s_cnt[c][tid >> 6] = v[c];
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t tot[4] = {0, 0, 0, 0};
    for (int w = 0; w < kKendallBlock / 64; ++w)
      for (int c = 0; c < 4; ++c) tot[c] += s_cnt[c][w];
    const uint64_t pairs = (uint64_t)n_per * (n_per - 1) / 2;
    counts[(size_t)snap * 5 + 0] = pairs - tot[0] - tot[1] - tot[2] - tot[3];
    counts[(size_t)snap * 5 + 1] = tot[0];
    counts[(size_t)snap * 5 + 2] = tot[1];
    counts[(size_t)snap * 5 + 3] = tot[2];
    counts[(size_t)snap * 5 + 4] = tot[3];
    float fx = s_bx[0];
    uint32_t fxi = s_bxi[0], fyi = s_byi[0];
    uint64_t fy = s_by[0];
    for (int w = 1; w < kKendallBlock / 64; ++w) {
      if (s_bxi[w] != kNone && (fxi == kNone || fbetter(s_bx[w], s_bxi[w], fx, fxi))) {
        fx = s_bx[w];
        fxi = s_bxi[w];
      }
      if (s_byi[w] != kNone && (fyi == kNone || ubetter(s_by[w], s_byi[w], fy, fyi))) {
        fy = s_by[w];
        fyi = s_byi[w];
      }
    }
    top1[snap] = s_bad ? (uint8_t)255 : (uint8_t)(fxi == fyi);
  }
}

// ---------------------------------------------- Kendall tau-b, sort-based

// The same five pair counts in O(n log^2 n) per snapshot (Knight's method):
// sort the pairs by (x, y); pairs tied in x, and in both, are counted from the
// sorted runs; the discordant pairs are the inversions of the y sequence in
// that order, counted while it is merge-sorted; pairs tied in y are counted
// from the finally sorted y.  Concordant = all pairs minus the rest.
constexpr int kSortBlock = 512;

// Order-preserving u32 image of a float, -0 and +0 taken as equal (scores
// are never NaN; a NaN has no place in the order).
__device__ __forceinline__ uint32_t float_key(uint32_t b) {
  if ((b & 0x7FFFFFFFu) == 0) b = 0;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}


// Entries per thread at the largest snapshot.
constexpr uint32_t kSortE = kKendallMax / kSortBlock;
// The merge levels use merge path (each thread merges its own 8 outputs)
// from runs of this width on; the narrower runs are sorted inside each
// thread's 8 consecutive entries.
constexpr uint32_t kMergeRun = 8;
// Sort and merge buffers store entry i at i + i / 8: a thread's 8
// consecutive entries then start 9 entries after its neighbour's, not 8,
// which spreads a wavefront's accesses over the banks; the bitonic groups
// below do the same.  In a merge level neighbouring lanes walk their runs
// about 4 entries apart, which the padding spreads too.
__host__ __device__ constexpr uint32_t mp_pad(uint32_t i) { return i + (i >> 3); }
// Entries of each sort buffer, the padding included.
__host__ __device__ __forceinline__ uint32_t sort_buf(uint32_t P) { return P + P / 8; }

// Orders a wavefront's LDS accesses before and after this point (its lanes
// then see each other's stores); no other wavefront waits.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bitonic passes run in groups, one LDS round trip per group: a thread holds
// the 8 entries whose indexes differ only in bits b, b+1 and b+2 and runs up
// to three consecutive passes on them in registers (strides 2^(b+2), 2^(b+1),
// 2^b).  Stage k = 2^L (L >= 4) splits its passes s = L-1 ... 0 (stride 2^s)
// from the top: L-1..L-3, L-4..L-6, ...; the last group holds the one to
// three passes left and uses bits 0..2.  Stages 2, 4 and 8 form one group on
// each thread's 8 consecutive entries, straight from the gather.
// A wavefront's 64 threads hold 512 entries: while every bit of a group is
// below 9, they are its own aligned block of 512 (the thread index fills the
// other bits from the bottom), so two such groups in a row need only the
// wavefront's in-order LDS accesses between them.
constexpr uint32_t kWaveSpanBits = 9;
__host__ __device__ constexpr uint32_t group_top(uint32_t L, uint32_t s) {
  return L - 1 - 3 * ((L - 1 - s) / 3);
}
__host__ __device__ constexpr uint32_t group_low(uint32_t top) { return top >= 2 ? top - 2 : 0; }
__host__ __device__ constexpr uint32_t group_high(uint32_t top) { return top >= 2 ? top : 2; }
__host__ __device__ constexpr uint32_t ilog2(uint32_t v) {
  uint32_t r = 0;
  while (v > 1) {
    v >>= 1;
    ++r;
  }
  return r;
}

// Whether bitonic pass (k, j) of a P-entry sort is followed by a workgroup
// barrier.  Inside a group the next pass runs in registers; the gathered
// stages end with the barrier that also publishes the argmax partials; the
// last group's entries become the merge input only after every wavefront
// has read its group (the merge buffers reuse the sort's LDS).
// By group: a full group (top >= 3) is followed by a lower group of the same
// stage, so it takes the barrier while its own top bit reaches 9; the last
// group of stage 2^L is followed by the next stage's first group (top L), or
// ends the sort (stage 2^Lp = P).
__host__ __device__ constexpr bool group_barrier_after(uint32_t Lp, uint32_t L, uint32_t top) {
  if (top >= 3) return top >= kWaveSpanBits;
  return L == Lp || L >= kWaveSpanBits;
}
__host__ __device__ constexpr bool bitonic_barrier_after(uint32_t P, uint32_t k, uint32_t j) {
  if (k <= 8) return k == 8 && j == 1;
  const uint32_t L = ilog2(k), s = ilog2(j);
  const uint32_t top = group_top(L, s);
  if (s != group_low(top)) return false;
  return group_barrier_after(ilog2(P), L, top);
}

// Whether merge level w (runs of w merged into runs of 2w, w >= 8) is
// followed by a workgroup barrier.  A thread's outputs and the pair of runs
// it reads lie in its wavefront's 512 consecutive entries (576 padded) while
// a pair of runs spans at most 512, so the barrier is needed only before a
// level whose pairs of runs are wider, and before the scan of the sorted y.
__host__ __device__ constexpr bool merge_barrier_after(uint32_t w, uint32_t P) {
  return !(4 * w <= (uint32_t)kSortBlock && 2 * w < P);
}

__device__ __forceinline__ void level_sync(uint32_t w, uint32_t P) {
  if (merge_barrier_after(w, P)) __syncthreads();
  else wave_lds_sync();
}

// Inclusive max-scan over the workgroup of v[e] at position tid * 8 + e
// (each thread's 8 positions in order): v[e] becomes the largest value at or
// before its position.  s_part: LDS [kSortBlock / 64], free again on return.
__device__ __forceinline__ void block_max_scan(uint32_t (&v)[kSortE], uint32_t* s_part,
                                               uint32_t tid) {
#pragma unroll
  for (uint32_t e = 1; e < kSortE; ++e) v[e] = v[e] > v[e - 1] ? v[e] : v[e - 1];
  const uint32_t lane = tid & 63u;
  uint32_t w = v[kSortE - 1];
#pragma unroll
  for (uint32_t d = 1; d < 64; d <<= 1) {
    const uint32_t o = (uint32_t)__shfl_up((int)w, d);
    if (lane >= d && o > w) w = o;
  }
  uint32_t pre = (uint32_t)__shfl_up((int)w, 1);
  if (lane == 0) pre = 0;
  if (lane == 63) s_part[tid >> 6] = w;
  __syncthreads();
  for (uint32_t k = 0; k < (tid >> 6); ++k) pre = s_part[k] > pre ? s_part[k] : pre;
#pragma unroll
  for (uint32_t e = 0; e < kSortE; ++e) v[e] = v[e] > pre ? v[e] : pre;
  __syncthreads();
}
static_assert(kSortE == 8 && kSortE * kSortBlock == kKendallMax, "8 outputs per thread");

// Compare-exchange of two sort entries, a 64-bit key k and (unless NARROW) a
// 32-bit tie-breaker r: afterwards a precedes b in (k, r) order when up,
// follows it otherwise (equal entries are identical).
template <bool NARROW>
__device__ __forceinline__ void sort_cx(uint64_t& ka, uint32_t& ra, uint64_t& kb, uint32_t& rb,
                                        bool up) {
  // selects, not a branch: the lanes of a pass swap independently
  const bool b_first = NARROW ? kb < ka : ((kb < ka) | ((kb == ka) & (rb < ra)));
  const bool sw = b_first == up;
  const uint64_t k0 = sw ? kb : ka, k1 = sw ? ka : kb;
  ka = k0;
  kb = k1;
  if (!NARROW) {
    const uint32_t r0 = sw ? rb : ra, r1 = sw ? ra : rb;
    ra = r0;
    rb = r1;
  }
}

// One bitonic pass inside a group: entries c and c + 2^M of the thread's 8.
template <uint32_t M, bool NARROW>
__device__ __forceinline__ void sort_pass(uint64_t (&kk)[kSortE], uint32_t (&kr)[kSortE], bool up) {
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c)
    if ((c & (1u << M)) == 0)
      sort_cx<NARROW>(kk[c], kr[c], kk[c | (1u << M)], kr[c | (1u << M)], up);
}

// The thread's entries of the group with low bit lo sit at the padded
// position of its base plus the padded position of c << lo (the base's bits
// below lo and those of c << lo never carry into each other).
__device__ __forceinline__ uint32_t group_base(uint32_t tid, uint32_t lo) {
  return ((tid >> lo) << (lo + 3)) | (tid & ((1u << lo) - 1u));
}

// A full group (three passes) with low bit lo >= 1: the offsets are the same
// for every lane.
template <bool NARROW>
__device__ __forceinline__ void sort_group3(uint32_t lo, uint64_t* s_k, uint32_t* s_r,
                                            uint32_t tid, uint32_t P, uint32_t k) {
  const uint32_t gb = group_base(tid, lo);
  if (gb >= P) return;
  uint64_t kk[kSortE];
  uint32_t kr[kSortE];
  uint64_t* gk = s_k + mp_pad(gb);
  uint32_t* gr = s_r + mp_pad(gb);
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c) {
    const uint32_t off = __builtin_amdgcn_readfirstlane(mp_pad(c << lo));
    kk[c] = gk[off];
    kr[c] = NARROW ? 0u : gr[off];
  }
  const bool up = (gb & k) == 0;
  sort_pass<2, NARROW>(kk, kr, up);
  sort_pass<1, NARROW>(kk, kr, up);
  sort_pass<0, NARROW>(kk, kr, up);
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c) {
    const uint32_t off = __builtin_amdgcn_readfirstlane(mp_pad(c << lo));
    gk[off] = kk[c];
    if (!NARROW) gr[off] = kr[c];
  }
}

// The last group of a stage: low bit 0 (the thread's 8 consecutive entries),
// NP passes.  LAST: the stage-P group that ends the sort keeps its entries in
// registers.
template <uint32_t NP, bool NARROW, bool LAST>
__device__ __forceinline__ void sort_group0(uint64_t (&ko)[kSortE], uint32_t (&ro)[kSortE],
                                            uint64_t* s_k, uint32_t* s_r, uint32_t tid,
                                            uint32_t P, uint32_t k) {
  const uint32_t gb = tid * kSortE;
  if (gb >= P) {
    if (LAST) {  // no entries: padding values (the caller's earlier ones are dead)
#pragma unroll
      for (uint32_t c = 0; c < kSortE; ++c) {
        ko[c] = ~0ull;
        ro[c] = ~0u;
      }
    }
    return;
  }
  uint64_t kk[kSortE];
  uint32_t kr[kSortE];
  const uint32_t pb = mp_pad(gb);
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c) {
    kk[c] = s_k[pb + c];
    kr[c] = NARROW ? 0u : s_r[pb + c];
  }
  const bool up = (gb & k) == 0;
  if (NP == 3) sort_pass<2, NARROW>(kk, kr, up);
  if (NP >= 2) sort_pass<1, NARROW>(kk, kr, up);
  sort_pass<0, NARROW>(kk, kr, up);
  if (!LAST) {
#pragma unroll
    for (uint32_t c = 0; c < kSortE; ++c) {
      s_k[pb + c] = kk[c];
      if (!NARROW) s_r[pb + c] = kr[c];
    }
  } else {
#pragma unroll
    for (uint32_t c = 0; c < kSortE; ++c) {
      ko[c] = kk[c];
      ro[c] = kr[c];
    }
  }
}

template <bool NARROW, bool LAST>
__device__ __forceinline__ void sort_group0_at(uint32_t top, uint64_t (&kk)[kSortE],
                                               uint32_t (&kr)[kSortE], uint64_t* s_k,
                                               uint32_t* s_r, uint32_t tid, uint32_t P,
                                               uint32_t k) {
  if (top == 0) sort_group0<1, NARROW, LAST>(kk, kr, s_k, s_r, tid, P, k);
  else if (top == 1) sort_group0<2, NARROW, LAST>(kk, kr, s_k, s_r, tid, P, k);
  else sort_group0<3, NARROW, LAST>(kk, kr, s_k, s_r, tid, P, k);
}

__device__ __forceinline__ void sort_min_max(uint32_t& a, uint32_t& b) {
  const uint32_t lo = min(a, b);
  b = max(a, b);
  a = lo;
}
__device__ __forceinline__ void sort_min_max(uint64_t& a, uint64_t& b) {
  const bool sw = b < a;
  const uint64_t lo = sw ? b : a;
  b = sw ? a : b;
  a = lo;
}

// The packed form's two merge buffers share the sort's LDS, the second one
// kMergeGap 4-byte words after the first ends, and kMergeGap words follow the
// second: a step may read one entry past a run (a value it never takes),
// which then lands in a gap, never on the other buffer.
constexpr uint32_t kMergeGap = 16;
// The wide form's second buffer starts kWideGap 8-byte entries after the
// first ends, and kWideGap entries follow it, for the same reads.
constexpr uint32_t kWideGap = 8;

// Knight's counts of one snapshot from its gathered entries (thread t holds
// entries 8t ... 8t+7; x as order-preserving u32 keys): the bitonic sort by
// (x, y), the ties in x and in both from the sorted runs, the inversions of y
// in that order counted while it is merge-sorted, the ties in y from the
// sorted y.  cnt = {discordant, ties in x, ties in y, ties in both}.
// NARROW: every y of the snapshot other than 2^64 - 1 lies below 2^32 - 1, so
// y -> (y == 2^64 - 1 ? 2^32 - 1 : y) keeps the order and the ties of y, and
// (x, y) packs into one 64-bit key; otherwise the key is x with the upper
// half of y, and the lower half breaks its ties.
// LDS: the keys sort in a buffer of sort_buf(P) 8-byte entries.  NARROW: the
// merge sort of y then runs in that buffer and the 2 kMergeGap words after it
// (two buffers of sort_buf(P) 4-byte words, the second kMergeGap words after
// the first); otherwise a second buffer of sort_buf(P) 8-byte entries,
// kWideGap entries after the first and followed by kWideGap more, holds the
// tie-breakers, and the merge sort of y starts there and alternates between
// the two.  Every merge buffer holds entry i at i + i / 8.
template <bool NARROW>
__device__ __forceinline__ void sorted_counts(const uint32_t (&kx)[kSortE],
                                              const uint64_t (&ky)[kSortE], uint32_t P,
                                              uint32_t n, uint32_t tid, uint64_t* s_dyn,
                                              uint64_t* s_ek, uint32_t* s_er, uint32_t* s_part,
                                              uint64_t (&cnt)[4]) {
  using Y = typename std::conditional<NARROW, uint32_t, uint64_t>::type;
  uint64_t* s_k = s_dyn;
  uint32_t* s_r = reinterpret_cast<uint32_t*>(s_dyn + sort_buf(P) + kWideGap);
  const uint32_t i0 = tid * kSortE;
  const bool active = i0 < P;
  uint64_t kk[kSortE];
  uint32_t kr[kSortE];
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c) {
    if (NARROW) {
      kk[c] = ((uint64_t)kx[c] << 32) | (ky[c] == ~0ull ? 0xFFFFFFFFu : (uint32_t)ky[c]);
      kr[c] = 0;
    } else {
      kk[c] = ((uint64_t)kx[c] << 32) | (ky[c] >> 32);
      kr[c] = (uint32_t)ky[c];
    }
  }

  // bitonic sort: stages 2, 4 and 8 on the gathered entries (the direction
  // of stage k follows bit k of the entry's index)
#pragma unroll
  for (uint32_t k = 2; k <= 8; k <<= 1)
#pragma unroll
    for (uint32_t j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (uint32_t c = 0; c < kSortE; ++c)
        if ((c & j) == 0) {
          const bool up = k == 8 ? (tid & 1u) == 0 : (c & k) == 0;
          sort_cx<NARROW>(kk[c], kr[c], kk[c | j], kr[c | j], up);
        }
  if (active) {
#pragma unroll
    for (uint32_t c = 0; c < kSortE; ++c) {
      s_k[mp_pad(i0 + c)] = kk[c];
      if (!NARROW) s_r[mp_pad(i0 + c)] = kr[c];
    }
  }
  __syncthreads();
  // then the grouped passes of stages 16 ... P; the last group keeps the
  // thread's 8 consecutive sorted entries in registers
  const uint32_t Lp = 31u - (uint32_t)__builtin_clz(P);
  for (uint32_t L = 4, k = 16; k <= P; ++L, k <<= 1) {
    uint32_t top = L - 1;
    for (; top >= 3; top -= 3) {
      sort_group3<NARROW>(top - 2, s_k, s_r, tid, P, k);
      if (group_barrier_after(Lp, L, top)) __syncthreads();
      else wave_lds_sync();
    }
    if (k == P) {
      sort_group0_at<NARROW, true>(top, kk, kr, s_k, s_r, tid, P, k);
    } else {
      sort_group0_at<NARROW, false>(top, kk, kr, s_k, s_r, tid, P, k);
      if (group_barrier_after(Lp, L, top)) __syncthreads();
      else wave_lds_sync();
    }
  }
  // the entry before the thread's first (the neighbouring thread's last)
  if ((tid & 63u) == 63u) {
    s_ek[tid >> 6] = kk[kSortE - 1];
    s_er[tid >> 6] = kr[kSortE - 1];
  }
  __syncthreads();  // every group is read: the merge buffers are free
  uint64_t pk = __shfl_up(kk[kSortE - 1], 1);
  uint32_t pr = __shfl_up(kr[kSortE - 1], 1);
  if ((tid & 63u) == 0 && tid > 0) {
    pk = s_ek[(tid >> 6) - 1];
    pr = s_er[(tid >> 6) - 1];
  }

  // a thread's counts stay below 2^16 at 4,096 entries: ties at most
  // 8 x 4,095; discordant pairs 28 inside its 8 entries and at most 8 w at
  // merge level w, 8 x (8 + 16 + ... + 2,048) over the levels
  uint32_t inv = 0, t_x = 0, t_xy = 0, t_y = 0;
  Y* src = NARROW ? reinterpret_cast<Y*>(s_dyn) : reinterpret_cast<Y*>(s_dyn + sort_buf(P) + kWideGap);
  Y* dst = NARROW ? reinterpret_cast<Y*>(s_dyn) + sort_buf(P) + kMergeGap : reinterpret_cast<Y*>(s_dyn);
  // pairs tied in x, and in x and y: each entry counts the earlier entries of
  // its run; a run starts where the key differs from the one before, and a
  // max-scan of those starts gives every entry the start of its run
  {
    uint32_t sx[kSortE], sxy[kSortE];
    Y yv[kSortE];
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = i0 + e;
      const bool ok = i < P;
      const bool new_x = i == 0 || (kk[e] >> 32) != (pk >> 32);
      const bool new_xy = new_x || kk[e] != pk || (!NARROW && kr[e] != pr);
      sx[e] = ok && new_x ? i : 0u;
      sxy[e] = ok && new_xy ? i : 0u;
      pk = kk[e];
      pr = kr[e];
      if (NARROW) yv[e] = (Y)(uint32_t)kk[e];
      else yv[e] = (Y)((kk[e] << 32) | kr[e]);
    }
    // merge levels of runs 1, 2 and 4 stay inside the thread's 8 entries:
    // their discordant pairs are the inversions among those 8 y values
    if (active) {
      uint32_t inv8 = 0;
#pragma unroll
      for (uint32_t p = 0; p < kSortE; ++p)
#pragma unroll
        for (uint32_t q = p + 1; q < kSortE; ++q) inv8 += yv[p] > yv[q] ? 1u : 0u;
      inv += inv8;
      // a 19-comparator sorting network on 8 inputs
      sort_min_max(yv[0], yv[2]);
      sort_min_max(yv[1], yv[3]);
      sort_min_max(yv[4], yv[6]);
      sort_min_max(yv[5], yv[7]);
      sort_min_max(yv[0], yv[4]);
      sort_min_max(yv[1], yv[5]);
      sort_min_max(yv[2], yv[6]);
      sort_min_max(yv[3], yv[7]);
      sort_min_max(yv[0], yv[1]);
      sort_min_max(yv[2], yv[3]);
      sort_min_max(yv[4], yv[5]);
      sort_min_max(yv[6], yv[7]);
      sort_min_max(yv[2], yv[4]);
      sort_min_max(yv[3], yv[5]);
      sort_min_max(yv[1], yv[4]);
      sort_min_max(yv[3], yv[6]);
      sort_min_max(yv[1], yv[2]);
      sort_min_max(yv[3], yv[4]);
      sort_min_max(yv[5], yv[6]);
#pragma unroll
      for (uint32_t e = 0; e < kSortE; ++e) src[mp_pad(i0) + e] = yv[e];
    }
    block_max_scan(sx, s_part, tid);
    block_max_scan(sxy, s_part, tid);
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = i0 + e;
      if (i < n) {
        t_x += i - sx[e];
        t_xy += i - sxy[e];
      }
    }
  }
  // merge sort of y in that order from runs of 8 (the scans' barriers
  // publish them); a right-run entry is discordant with every larger entry of
  // its left run.  A left-run entry lands after the entries of the right run
  // below it, a right-run entry after those of the left run at or below it.
  for (uint32_t w = kMergeRun; w < P; w <<= 1) {
    // merge path: thread t writes outputs [8t, 8t + 8) of its pair of runs A
    // (left) and B (right).  A binary search on its diagonal finds how many
    // of them come from A; then it merges sequentially, A first on equal
    // values, and each B entry taken adds the A entries still waiting, all of
    // them larger.
    if (active) {
      const uint32_t b0 = i0 & ~(2 * w - 1);
      const uint32_t d = i0 - b0;
      uint32_t lo = d > w ? d - w : 0u, hi = d < w ? d : w;
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (src[mp_pad(b0 + mid)] <= src[mp_pad(b0 + w + d - 1 - mid)]) lo = mid + 1;
        else hi = mid;
      }
      // Each step takes the smaller head (A's on equal values) and reloads
      // only the run it took from, by selects rather than a branch.  A run
      // with no entries left has its head one past its end: that value is
      // read but never taken.
      uint32_t xa = b0 + lo, xb = b0 + w + (d - lo);
      uint32_t na = w - lo, nb = w - (d - lo), waiting = 0;
      Y a = src[mp_pad(xa)], b = src[mp_pad(xb)];
      Y out[kSortE];
#pragma unroll
      for (uint32_t e = 0; e < kSortE; ++e) {
        const bool take_a = (na != 0) & ((nb == 0) | (a <= b));
        out[e] = take_a ? a : b;
        waiting += take_a ? 0u : na;
        na -= take_a ? 1u : 0u;
        nb -= take_a ? 0u : 1u;
        xa += take_a ? 1u : 0u;
        xb += take_a ? 0u : 1u;
        const Y v = src[mp_pad(take_a ? xa : xb)];
        a = take_a ? v : a;
        b = take_a ? b : v;
      }
#pragma unroll
      for (uint32_t e = 0; e < kSortE; ++e) dst[mp_pad(i0) + e] = out[e];
      inv += waiting;
    }
    level_sync(w, P);
    Y* tmp = src;
    src = dst;
    dst = tmp;
  }
  // pairs tied in y: each entry counts the earlier equal entries of the
  // sorted y (real entries hold positions [0, n): the padding sorts last)
  {
    uint32_t sy[kSortE];
    Y py = i0 > 0 && i0 < P ? src[mp_pad(i0 - 1)] : (Y)0;
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = i0 + e;
      const bool ok = i < P;
      const Y yk = ok ? src[mp_pad(i)] : (Y)0;
      sy[e] = ok && (i == 0 || yk != py) ? i : 0u;
      py = yk;
    }
    block_max_scan(sy, s_part, tid);
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = i0 + e;
      if (i < n) t_y += i - sy[e];
    }
  }
  cnt[0] = inv;
  cnt[1] = t_x;
  cnt[2] = t_y;
  cnt[3] = t_xy;
}

// The top-1 value a snapshot keeps between the two launches when its y values
// need the wide form.
constexpr uint8_t kWideMark = 254;

// NARROW: every snapshot whose y values pack (see sorted_counts) is counted
// here with half the LDS, so four snapshots share a CU; the others are left
// marked in top1.  Otherwise only the marked snapshots are counted.  The
// packed form asks for eight wavefronts per SIMD (at most 64 VGPRs), so that
// four of its blocks fit a CU as its LDS allows.
template <bool NARROW>
__global__ __launch_bounds__(kSortBlock, NARROW ? 8 : 4)
void kendall_sort_kernel(uint32_t n_per, uint32_t P, uint64_t n_x, const float* x,
                         const uint64_t* y, const uint32_t* idx, uint64_t* counts,
                         uint8_t* top1) {
  // one (NARROW, and 2 kMergeGap 4-byte words) or two buffers of P + P/8
  // 8-byte entries (and 2 kWideGap entries): 36 or 72 KiB at 4,096 entries
  extern __shared__ __attribute__((aligned(16))) uint64_t s_dyn[];
  __shared__ uint64_t s_sum[4][kSortBlock / 64];
  __shared__ float s_bx[kSortBlock / 64];
  __shared__ uint32_t s_bxi[kSortBlock / 64], s_byi[kSortBlock / 64];
  __shared__ uint64_t s_by[kSortBlock / 64];
  __shared__ uint32_t s_bad, s_wide;
  __shared__ uint32_t s_part[kSortBlock / 64];
  __shared__ uint64_t s_ek[kSortBlock / 64];
  __shared__ uint32_t s_er[kSortBlock / 64];
  const uint32_t snap = blockIdx.x;
  const uint32_t tid = threadIdx.x;
  const size_t base = (size_t)snap * n_per;
  const uint32_t n = n_per;
  if (!NARROW && top1[snap] != kWideMark) return;

  // gather each thread's 8 consecutive entries into registers, both argmaxes
  // (ties to the earlier position), padding that sorts last, and whether a y
  // other than 2^64 - 1 reaches 2^32 - 1
  if (tid == 0) {
    s_bad = 0;
    s_wide = 0;
  }
  __syncthreads();
  float bx = 0.0f;
  uint32_t bxi = kNone, byi = kNone;
  uint64_t by = 0;
  const uint32_t i0 = tid * kSortE;
  uint32_t kx[kSortE];
  uint64_t ky[kSortE];
  bool wide = false;
#pragma unroll
  for (uint32_t c = 0; c < kSortE; ++c) {
    const uint32_t i = i0 + c;
    kx[c] = 0xFFFFFFFFu;
    ky[c] = ~0ull;
    if (i < n) {
      size_t e = idx ? (size_t)idx[base + i] : base + i;
      if (e >= n_x) {
        s_bad = 1;
        e = 0;
      }
      const float xv = x[e];
      const uint64_t yv = y[e];
      kx[c] = float_key(__float_as_uint(xv));
      ky[c] = yv;
      wide = wide || (yv != ~0ull && yv >= 0xFFFFFFFFull);
      if (bxi == kNone || fbetter(xv, i, bx, bxi)) { bx = xv; bxi = i; }
      if (byi == kNone || ubetter(yv, i, by, byi)) { by = yv; byi = i; }
    }
  }
  if (wide) s_wide = 1;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const float ox = __shfl_xor(bx, m);
    const uint32_t oxi = __shfl_xor(bxi, m);
    const uint64_t oy = __shfl_xor(by, m);
    const uint32_t oyi = __shfl_xor(byi, m);
    if (oxi != kNone && (bxi == kNone || fbetter(ox, oxi, bx, bxi))) { bx = ox; bxi = oxi; }
    if (oyi != kNone && (byi == kNone || ubetter(oy, oyi, by, byi))) { by = oy; byi = oyi; }
  }
  if ((tid & 63u) == 0) {
    s_bx[tid >> 6] = bx;
    s_bxi[tid >> 6] = bxi;
    s_by[tid >> 6] = by;
    s_byi[tid >> 6] = byi;
  }
  __syncthreads();

  if (NARROW && __builtin_amdgcn_readfirstlane(s_wide)) {
    if (tid == 0) top1[snap] = kWideMark;
    return;
  }
  uint64_t v[4];
  sorted_counts<NARROW>(kx, ky, P, n, tid, s_dyn, s_ek, s_er, s_part, v);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v[c] += __shfl_xor(v[c], m);
    if ((tid & 63u) == 0) s_sum[c][tid >> 6] = v[c];
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t tot[4] = {0, 0, 0, 0};
    for (int w = 0; w < kSortBlock / 64; ++w)
      for (int c = 0; c < 4; ++c) tot[c] += s_sum[c][w];
    const uint64_t pairs = (uint64_t)n * (n - 1) / 2;
    const uint64_t d = tot[0], both = tot[3];
    const uint64_t only_x = tot[1] - both, only_y = tot[2] - both;
    counts[(size_t)snap * 5 + 0] = pairs - d - only_x - only_y - both;
    counts[(size_t)snap * 5 + 1] = d;
    counts[(size_t)snap * 5 + 2] = only_x;
    counts[(size_t)snap * 5 + 3] = only_y;
    counts[(size_t)snap * 5 + 4] = both;
    float fx = s_bx[0];
    uint32_t fxi = s_bxi[0], fyi = s_byi[0];
    uint64_t fy = s_by[0];
    for (int w = 1; w < kSortBlock / 64; ++w) {
      if (s_bxi[w] != kNone && (fxi == kNone || fbetter(s_bx[w], s_bxi[w], fx, fxi))) {
        fx = s_bx[w];
        fxi = s_bxi[w];
      }
      if (s_byi[w] != kNone && (fyi == kNone || ubetter(s_by[w], s_byi[w], fy, fyi))) {
        fy = s_by[w];
        fyi = s_byi[w];
      }
    }
    top1[snap] = s_bad ? (uint8_t)255 : (uint8_t)(fxi == fyi);
  }
}

hipError_t launch_ema_replay(uint32_t n, uint32_t max_hist, const uint64_t* gaps,
                             const uint8_t* n_hist, uint32_t b_g, uint64_t tau, float* g,
                             uint64_t* gq, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(ema_replay_kernel, dim3((n + 255) / 256), dim3(256), 0, s, n, max_hist, gaps,
                     n_hist, b_g, tau, g, gq);
  return hipGetLastError();
}

hipError_t launch_score_fp32(uint32_t n, const uint8_t* turn, const float* g, const uint8_t* done,
                             const uint32_t* d, const uint32_t* nn, float P, float* out,
                             hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(score_fp32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, n, turn, g, done, d,
                     nn, P, out);
  return hipGetLastError();
}

hipError_t launch_score_fixed(uint32_t n, const uint8_t* turn, const uint64_t* gq,
                              const uint8_t* done, const uint32_t* d, const uint32_t* nn,
                              uint32_t b_h, uint64_t p_z, uint32_t recip_bits, uint64_t* out,
                              hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(score_fixed_kernel, dim3((n + 255) / 256), dim3(256), 0, s, n, turn, gq, done,
                     d, nn, b_h, p_z, recip_bits, out);
  return hipGetLastError();
}

hipError_t launch_kendall(uint32_t n_snap, uint32_t n_per, uint64_t n_x, const float* x,
                          const uint64_t* y, const uint32_t* idx, uint64_t* counts, uint8_t* top1,
                          hipStream_t s) {
  if (n_snap == 0) return hipSuccess;
  if (n_per < kKendallSortFrom) {
    const size_t lds = (size_t)(n_per ? n_per : 1) * (sizeof(uint64_t) + sizeof(float));
    hipLaunchKernelGGL(kendall_kernel, dim3(n_snap), dim3(kKendallBlock), lds, s, n_per, n_x, x, y,
                       idx, counts, top1);
  } else {
    uint32_t P = 2;
    while (P < n_per) P <<= 1;
    // the packed form first; then the snapshots it left marked
    const size_t lds = (size_t)sort_buf(P) * sizeof(uint64_t);
    hipLaunchKernelGGL(kendall_sort_kernel<true>, dim3(n_snap), dim3(kSortBlock),
                       lds + 2 * kMergeGap * sizeof(uint32_t), s, n_per, P,
                       n_x, x, y, idx, counts, top1);
    hipLaunchKernelGGL(kendall_sort_kernel<false>, dim3(n_snap), dim3(kSortBlock),
                       2 * lds + 2 * kWideGap * sizeof(uint64_t), s, n_per,
                       P, n_x, x, y, idx, counts, top1);
  }
  return hipGetLastError();
}

uint32_t kendall_max_per() { return kKendallMax; }

// The sort kernel's barrier plan, for host-side checks: 1 when the step is
// followed by a workgroup barrier, 0 when by the wavefront-local fence.
int kendall_barrier_after(uint32_t P, uint32_t step, uint32_t a, uint32_t b) {
  if (P < kKendallSortFrom || P > kKendallMax || (P & (P - 1))) return -1;
  if (step == 0) {  // bitonic pass (k = a, j = b)
    if (a < 2 || a > P || (a & (a - 1)) || b == 0 || b >= a || (b & (b - 1))) return -1;
    return bitonic_barrier_after(P, a, b) ? 1 : 0;
  }
  if (step == 1) {  // merge level w = a (runs below 8 are merged in registers)
    if (a < kMergeRun || a >= P || (a & (a - 1))) return -1;
    return merge_barrier_after(a, P) ? 1 : 0;
  }
  return -1;
}

}  // namespace unison
