// rank.hip -- register-file EMA replay, the two scorers and the batched
// Kendall tau-b statistics of the ranking-fidelity study (Sec. IV-C, Sec. VI-F).
//
// The scorers are elementwise and HBM-bound (one thread per session, coalesced
// loads, the hazard table in LDS).  The Kendall kernels give each snapshot one
// workgroup and gather its (x, y) pairs into LDS once.  Small snapshots are
// classified pair by pair (each thread owns rows i and walks j > i with all
// lanes of a wave reading the same LDS word, a broadcast); from 256 entries
// on, a bitonic sort and a counting merge sort (merge path from runs of 8)
// find the same counts in O(n log^2 n).
#include <hip/hip_runtime.h>

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


__device__ __forceinline__ bool pair_less(uint32_t xa, uint64_t ya, uint32_t xb, uint64_t yb) {
  return xa < xb || (xa == xb && ya < yb);
}

// Entries per thread and compare-exchanges per thread and pass at the largest
// snapshot.  Each thread runs its compare-exchanges (and its searches) in
// lockstep, so their LDS loads are in flight together.
constexpr uint32_t kSortE = kKendallMax / kSortBlock;
constexpr uint32_t kSortQ = kSortE / 2;
// From runs of this width on, the merge levels use merge path (each thread
// merges its own 8 outputs); narrower runs place each entry by a short
// binary search.
constexpr uint32_t kMergeRun = 8;
// Merge-path levels store entry i at i + i / 8: a thread's 8 consecutive
// outputs then start 72 B after its neighbour's, not 64 B, which spreads a
// wavefront's stores over the LDS banks.
__device__ __forceinline__ uint32_t mp_pad(uint32_t i) { return i + (i >> 3); }
// Entries of each sort buffer, the padding included.
__host__ __device__ __forceinline__ uint32_t sort_buf(uint32_t P) { return P + P / 8; }

// Orders a wavefront's LDS accesses before and after this point (its lanes
// then see each other's stores); no other wavefront waits.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Whether bitonic pass (k, j) is followed by a workgroup barrier.  With
// strides up to 64 every compare-exchange stays inside the 128 entries that
// one wavefront owns for each q (t = tid + q * 512), so two such passes in a
// row need only the wavefront's own in-order LDS accesses between them;
// passes of longer strides exchange entries across wavefronts and take a
// workgroup barrier on both sides (the last pass of a stage precedes the
// first, longest-stride pass of the next).
__host__ __device__ constexpr bool bitonic_barrier_after(uint32_t k, uint32_t j) {
  return j >= 128 || (j == 1 && k >= 128);
}

// Whether merge level w (runs of w merged into runs of 2w) is followed by a
// workgroup barrier.  Levels of runs below 4 keep each entry p = tid + e * 512
// inside its aligned group of 8, which one wavefront owns.  Merge-path levels
// after the first keep a thread's outputs and the runs it reads inside one
// wavefront's 512 consecutive entries (576 padded) while the pair of runs of
// the next level spans at most 512.  The first merge-path level (w = 8) reads
// the plain layout that the search levels wrote, and the next level stores
// padded positions into that same buffer: a wavefront's padded stores there
// reach past its own 512 plain entries into those its neighbour reads at
// w = 8, so that step takes the barrier.  Elsewhere entries cross wavefronts,
// and the last level is followed by the scan of the sorted y.
__host__ __device__ constexpr bool merge_barrier_after(uint32_t w, uint32_t P) {
  return !(w < kMergeRun / 2 ||
           (w > kMergeRun && 4 * w <= (uint32_t)kSortBlock && 2 * w < P));
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

__global__ __launch_bounds__(kSortBlock) void kendall_sort_kernel(uint32_t n_per, uint32_t P,
                                                                  uint64_t n_x, const float* x,
                                                                  const uint64_t* y,
                                                                  const uint32_t* idx,
                                                                  uint64_t* counts, uint8_t* top1) {
  // [P] y, then merge buffer A; [P] merge buffer B, which holds the x keys
  // until the merge sort starts (two buffers of P + P/8 entries, 18 B of LDS
  // per entry: 72 KiB at 4,096, so two snapshots share a CU)
  extern __shared__ uint64_t s_dyn[];
  uint64_t* s_ky = s_dyn;
  uint64_t* s_yb = s_dyn + sort_buf(P);
  uint32_t* s_kx = reinterpret_cast<uint32_t*>(s_yb);
  __shared__ uint64_t s_sum[4][kSortBlock / 64];
  __shared__ float s_bx[kSortBlock / 64];
  __shared__ uint32_t s_bxi[kSortBlock / 64], s_byi[kSortBlock / 64];
  __shared__ uint64_t s_by[kSortBlock / 64];
  __shared__ uint32_t s_bad;
  __shared__ uint32_t s_part[kSortBlock / 64];
  const uint32_t snap = blockIdx.x;
  const uint32_t tid = threadIdx.x;
  const size_t base = (size_t)snap * n_per;
  const uint32_t n = n_per;

  // gather, both argmaxes (ties to the earlier position), padding that sorts last
  if (tid == 0) s_bad = 0;
  __syncthreads();
  float bx = 0.0f;
  uint32_t bxi = kNone, byi = kNone;
  uint64_t by = 0;
  for (uint32_t i = tid; i < P; i += kSortBlock) {
    if (i < n) {
      size_t e = idx ? (size_t)idx[base + i] : base + i;
      if (e >= n_x) {
        s_bad = 1;
        e = 0;
      }
      const float xv = x[e];
      const uint64_t yv = y[e];
      s_kx[i] = float_key(__float_as_uint(xv));
      s_ky[i] = yv;
      if (bxi == kNone || fbetter(xv, i, bx, bxi)) { bx = xv; bxi = i; }
      if (byi == kNone || ubetter(yv, i, by, byi)) { by = yv; byi = i; }
    } else {
      s_kx[i] = 0xFFFFFFFFu;
      s_ky[i] = ~0ull;
    }
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

  uint64_t inv = 0, t_x = 0, t_xy = 0, t_y = 0;
  // bitonic sort of the P pairs by (x, y); a pass's compare-exchanges touch
  // disjoint pairs, so each thread loads all of its pairs before storing any
  for (uint32_t k = 2; k <= P; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      uint32_t ia[kSortQ], xa[kSortQ], xb[kSortQ];
      uint64_t ya[kSortQ], yb[kSortQ];
#pragma unroll
      for (uint32_t q = 0; q < kSortQ; ++q) {
        const uint32_t t = tid + q * kSortBlock;
        const uint32_t i = t < (P >> 1) ? ((t & ~(j - 1)) << 1) | (t & (j - 1)) : 0u;
        ia[q] = t < (P >> 1) ? i : ~0u;
        xa[q] = s_kx[i];
        xb[q] = s_kx[i + j];
        ya[q] = s_ky[i];
        yb[q] = s_ky[i + j];
      }
#pragma unroll
      for (uint32_t q = 0; q < kSortQ; ++q) {
        const uint32_t i = ia[q];
        if (i != ~0u) {
          const bool up = (i & k) == 0;
          if (up ? pair_less(xb[q], yb[q], xa[q], ya[q]) : pair_less(xa[q], ya[q], xb[q], yb[q])) {
            s_kx[i] = xb[q];
            s_kx[i + j] = xa[q];
            s_ky[i] = yb[q];
            s_ky[i + j] = ya[q];
          }
        }
      }
      if (bitonic_barrier_after(k, j)) __syncthreads();
      else wave_lds_sync();
    }
  }
  // pairs tied in x, and in x and y: each entry counts the earlier entries of
  // its run; a run starts where the key differs from the one before, and a
  // max-scan of those starts gives every entry the start of its run
  {
    const uint32_t b = tid * kSortE;
    uint32_t sx[kSortE], sxy[kSortE];
    uint32_t px = 0;
    uint64_t py = 0;
    if (b > 0 && b < P) {
      px = s_kx[b - 1];
      py = s_ky[b - 1];
    }
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = b + e;
      const bool ok = i < P;
      const uint32_t xk = ok ? s_kx[i] : 0u;
      const uint64_t yk = ok ? s_ky[i] : 0ull;
      const bool new_x = i == 0 || xk != px;
      sx[e] = ok && new_x ? i : 0u;
      sxy[e] = ok && (new_x || yk != py) ? i : 0u;
      px = xk;
      py = yk;
    }
    block_max_scan(sx, s_part, tid);
    block_max_scan(sxy, s_part, tid);
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = b + e;
      if (i < n) {
        t_x += i - sx[e];
        t_xy += i - sxy[e];
      }
    }
  }
  __syncthreads();  // the x keys are read for the last time; buffer B is free
  // merge sort of y in that order; a right-run entry is discordant with every
  // larger entry of its left run.  A left-run entry lands after the entries
  // of the right run below it, a right-run entry after those of the left run
  // at or below it.
  uint64_t* src = s_ky;
  uint64_t* dst = s_yb;
  uint32_t steps = 1;  // log2(w) + 1 binary-search steps over a run of w
  for (uint32_t w = 1; w < P; w <<= 1, ++steps) {
    if (w >= kMergeRun) {
      // merge path: thread t writes outputs [8t, 8t + 8) of its pair of
      // runs A (left) and B (right).  A binary search on its diagonal finds
      // how many of them come from A; then it merges sequentially, A first
      // on equal values, and each B entry taken adds the A entries still
      // waiting, all of them larger.
      const uint32_t o0 = tid * kSortE;
      if (o0 < P) {
        const uint32_t b0 = o0 & ~(2 * w - 1);
        const uint32_t d = o0 - b0;
        // the first merge-path level reads the plain layout
        const bool padded = w > kMergeRun;
        auto at = [&](uint32_t k) { return src[padded ? mp_pad(k) : k]; };
        const uint32_t bb = b0 + w;
        uint32_t lo = d > w ? d - w : 0u, hi = d < w ? d : w;
        while (lo < hi) {
          const uint32_t mid = (lo + hi) >> 1;
          if (at(b0 + mid) <= at(bb + d - 1 - mid)) lo = mid + 1;
          else hi = mid;
        }
        uint32_t i = lo, j = d - lo;
        uint64_t a = i < w ? at(b0 + i) : 0ull, b = j < w ? at(bb + j) : 0ull;
#pragma unroll
        for (uint32_t e = 0; e < kSortE; ++e) {
          const bool take_a = i < w && (j >= w || a <= b);
          dst[mp_pad(o0 + e)] = take_a ? a : b;
          if (take_a) {
            ++i;
            a = i < w ? at(b0 + i) : 0ull;
          } else {
            inv += w - i;
            ++j;
            b = j < w ? at(bb + j) : 0ull;
          }
        }
      }
      level_sync(w, P);
      uint64_t* tmp = src;
      src = dst;
      dst = tmp;
      continue;
    }
    uint32_t lo[kSortE], hi[kSortE], rb[kSortE];
    uint64_t v[kSortE];
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t p = tid + e * kSortBlock;
      const bool ok = p < P;
      const uint32_t b0 = p & ~(2 * w - 1);
      const bool left = (p - b0) < w;
      v[e] = ok ? src[p] : 0ull;
      rb[e] = left ? b0 + w : b0;  // the other run
      lo[e] = 0;
      hi[e] = ok ? w : 0u;
    }
    for (uint32_t step = 0; step < steps; ++step) {
#pragma unroll
      for (uint32_t e = 0; e < kSortE; ++e) {
        const uint32_t p = tid + e * kSortBlock;
        const bool left = (p & (2 * w - 1)) < w;
        const uint32_t m = (lo[e] + hi[e]) >> 1;
        const bool open = lo[e] < hi[e];
        const uint64_t a = src[open ? rb[e] + m : 0u];
        const bool goes_right = left ? a < v[e] : a <= v[e];
        lo[e] = open && goes_right ? m + 1 : lo[e];
        hi[e] = open && !goes_right ? m : hi[e];
      }
    }
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t p = tid + e * kSortBlock;
      if (p < P) {
        const uint32_t b0 = p & ~(2 * w - 1);
        const uint32_t off = p - b0;
        if (off < w) {
          dst[b0 + off + lo[e]] = v[e];
        } else {
          dst[b0 + (off - w) + lo[e]] = v[e];
          inv += w - lo[e];
        }
      }
    }
    level_sync(w, P);
    uint64_t* tmp = src;
    src = dst;
    dst = tmp;
  }
  // pairs tied in y: each entry counts the earlier equal entries of the
  // sorted y (real entries hold positions [0, n): the padding sorts last)
  {
    const uint32_t b = tid * kSortE;
    uint32_t sy[kSortE];
    uint64_t py = b > 0 && b < P ? src[mp_pad(b - 1)] : 0ull;
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = b + e;
      const bool ok = i < P;
      const uint64_t yk = ok ? src[mp_pad(i)] : 0ull;
      sy[e] = ok && (i == 0 || yk != py) ? i : 0u;
      py = yk;
    }
    block_max_scan(sy, s_part, tid);
#pragma unroll
    for (uint32_t e = 0; e < kSortE; ++e) {
      const uint32_t i = b + e;
      if (i < n) t_y += i - sy[e];
    }
  }

  uint64_t v[4] = {inv, t_x, t_y, t_xy};
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
    const size_t lds = (size_t)sort_buf(P) * 2 * sizeof(uint64_t);
    hipLaunchKernelGGL(kendall_sort_kernel, dim3(n_snap), dim3(kSortBlock), lds, s, n_per, P, n_x,
                       x, y, idx, counts, top1);
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
    return bitonic_barrier_after(a, b) ? 1 : 0;
  }
  if (step == 1) {  // merge level w = a
    if (a == 0 || a >= P || (a & (a - 1))) return -1;
    return merge_barrier_after(a, P) ? 1 : 0;
  }
  return -1;
}

}  // namespace unison
