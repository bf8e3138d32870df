// api.cpp -- host side of the libunison C ABI (see include/unison.h).
//
// Validates arguments, carves the caller's workspace into the simulation
// state regions, copies the small host-side tables (offsets, parameters) into
// it and launches the kernels on the caller's stream.  No device memory is
// allocated here and no exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "unison_device.h"

namespace unison {
hipError_t launch_sim(const SimArgs& a, uint32_t max_sess_in_batch, uint64_t max_slots, hipStream_t stream,
                      int force_variant, int force_cache_slots);
uint32_t sim_variant_capacity(int v);
int sim_auto_variant(uint32_t max_sess, uint64_t max_slots);
bool sim_variant_slots_ok(int v, uint64_t max_slots);
uint64_t sim_variant_max_slots(int v);
uint32_t sim_variant_lanes(int v);
hipError_t launch_hazard_counts(const uint32_t* turns, uint32_t n, uint32_t* d, uint32_t* nn,
                                hipStream_t stream);
hipError_t launch_eta_fit(uint64_t n, const uint64_t* t, const uint32_t* info, const uint32_t* tool,
                          const uint64_t* next, uint64_t* mean, hipStream_t stream);
hipError_t launch_max_time(const uint64_t* t, const uint64_t* next, uint64_t n, uint64_t* out,
                           hipStream_t stream);
hipError_t launch_ema_replay(uint32_t n, uint32_t max_hist, const uint64_t* gaps,
                             const uint8_t* n_hist, uint32_t b_g, uint64_t tau, float* g,
                             uint64_t* gq, hipStream_t s);
hipError_t launch_score_fp32(uint32_t n, const uint8_t* turn, const float* g, const uint8_t* done,
                             const uint32_t* d, const uint32_t* nn, float P, float* out,
                             hipStream_t s);
hipError_t launch_score_fixed(uint32_t n, const uint8_t* turn, const uint64_t* gq,
                              const uint8_t* done, const uint32_t* d, const uint32_t* nn,
                              uint32_t b_h, uint64_t p_z, uint32_t recip_bits, uint64_t* out,
                              hipStream_t s);
hipError_t launch_kendall(uint32_t n_snap, uint32_t n_per, uint64_t n_x, const float* x,
                          const uint64_t* y, const uint32_t* idx, uint64_t* counts, uint8_t* top1,
                          hipStream_t s);
uint32_t kendall_max_per();
int kendall_barrier_after(uint32_t P, uint32_t step, uint32_t a, uint32_t b);
}  // namespace unison

using namespace unison;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Workspace layout; offsets in bytes from the workspace base.
struct Layout {
  size_t params, ev_off, first_bad, sess_off, lut_d, lut_n, eta, state, counters, hcount, mg, gq, len,
      last, next, slot, views, log, slots, scratch, total;
};

bool make_layout(const unison_dims& d, Layout& L) {
  const size_t entries = (size_t)d.n_sims * d.max_sessions;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.params = take(sizeof(unison_sim_params) * d.n_sims);
  L.ev_off = take(sizeof(uint64_t) * (d.n_traces + 1));
  L.first_bad = take(sizeof(uint64_t) * d.n_traces);
  L.sess_off = take(sizeof(uint64_t) * (d.n_traces + 1));
  L.lut_d = take(sizeof(uint32_t) * kLut * d.n_luts);
  L.lut_n = take(sizeof(uint32_t) * kLut * d.n_luts);
  L.eta = take(sizeof(uint64_t) * UNISON_ETA_CLASSES * d.n_traces);
  L.state = take(sizeof(SimState) * d.n_sims);
  L.counters = take(sizeof(unison_counters) * d.n_sims);
  L.hcount = take(sizeof(uint32_t) * 2 * kLut * d.n_sims);
  L.mg = take(sizeof(uint64_t) * entries);
  L.gq = take(sizeof(uint64_t) * entries);
  L.len = take(sizeof(uint32_t) * entries);
  L.last = take(sizeof(uint64_t) * entries);
  L.next = take(sizeof(uint64_t) * entries);
  L.slot = take(sizeof(uint32_t) * entries);
  L.views = take(d.views ? sizeof(uint64_t) * 8 * entries : 0);
  L.log = take(sizeof(unison_record) * (size_t)d.log_cap * d.n_sims);
  // register-table lane groups -> simulations: at most one partly filled
  // wavefront per simulation, of up to kMaxGroupsPerWave groups
  L.slots = take(sizeof(uint32_t) * (size_t)kMaxGroupsPerWave * d.n_sims);
  L.scratch = take(256);
  L.total = off;
  return true;
}

// Index of the first event of a trace that breaks the event format, or ~0:
// a session id past the trace's sessions, a kind above DONE, a time before
// the previous event's; an ARRIVE of turn 0 for a session already seen, of
// turn k >= 1 that does not follow the GAP_START of turn k - 1 or shortens the
// prefix; a GAP_START or DONE of a session that is not being served; a
// GAP_START whose tool class is UNISON_ETA_CLASSES or more.  These depend on
// the trace alone, so they are checked once per load.
uint64_t first_bad_event(const uint64_t* t, const uint32_t* sid, const uint32_t* info,
                         const uint32_t* len, const uint32_t* tool, uint64_t n, uint32_t n_sess) {
  struct Sess {
    uint32_t phase, turn, len;  // phase: 0 unseen, 1 served, 2 in a gap, 3 completed
  };
  std::vector<Sess> st(n_sess, Sess{0, 0, 0});
  uint64_t prev = 0;
  for (uint64_t e = 0; e < n; ++e) {
    const uint32_t s = sid[e], kind = info[e] >> 24, turn = info[e] & 0xFFFFFFu;
    if (s >= n_sess || kind > 2 || t[e] < prev) return e;
    prev = t[e];
    Sess& x = st[s];
    if (kind == 0) {
      if (turn == 0 ? x.phase != 0 : (x.phase != 2 || turn != x.turn + 1 || len[e] < x.len)) return e;
      x.phase = 1;
      x.turn = turn;
      x.len = len[e];
    } else {
      if (x.phase != 1) return e;
      if (kind == 1 && tool && tool[e] >= UNISON_ETA_CLASSES) return e;
      x.phase = kind == 1 ? 2 : 3;
    }
  }
  return ~0ull;
}

// The workspace of contexts made by unison_create_static: a file-scope
// device array, one copy per GPU the library runs on, held until the
// process ends.  Host code never passes the array's name to a kernel or a
// copy (on the host it is only a stand-in for the symbol): it takes each
// device's address once, with hipGetSymbolAddress on that device, and uses
// that address wherever the workspace is needed.
constexpr int kStaticMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[UNISON_STATIC_WORKSPACE_BYTES];

struct StaticWorkspace {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
  std::atomic<uint64_t> gen{0};  // bumped by every unison_create_static on the device
};
StaticWorkspace g_static[kStaticMaxDevices];

// Message of the latest failed create call on this thread (no context yet).
thread_local char g_create_err[256] = "";

int create_fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_create_err, sizeof g_create_err, fmt, ap);
  va_end(ap);
  return code;
}

bool dims_ok(const unison_dims* d) {
  return d && d->n_sims >= 1 && d->n_traces >= 1 && d->n_luts >= 1 && d->max_sessions >= 1 &&
         d->max_sessions <= UNISON_MAX_SESSIONS && d->views <= 1;
}

}  // namespace

struct unison_ctx {
  unison_dims dims;
  hipStream_t stream;
  char* ws;
  size_t ws_bytes;
  Layout L;
  unison_trace_batch tb;
  std::vector<uint64_t> h_ev_off, h_sess_off, h_first_bad;
  std::vector<unison_sim_params> h_params;
  std::vector<uint8_t> lut_set;
  std::vector<uint8_t> eta_set;  // per trace: an ETA table was installed
  bool traces_loaded = false, params_set = false, ran = false;
  bool time44 = false;  // every trace time is below 2^44 - 1 ns
  bool dual = false;    // some row uses the dual register-file design
  uint32_t max_sess_batch = 0;
  uint64_t max_slots_batch = 0;  // largest N_sess of the parameter rows
  int force_variant = -1;
  int force_cache_slots = -1;  // test hook: resident-cache slots of the streamed tables
  // the register-table kernels' lane-group -> simulation map (slot_map)
  std::vector<uint32_t> h_slots;
  uint64_t params_gen = 0;         // bumped by every unison_set_params
  uint64_t slots_for = ~0ull;      // (params_gen, policy override, lanes) the map was built for
  bool slots_identity = true;
  uint32_t n_slots = 0;
  int static_dev = -1;       // unison_create_static: the device whose array is the workspace
  uint64_t static_gen = 0;   // and the array's generation this context was made for
  char err[512];

  template <class T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }

  int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(err, sizeof err, fmt, ap);
    va_end(ap);
    return code;
  }
  int hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return UNISON_OK;
    return fail(UNISON_E_HIP, "%s: %s", what, hipGetErrorString(e));
  }
  // A context on the device's static array is superseded once a newer one
  // takes the array over.
  bool superseded() const {
    return static_dev >= 0 && g_static[static_dev].gen.load() != static_gen;
  }
  int refuse_superseded() {
    return fail(UNISON_E_INVALID,
                "context superseded: a later unison_create_static on device %d took over its "
                "workspace", static_dev);
  }
};

#define UNISON_LIVE(ctx)                                   \
  do {                                                     \
    if ((ctx)->superseded()) return (ctx)->refuse_superseded(); \
  } while (0)

extern "C" {

uint32_t unison_version(void) { return 1u; }

const char* unison_strerror(int code) {
  switch (code) {
    case UNISON_OK: return "ok";
    case UNISON_E_INVALID: return "invalid argument";
    case UNISON_E_BAD_TRACE: return "trace breaks the event format";
    case UNISON_E_CAPACITY: return "session count above the supported maximum";
    case UNISON_E_HIP: return "HIP runtime error";
    case UNISON_E_NOT_READY: return "traces, hazard tables or parameters missing";
    default: return "unknown error";
  }
}

const char* unison_last_error(const unison_ctx* ctx) {
  if (ctx) return ctx->err;
  return g_create_err[0] ? g_create_err : "null context";
}

int unison_workspace_size(const unison_dims* d, size_t* bytes) {
  if (!dims_ok(d) || !bytes) return UNISON_E_INVALID;
  Layout L;
  make_layout(*d, L);
  *bytes = L.total;
  return UNISON_OK;
}

int unison_create(unison_ctx** out, const unison_dims* d, void* hip_stream, void* workspace,
                  size_t workspace_bytes) {
  if (!out || !dims_ok(d) || !workspace) return UNISON_E_INVALID;
  *out = nullptr;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign) return UNISON_E_INVALID;
  Layout L;
  make_layout(*d, L);
  if (workspace_bytes < L.total) return UNISON_E_INVALID;
  unison_ctx* c = new (std::nothrow) unison_ctx();
  if (!c) return UNISON_E_INVALID;
  c->dims = *d;
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  c->ws = reinterpret_cast<char*>(workspace);
  c->ws_bytes = workspace_bytes;
  c->L = L;
  c->lut_set.assign(d->n_luts, 0);
  c->err[0] = 0;
  std::memset(&c->tb, 0, sizeof c->tb);
  *out = c;
  return UNISON_OK;
}

int unison_create_static(unison_ctx** out, const unison_dims* d, void* hip_stream) {
  if (!out || !dims_ok(d)) return create_fail(UNISON_E_INVALID, "null output or invalid dims");
  *out = nullptr;
  Layout L;
  make_layout(*d, L);
  if (L.total > (size_t)UNISON_STATIC_WORKSPACE_BYTES)
    return create_fail(UNISON_E_CAPACITY,
                       "these dims need a workspace of %zu bytes; the static workspace holds %zu",
                       L.total, (size_t)UNISON_STATIC_WORKSPACE_BYTES);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kStaticMaxDevices)
    return create_fail(UNISON_E_HIP, "no current HIP device (or device id above %d)",
                       kStaticMaxDevices - 1);
  StaticWorkspace& sw = g_static[dev];
  std::call_once(sw.once, [&] { sw.err = hipGetSymbolAddress(&sw.ptr, HIP_SYMBOL(scratch)); });
  if (sw.err != hipSuccess || !sw.ptr)
    return create_fail(UNISON_E_HIP, "address of the static workspace on device %d: %s", dev,
                       hipGetErrorString(sw.err));
  unison_ctx* c = new (std::nothrow) unison_ctx();
  if (!c) return create_fail(UNISON_E_INVALID, "out of host memory for the context");
  c->dims = *d;
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  c->ws = reinterpret_cast<char*>(sw.ptr);
  c->ws_bytes = UNISON_STATIC_WORKSPACE_BYTES;
  c->L = L;
  c->lut_set.assign(d->n_luts, 0);
  c->err[0] = 0;
  std::memset(&c->tb, 0, sizeof c->tb);
  c->static_dev = dev;
  c->static_gen = sw.gen.fetch_add(1) + 1;
  g_create_err[0] = 0;
  *out = c;
  return UNISON_OK;
}

void unison_destroy(unison_ctx* ctx) { delete ctx; }

int unison_set_stream(unison_ctx* ctx, void* hip_stream) {
  if (!ctx) return UNISON_E_INVALID;
  ctx->stream = reinterpret_cast<hipStream_t>(hip_stream);
  return UNISON_OK;
}

int unison_load_traces(unison_ctx* ctx, const unison_trace_batch* tb) {
  if (!ctx || !tb) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  const uint32_t nt = tb->n_traces;
  if (nt != ctx->dims.n_traces)
    return ctx->fail(UNISON_E_INVALID, "n_traces %u differs from dims %u", nt, ctx->dims.n_traces);
  if (!tb->ev_offset || !tb->sess_offset || !tb->ev_t_ns || !tb->ev_sid || !tb->ev_info ||
      !tb->ev_len || !tb->ev_next_ns || !tb->sess_kvb)
    return ctx->fail(UNISON_E_INVALID, "null trace array");
  for (uint32_t i = 0; i < nt; ++i) {
    if (tb->ev_offset[i + 1] < tb->ev_offset[i] || tb->sess_offset[i + 1] < tb->sess_offset[i])
      return ctx->fail(UNISON_E_INVALID, "trace %u: offsets decrease", i);
    if (tb->ev_offset[i + 1] - tb->ev_offset[i] > 0xFFFFFFFFull)
      return ctx->fail(UNISON_E_INVALID, "trace %u: more than 2^32-1 events", i);
    const uint64_t ns = tb->sess_offset[i + 1] - tb->sess_offset[i];
    if (ns > ctx->dims.max_sessions)
      return ctx->fail(UNISON_E_CAPACITY, "trace %u has %llu sessions > max_sessions %u", i,
                       (unsigned long long)ns, ctx->dims.max_sessions);
  }
  ctx->tb = *tb;
  ctx->eta_set.assign(nt, 0);
  ctx->h_ev_off.assign(tb->ev_offset, tb->ev_offset + nt + 1);
  ctx->h_sess_off.assign(tb->sess_offset, tb->sess_offset + nt + 1);
  int rc = ctx->hip(hipMemcpyAsync(ctx->at<uint64_t>(ctx->L.ev_off), ctx->h_ev_off.data(),
                                   sizeof(uint64_t) * (nt + 1), hipMemcpyHostToDevice, ctx->stream),
                    "copy event offsets");
  if (rc) return rc;
  rc = ctx->hip(hipMemcpyAsync(ctx->at<uint64_t>(ctx->L.sess_off), ctx->h_sess_off.data(),
                               sizeof(uint64_t) * (nt + 1), hipMemcpyHostToDevice, ctx->stream),
                "copy session offsets");
  if (rc) return rc;
  // the largest time decides whether recency / Belady keys pack into 44 bits
  uint64_t* d_max = ctx->at<uint64_t>(ctx->L.scratch);
  rc = ctx->hip(launch_max_time(tb->ev_t_ns, tb->ev_next_ns, tb->ev_offset[nt], d_max, ctx->stream),
                "largest trace time");
  if (rc) return rc;
  uint64_t h_max = 0;
  rc = ctx->hip(hipMemcpyAsync(&h_max, d_max, sizeof h_max, hipMemcpyDeviceToHost, ctx->stream),
                "copy largest trace time");
  if (rc) return rc;
  rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise after offsets");
  if (rc) return rc;
  ctx->time44 = h_max < (1ull << 44) - 1;
  // the event format, checked once per trace on a host copy of its events
  ctx->h_first_bad.assign(nt, ~0ull);
  std::vector<uint64_t> ht;
  std::vector<uint32_t> hs, hi, hl, hk;
  for (uint32_t i = 0; i < nt; ++i) {
    const uint64_t b = tb->ev_offset[i], n = tb->ev_offset[i + 1] - b;
    if (n == 0) continue;
    ht.resize(n);
    hs.resize(n);
    hi.resize(n);
    hl.resize(n);
    hk.resize(tb->ev_tool ? n : 0);
    rc = ctx->hip(hipMemcpyAsync(ht.data(), tb->ev_t_ns + b, n * sizeof(uint64_t), hipMemcpyDeviceToHost,
                                 ctx->stream), "copy trace times");
    if (rc == UNISON_OK)
      rc = ctx->hip(hipMemcpyAsync(hs.data(), tb->ev_sid + b, n * sizeof(uint32_t), hipMemcpyDeviceToHost,
                                   ctx->stream), "copy trace sessions");
    if (rc == UNISON_OK)
      rc = ctx->hip(hipMemcpyAsync(hi.data(), tb->ev_info + b, n * sizeof(uint32_t), hipMemcpyDeviceToHost,
                                   ctx->stream), "copy trace kinds");
    if (rc == UNISON_OK)
      rc = ctx->hip(hipMemcpyAsync(hl.data(), tb->ev_len + b, n * sizeof(uint32_t), hipMemcpyDeviceToHost,
                                   ctx->stream), "copy trace lengths");
    if (rc == UNISON_OK && tb->ev_tool)
      rc = ctx->hip(hipMemcpyAsync(hk.data(), tb->ev_tool + b, n * sizeof(uint32_t), hipMemcpyDeviceToHost,
                                   ctx->stream), "copy trace tool classes");
    if (rc == UNISON_OK) rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise trace copy");
    if (rc) return rc;
    ctx->h_first_bad[i] = first_bad_event(ht.data(), hs.data(), hi.data(), hl.data(),
                                          tb->ev_tool ? hk.data() : nullptr, n,
                                          (uint32_t)(tb->sess_offset[i + 1] - tb->sess_offset[i]));
  }
  rc = ctx->hip(hipMemcpyAsync(ctx->at<uint64_t>(ctx->L.first_bad), ctx->h_first_bad.data(),
                               sizeof(uint64_t) * nt, hipMemcpyHostToDevice, ctx->stream),
                "copy format checks");
  if (rc) return rc;
  rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise format checks");
  if (rc) return rc;
  ctx->traces_loaded = true;
  return UNISON_OK;
}

int unison_hazard_counts(void* hip_stream, const uint32_t* turns, uint32_t n, uint32_t* d_out,
                         uint32_t* n_out) {
  if ((!turns && n) || !d_out || !n_out) return UNISON_E_INVALID;
  hipError_t e = launch_hazard_counts(turns, n, d_out, n_out, reinterpret_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? UNISON_OK : UNISON_E_HIP;
}

int unison_eta_fit(void* hip_stream, uint64_t n_events, const uint64_t* ev_t_ns, const uint32_t* ev_info,
                   const uint32_t* ev_tool, const uint64_t* ev_next_ns, uint64_t* mean_out) {
  if (!mean_out || (n_events && (!ev_t_ns || !ev_info || !ev_next_ns))) return UNISON_E_INVALID;
  hipError_t e = launch_eta_fit(n_events, ev_t_ns, ev_info, ev_tool, ev_next_ns, mean_out,
                                reinterpret_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? UNISON_OK : UNISON_E_HIP;
}

int unison_set_eta(unison_ctx* ctx, uint32_t trace, const uint64_t* mean) {
  if (!ctx || !mean) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (!ctx->traces_loaded) return ctx->fail(UNISON_E_NOT_READY, "load traces before ETA tables");
  if (trace >= ctx->dims.n_traces) return ctx->fail(UNISON_E_INVALID, "trace %u >= n_traces", trace);
  int rc = ctx->hip(hipMemcpyAsync(ctx->at<uint64_t>(ctx->L.eta) + (size_t)trace * UNISON_ETA_CLASSES,
                                   mean, sizeof(uint64_t) * UNISON_ETA_CLASSES,
                                   hipMemcpyDeviceToDevice, ctx->stream),
                    "copy ETA table");
  if (rc) return rc;
  ctx->eta_set[trace] = 1;
  return UNISON_OK;
}

int unison_set_hazard(unison_ctx* ctx, uint32_t lut, const uint32_t* d, const uint32_t* n) {
  if (!ctx || !d || !n) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (lut >= ctx->dims.n_luts) return ctx->fail(UNISON_E_INVALID, "lut %u >= n_luts", lut);
  int rc = ctx->hip(hipMemcpyAsync(ctx->at<uint32_t>(ctx->L.lut_d) + (size_t)lut * kLut, d,
                                   sizeof(uint32_t) * kLut, hipMemcpyDeviceToDevice, ctx->stream),
                    "copy hazard d");
  if (rc) return rc;
  rc = ctx->hip(hipMemcpyAsync(ctx->at<uint32_t>(ctx->L.lut_n) + (size_t)lut * kLut, n,
                               sizeof(uint32_t) * kLut, hipMemcpyDeviceToDevice, ctx->stream),
                "copy hazard n");
  if (rc) return rc;
  ctx->lut_set[lut] = 1;
  return UNISON_OK;
}

int unison_set_params(unison_ctx* ctx, const unison_sim_params* params) {
  if (!ctx || !params) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (!ctx->traces_loaded) return ctx->fail(UNISON_E_NOT_READY, "load traces before parameters");
  uint32_t max_sess = 0;
  uint64_t max_slots = 0;
  for (uint32_t i = 0; i < ctx->dims.n_sims; ++i) {
    const unison_sim_params& p = params[i];
    if (p.dual_sync > UNISON_DUAL_GAP || (p.dual_sync && !ctx->dims.views))
      return ctx->fail(UNISON_E_INVALID, "parameter row %u: dual_sync %u (dims.views = %u)", i,
                       p.dual_sync, ctx->dims.views);
    if (p.policy > UNISON_POLICY_ETA || p.tide > 1 || p.score_mode > 1 || p.hazard_online > 1 ||
        p.lut >= ctx->dims.n_luts || p.trace >= ctx->dims.n_traces || p.b_h < 6 || p.b_h > 16 ||
        p.b_g < 1 || p.b_g > 64 || p.tau_ns < 1 || p.n_slots < 1 || p.dma_B_per_us < 1 ||
        p.recip_bits > 32 ||
        !(p.penalty_us >= 0.0f) || std::isinf(p.penalty_us) || !std::isfinite(p.t_s_ns_per_B) ||
        !std::isfinite(p.t_h_ns_per_B) || !std::isfinite(p.t_p_ns_per_tok))
      return ctx->fail(UNISON_E_INVALID, "parameter row %u out of range", i);
    const uint64_t ns = ctx->h_sess_off[p.trace + 1] - ctx->h_sess_off[p.trace];
    max_sess = std::max<uint32_t>(max_sess, (uint32_t)ns);
    max_slots = std::max<uint64_t>(max_slots, p.n_slots);
  }
  ctx->h_params.assign(params, params + ctx->dims.n_sims);
  ctx->dual = false;
  for (uint32_t i = 0; i < ctx->dims.n_sims; ++i) ctx->dual = ctx->dual || params[i].dual_sync != 0;
  int rc = ctx->hip(hipMemcpyAsync(ctx->at<unison_sim_params>(ctx->L.params), ctx->h_params.data(),
                                   sizeof(unison_sim_params) * ctx->dims.n_sims,
                                   hipMemcpyHostToDevice, ctx->stream),
                    "copy parameters");
  if (rc) return rc;
  rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise after parameters");
  if (rc) return rc;
  ctx->max_sess_batch = max_sess;
  ctx->max_slots_batch = max_slots;
  ctx->params_set = true;
  ctx->params_gen++;
  return UNISON_OK;
}

// Register-table kernels run a group of `lanes` lanes per simulation, 64 /
// lanes groups to a wavefront, and a wavefront executes every path any of
// its simulations takes.  The map puts simulations that share policy, score
// form and trace side by side and starts a new wavefront where they change
// (the groups left over stay empty), so a wavefront never serialises two
// policies or two traces' event kinds.  A batch already in that order keeps
// the identity map (no map at all).
static int slot_map(unison_ctx* ctx, uint32_t policy_override, uint32_t lanes) {
  const uint64_t key = (ctx->params_gen << 16) ^ ((uint64_t)policy_override << 8) ^ lanes;
  if (ctx->slots_for == key) return UNISON_OK;
  const uint32_t n = ctx->dims.n_sims;
  const uint32_t gpw = 64u / lanes;
  if (gpw == 1) {  // one simulation per wavefront: nothing to group
    ctx->slots_identity = true;
    ctx->n_slots = n;
    ctx->slots_for = key;
    return UNISON_OK;
  }
  auto sort_key = [&](uint32_t i) {
    const unison_sim_params& p = ctx->h_params[i];
    const uint32_t pol = policy_override == UNISON_POLICY_PARAMS ? p.policy : policy_override;
    const uint32_t mode = pol == UNISON_POLICY_SPEAR ? p.score_mode : 0u;
    return ((uint64_t)pol << 40) | ((uint64_t)mode << 32) | p.trace;
  };
  std::vector<uint32_t> order(n);
  for (uint32_t i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](uint32_t a, uint32_t b) { return sort_key(a) < sort_key(b); });
  ctx->h_slots.clear();
  for (uint32_t j = 0; j < n; ++j) {
    if (j && sort_key(order[j]) != sort_key(order[j - 1]))
      while (ctx->h_slots.size() % gpw) ctx->h_slots.push_back(0xFFFFFFFFu);
    ctx->h_slots.push_back(order[j]);
  }
  bool identity = ctx->h_slots.size() == n;
  for (uint32_t j = 0; identity && j < n; ++j) identity = ctx->h_slots[j] == j;
  ctx->slots_identity = identity;
  ctx->n_slots = identity ? n : (uint32_t)ctx->h_slots.size();
  if (!identity) {
    int rc = ctx->hip(hipMemcpyAsync(ctx->at<uint32_t>(ctx->L.slots), ctx->h_slots.data(),
                                     sizeof(uint32_t) * ctx->h_slots.size(), hipMemcpyHostToDevice,
                                     ctx->stream),
                      "copy lane-group map");
    if (rc) return rc;
    rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise after lane-group map");
    if (rc) return rc;
  }
  ctx->slots_for = key;
  return UNISON_OK;
}

int unison_run(unison_ctx* ctx, uint32_t policy_override, uint32_t flags, uint64_t max_events) {
  if (!ctx) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (!ctx->traces_loaded || !ctx->params_set)
    return ctx->fail(UNISON_E_NOT_READY, "traces and parameters must be set before a run");
  for (const auto& p : ctx->h_params)
    if (!ctx->lut_set[p.lut]) return ctx->fail(UNISON_E_NOT_READY, "hazard table %u not set", p.lut);
  if (policy_override != UNISON_POLICY_PARAMS && policy_override > UNISON_POLICY_ETA)
    return ctx->fail(UNISON_E_INVALID, "policy %u", policy_override);
  for (const auto& p : ctx->h_params) {
    const uint32_t pol = policy_override == UNISON_POLICY_PARAMS ? p.policy : policy_override;
    if (pol == UNISON_POLICY_ETA && !ctx->eta_set[p.trace])
      return ctx->fail(UNISON_E_NOT_READY, "ETA table of trace %u not set", p.trace);
  }
  if (flags & ~(UNISON_RUN_CONTINUE | UNISON_RUN_LOG | UNISON_RUN_LOG_VICTIM))
    return ctx->fail(UNISON_E_INVALID, "flags");
  if ((flags & UNISON_RUN_CONTINUE) && !ctx->ran)
    return ctx->fail(UNISON_E_NOT_READY, "UNISON_RUN_CONTINUE before any run on this context");
  SimArgs a;
  std::memset(&a, 0, sizeof a);
  a.params = ctx->at<unison_sim_params>(ctx->L.params);
  a.ev_off = ctx->at<uint64_t>(ctx->L.ev_off);
  a.first_bad = ctx->at<uint64_t>(ctx->L.first_bad);
  a.sess_off = ctx->at<uint64_t>(ctx->L.sess_off);
  a.ev_t = ctx->tb.ev_t_ns;
  a.ev_sid = ctx->tb.ev_sid;
  a.ev_info = ctx->tb.ev_info;
  a.ev_len = ctx->tb.ev_len;
  a.ev_next = ctx->tb.ev_next_ns;
  a.ev_tool = ctx->tb.ev_tool;
  a.eta = ctx->at<uint64_t>(ctx->L.eta);
  a.sess_kvb = ctx->tb.sess_kvb;
  a.lut_d = ctx->at<uint32_t>(ctx->L.lut_d);
  a.lut_n = ctx->at<uint32_t>(ctx->L.lut_n);
  a.state = ctx->at<SimState>(ctx->L.state);
  a.counters = ctx->at<unison_counters>(ctx->L.counters);
  a.t_mg = ctx->at<uint64_t>(ctx->L.mg);
  a.t_gq = ctx->at<uint64_t>(ctx->L.gq);
  a.t_len = ctx->at<uint32_t>(ctx->L.len);
  a.t_last = ctx->at<uint64_t>(ctx->L.last);
  a.t_next = ctx->at<uint64_t>(ctx->L.next);
  a.t_slot = ctx->at<uint32_t>(ctx->L.slot);
  a.log = ctx->dims.log_cap ? ctx->at<unison_record>(ctx->L.log) : nullptr;
  a.hcount = ctx->at<uint32_t>(ctx->L.hcount);
  a.views = ctx->dims.views ? ctx->at<uint64_t>(ctx->L.views) : nullptr;
  a.max_events = max_events;
  a.n_sims = ctx->dims.n_sims;
  a.max_sessions = ctx->dims.max_sessions;
  a.log_cap = ctx->dims.log_cap;
  a.flags = flags;
  a.policy_override = policy_override;
  a.time44 = ctx->time44 ? 1u : 0u;
  int v = ctx->force_variant;
  // the dual design's copies live in the workspace: its streamed-table kernel runs it
  if (ctx->dual) {
    if (v < 0) v = 11;
    if (v != 11)
      return ctx->fail(UNISON_E_INVALID, "dual register files run on variant 11, not %d", v);
  }
  if (v >= 0 && (sim_variant_capacity(v) == 0 || sim_variant_capacity(v) < ctx->max_sess_batch))
    return ctx->fail(UNISON_E_CAPACITY, "forced kernel variant %d holds %u sessions < %u", v,
                     sim_variant_capacity(v), ctx->max_sess_batch);
  // residents never exceed min(N_sess, sessions) of a simulation
  const uint64_t max_res = std::min<uint64_t>(ctx->max_slots_batch, ctx->max_sess_batch);
  if (v >= 0 && !sim_variant_slots_ok(v, max_res))
    return ctx->fail(UNISON_E_CAPACITY, "forced kernel variant %d holds up to %llu residents, not %llu", v,
                     (unsigned long long)sim_variant_max_slots(v), (unsigned long long)max_res);
  if (v < 0) {
    v = sim_auto_variant(ctx->max_sess_batch, max_res);
    if (sim_variant_capacity(v) < ctx->max_sess_batch)
      return ctx->fail(UNISON_E_CAPACITY, "%u sessions exceed every kernel variant (largest %u)",
                       ctx->max_sess_batch, sim_variant_capacity(v));
  }
  a.slot_sim = nullptr;
  a.n_slots = a.n_sims;
  if (const uint32_t lanes = sim_variant_lanes(v)) {
    const int mrc = slot_map(ctx, policy_override, lanes);
    if (mrc) return mrc;
    if (!ctx->slots_identity) {
      a.slot_sim = ctx->at<uint32_t>(ctx->L.slots);
      a.n_slots = ctx->n_slots;
    }
  }
  int rc = ctx->hip(launch_sim(a, ctx->max_sess_batch, max_res, ctx->stream, v,
                               ctx->force_cache_slots),
                    "launch simulation");
  if (rc == UNISON_OK) ctx->ran = true;
  return rc;
}

int unison_read_counters(unison_ctx* ctx, unison_counters* dst, uint32_t first, uint32_t n) {
  if (!ctx || (!dst && n)) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if ((uint64_t)first + n > ctx->dims.n_sims) return ctx->fail(UNISON_E_INVALID, "range");
  int rc = ctx->hip(hipMemcpyAsync(dst, ctx->at<unison_counters>(ctx->L.counters) + first,
                                   sizeof(unison_counters) * n, hipMemcpyDeviceToHost, ctx->stream),
                    "copy counters");
  if (rc) return rc;
  rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise counters");
  if (rc) return rc;
  for (uint32_t i = 0; i < n; ++i)
    if (dst[i].error) return ctx->fail(UNISON_E_BAD_TRACE, "simulation %u stopped at event %llu", first + i,
                                       (unsigned long long)(dst[i].error - 1));
  return UNISON_OK;
}

int unison_counters_device(unison_ctx* ctx, const unison_counters** out) {
  if (!ctx || !out) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  *out = ctx->at<unison_counters>(ctx->L.counters);
  return UNISON_OK;
}

int unison_read_log(unison_ctx* ctx, uint32_t sim, unison_record* dst, uint32_t cap, uint64_t* n_total) {
  if (!ctx || !n_total || (!dst && cap)) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (sim >= ctx->dims.n_sims) return ctx->fail(UNISON_E_INVALID, "sim %u", sim);
  SimState st;
  int rc = ctx->hip(hipMemcpyAsync(&st, ctx->at<SimState>(ctx->L.state) + sim, sizeof st,
                                   hipMemcpyDeviceToHost, ctx->stream),
                    "copy state");
  if (rc) return rc;
  rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise state");
  if (rc) return rc;
  *n_total = st.log_len;
  const uint64_t kept = std::min<uint64_t>(st.log_len, ctx->dims.log_cap);
  const uint64_t n = std::min<uint64_t>(kept, cap);
  if (n) {
    rc = ctx->hip(hipMemcpyAsync(dst, ctx->at<unison_record>(ctx->L.log) + (size_t)sim * ctx->dims.log_cap,
                                 sizeof(unison_record) * n, hipMemcpyDeviceToHost, ctx->stream),
                  "copy log");
    if (rc) return rc;
    rc = ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise log");
  }
  return rc;
}

int unison_read_hazard(unison_ctx* ctx, uint32_t sim, uint32_t* d_out, uint32_t* n_out) {
  if (!ctx || !d_out || !n_out) return UNISON_E_INVALID;
  UNISON_LIVE(ctx);
  if (sim >= ctx->dims.n_sims) return ctx->fail(UNISON_E_INVALID, "sim %u", sim);
  if (!ctx->ran) return ctx->fail(UNISON_E_NOT_READY, "no run on this context yet");
  // an online table's counts are in the workspace; a fixed table's are its own
  const unison_sim_params& p = ctx->h_params[sim];
  const uint32_t* src_d = p.hazard_online ? ctx->at<uint32_t>(ctx->L.hcount) + (size_t)sim * 2 * kLut
                                          : ctx->at<uint32_t>(ctx->L.lut_d) + (size_t)p.lut * kLut;
  const uint32_t* src_n = p.hazard_online ? src_d + kLut
                                          : ctx->at<uint32_t>(ctx->L.lut_n) + (size_t)p.lut * kLut;
  int rc = ctx->hip(hipMemcpyAsync(d_out, src_d, sizeof(uint32_t) * kLut, hipMemcpyDeviceToHost,
                                   ctx->stream),
                    "copy hazard counts d");
  if (rc) return rc;
  rc = ctx->hip(hipMemcpyAsync(n_out, src_n, sizeof(uint32_t) * kLut, hipMemcpyDeviceToHost,
                               ctx->stream),
                "copy hazard counts n");
  if (rc) return rc;
  return ctx->hip(hipStreamSynchronize(ctx->stream), "synchronise hazard counts");
}

// Test hook: pin the simulation kernel variant (-1 = automatic).
int unison_debug_force_variant(unison_ctx* ctx, int variant) {
  if (!ctx) return UNISON_E_INVALID;
  ctx->force_variant = variant;
  return UNISON_OK;
}

// Test hook: cap the streamed tables' resident-cache slots (-1 = automatic).
int unison_debug_cache_slots(unison_ctx* ctx, int slots) {
  if (!ctx || slots < -1) return UNISON_E_INVALID;
  ctx->force_cache_slots = slots;
  return UNISON_OK;
}

// Test hook: the Kendall sort kernel's barrier plan (host only).
int unison_debug_kendall_barrier(uint32_t n_pad, uint32_t step, uint32_t a, uint32_t b) {
  const int r = kendall_barrier_after(n_pad, step, a, b);
  return r < 0 ? UNISON_E_INVALID : r;
}

int unison_ema_replay(void* hip_stream, uint32_t n, uint32_t max_hist, const uint64_t* gaps_ns,
                      const uint8_t* n_hist, uint32_t b_g, uint64_t tau_ns, float* g_out,
                      uint64_t* gq_out) {
  if (n && (!gaps_ns || !n_hist || !g_out || !gq_out)) return UNISON_E_INVALID;
  if (max_hist == 0 || b_g < 1 || b_g > 64 || tau_ns < 1) return UNISON_E_INVALID;
  return launch_ema_replay(n, max_hist, gaps_ns, n_hist, b_g, tau_ns, g_out, gq_out,
                           reinterpret_cast<hipStream_t>(hip_stream)) == hipSuccess
             ? UNISON_OK
             : UNISON_E_HIP;
}

int unison_score_fp32(void* hip_stream, uint32_t n, const uint8_t* turn, const float* g,
                      const uint8_t* done, const uint32_t* lut_d, const uint32_t* lut_n,
                      float penalty_us, float* out) {
  if (n && (!turn || !g || !done || !out)) return UNISON_E_INVALID;
  if (!lut_d || !lut_n || !(penalty_us >= 0.0f) || std::isinf(penalty_us)) return UNISON_E_INVALID;
  return launch_score_fp32(n, turn, g, done, lut_d, lut_n, penalty_us, out,
                           reinterpret_cast<hipStream_t>(hip_stream)) == hipSuccess
             ? UNISON_OK
             : UNISON_E_HIP;
}

int unison_score_fixed(void* hip_stream, uint32_t n, const uint8_t* turn, const uint64_t* gq,
                       const uint8_t* done, const uint32_t* lut_d, const uint32_t* lut_n,
                       uint32_t b_h, uint64_t p_z, uint32_t recip_bits, uint64_t* out) {
  if (n && (!turn || !gq || !done || !out)) return UNISON_E_INVALID;
  if (!lut_d || !lut_n || b_h < 6 || b_h > 16 || recip_bits > 32) return UNISON_E_INVALID;
  return launch_score_fixed(n, turn, gq, done, lut_d, lut_n, b_h, p_z, recip_bits, out,
                            reinterpret_cast<hipStream_t>(hip_stream)) == hipSuccess
             ? UNISON_OK
             : UNISON_E_HIP;
}

int unison_kendall(void* hip_stream, uint32_t n_snap, uint32_t n_per, uint64_t n_x, const float* x,
                   const uint64_t* y, const uint32_t* idx, uint64_t* counts, uint8_t* top1) {
  if (n_snap && (!x || !y || !counts || !top1)) return UNISON_E_INVALID;
  if (n_per < 2 || n_per > kendall_max_per()) return UNISON_E_INVALID;
  if (!idx && (uint64_t)n_snap * n_per > n_x) return UNISON_E_INVALID;
  return launch_kendall(n_snap, n_per, n_x, x, y, idx, counts, top1,
                        reinterpret_cast<hipStream_t>(hip_stream)) == hipSuccess
             ? UNISON_OK
             : UNISON_E_HIP;
}

}  // extern "C"
