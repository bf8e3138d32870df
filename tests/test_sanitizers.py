"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle: its C source, built with both sanitizers into a small driver,
  replays the tiny trace, the hand-worked TIDE and ETA traces and a batch of
  random traces under every policy (logs, per-event states, online tables,
  dual copies, both score forms and dividers), plus the scorers, the EMA
  replay, the ETA fit and the Kendall counts.
* The C ABI's host side: api.cpp compiled for the host only, with both
  sanitizers, against stand-ins for the HIP runtime calls it makes (copies
  become host copies, kernel launches do nothing), driven through every
  entry point with valid and invalid arguments, including traces that break
  the event format.

Any sanitizer report fails the test."""
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

import eta_cases
import tide_cases
from paper_2609_09643_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_C = os.path.join(ROOT, "oracle", "unison_oracle.c")
API_CPP = os.path.join(ROOT, "paper_2609_09643_amd", "csrc", "api.cpp")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g",
       "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")

# ------------------------------------------------------------------ oracle

ORACLE_DRIVER = r"""
#include "unison_oracle.c"
#include <stdio.h>

static void* slurp(FILE* f, size_t n) {
  void* p = malloc(n ? n : 1);
  if (n && fread(p, 1, n, f) != n) { fprintf(stderr, "short read\n"); exit(3); }
  return p;
}

int main(int argc, char** argv) {
  FILE* f = fopen(argv[1], "rb");
  uint64_t n_cases;
  if (fread(&n_cases, 8, 1, f) != 1) return 3;
  uint64_t sims = 0;
  for (uint64_t c = 0; c < n_cases; c++) {
    uint64_t hdr[3];  /* events, sessions, rows */
    if (fread(hdr, 8, 3, f) != 3) return 3;
    uint64_t ne = hdr[0], ns = hdr[1], nr = hdr[2];
    uint64_t* t = slurp(f, 8 * ne);
    uint32_t* sid = slurp(f, 4 * ne);
    uint32_t* info = slurp(f, 4 * ne);
    uint32_t* len = slurp(f, 4 * ne);
    uint64_t* nxt = slurp(f, 8 * ne);
    uint32_t* tool = slurp(f, 4 * ne);
    uint32_t* kvb = slurp(f, 4 * ns);
    uint32_t* turns = slurp(f, 4 * ns);
    orc_params* rows = slurp(f, sizeof(orc_params) * nr);
    uint32_t d[LUT_LEN], n[LUT_LEN], counts[2 * LUT_LEN];
    uint64_t eta[ETA_CLASSES];
    orc_hazard_counts(turns, (uint32_t)ns, d, n);
    orc_eta_fit(ne, t, info, tool, nxt, eta);
    for (uint64_t r = 0; r < nr; r++) {
      orc_counters out;
      uint32_t cap = 4096, log_len = 0;
      orc_rec* log = calloc(cap, sizeof(orc_rec));
      orc_state* st = calloc(ne ? ne : 1, sizeof(orc_state));
      uint64_t el = 0;
      int rc = orc_run(&rows[r], ne, t, sid, info, len, nxt, (uint32_t)ns, kvb, d, n, UINT64_MAX,
                       &out, log, cap, &log_len, st, counts, &el, tool, eta);
      if (rc != ORC_OK && rc != ORC_E_BAD_TRACE) { fprintf(stderr, "rc %d\n", rc); return 4; }
      rc = orc_run(&rows[r], ne, t, sid, info, len, nxt, (uint32_t)ns, kvb, d, n, ne / 2,
                   &out, NULL, 0, NULL, NULL, NULL, NULL, tool, eta);
      free(log);
      free(st);
      sims++;
    }
    /* the scorers, the EMA replay and Kendall on the trace's own sessions */
    uint32_t m = (uint32_t)(ns < 300 ? ns : 300);
    uint8_t* tu = calloc(m + 1, 1);
    uint8_t* dn = calloc(m + 1, 1);
    uint8_t* nh = calloc(m + 1, 1);
    uint64_t* gaps = calloc((size_t)(m + 1) * 4, 8);
    float* g = calloc(m + 1, 4);
    float* hf = calloc(LUT_LEN, 4);
    float* sf = calloc(m + 1, 4);
    uint64_t* gq = calloc(m + 1, 8);
    uint64_t* hq = calloc(LUT_LEN, 8);
    uint64_t* sq = calloc(m + 1, 8);
    for (uint32_t i = 0; i < m; i++) {
      tu[i] = (uint8_t)(turns[i] % 61);
      dn[i] = (uint8_t)(i % 17 == 0);
      nh[i] = (uint8_t)(i % 5);
      for (int k = 0; k < 4; k++) gaps[(size_t)i * 4 + k] = (uint64_t)(i + 1) * 1234567u * (k + 1);
    }
    orc_ema_replay(m, 4, gaps, nh, 32, 1000, g, gq);
    orc_lut_f32(d, n, hf);
    for (uint32_t bh = 6; bh <= 16; bh += 5) {
      orc_lut_q(d, n, bh, hq);
      for (uint32_t w = 0; w <= 32; w += 8)
        if (orc_score_fixed(m, tu, gq, dn, hq, bh, 500000000u, w, sq) != ORC_OK) return 5;
    }
    if (orc_score_fixed(m, tu, gq, dn, hq, 5, 1u, 0, sq) != ORC_E_INVALID) return 6;
    orc_score_f32(m, tu, g, dn, hf, 5e8f, sf);
    if (m >= 2) {
      uint64_t cnt[5 * 2];
      uint8_t top[2];
      uint32_t per = m / 2;
      orc_kendall(2, per, sf, sq, NULL, cnt, top);
    }
    free(tu); free(dn); free(nh); free(gaps); free(g); free(hf); free(sf); free(gq); free(hq); free(sq);
    free(t); free(sid); free(info); free(len); free(nxt); free(tool); free(kvb); free(turns); free(rows);
  }
  fclose(f);
  printf("ok %llu\n", (unsigned long long)sims);
  return 0;
}
"""


def _rows(rng, n_rows):
    """Parameter rows in the oracle's layout, over every policy and option."""
    import oracle
    out = []
    formats = synth.format_grid_dividers()
    for _ in range(n_rows):
        p = synth.default_params(1)
        pol = int(rng.integers(0, 5))
        synth.set_policy(p, pol, tide=int(rng.integers(0, 2)))
        if pol == synth.POLICY_SPEAR and rng.random() < 0.5:
            bh, bg, tau, wb = formats[int(rng.integers(len(formats)))]
            p["score_mode"], p["b_h"], p["b_g"], p["tau_ns"], p["recip_bits"] = 1, bh, bg, tau, wb
        p["cap_sram_B"] = int(rng.choice([0, 1, 64])) * synth.MIB
        p["cap_hbm_B"] = int(rng.choice([0, 1, 16])) * synth.GIB
        p["n_slots"] = int(rng.choice([1, 3, 64]))
        p["ttl_ns"] = int(rng.choice([1, 2000, 30_000])) * 1_000_000
        p["dma_B_per_us"] = int(rng.choice([1, 100_000]))
        p["dual_sync"] = int(rng.integers(0, 4)) if rng.random() < 0.3 else 0
        if rng.random() < 0.25:
            p["hazard_online"], p["online_sessions"] = 1, int(rng.choice([0, 3, 0xFFFFFFFF]))
        out.append(bytes(oracle.params_struct(p[0])))
    return out


def _write_cases(path):
    rng = np.random.Generator(np.random.PCG64(99))
    cases = [(synth.c1_tiny().traces[0], 8)]
    for build in list(tide_cases.CASES.values()):
        cases.append((build()[0], 4))
    cases.append((eta_cases.predicted_and_true_returns_disagree()[0], 4))
    for _ in range(6):
        n = int(rng.integers(1, 60))
        tr = synth.build_trace(rng, rng.geometric(0.35, n).clip(max=6),
                               synth.poisson_arrivals(rng, n, 5.0), synth.gaps_mixture,
                               rng.choice(np.array([1, 64, 160]) * 1024, n))
        cases.append((tr, 10))
    bad = synth.tiny_trace(3, n_sessions=5, turns=3)
    bad.info = bad.info.copy()
    bad.info[7] = (2 << 24) | 0                               # an end without its arrival
    cases.append((bad, 3))
    with open(path, "wb") as f:
        np.array([len(cases)], np.uint64).tofile(f)
        for tr, n_rows in cases:
            np.array([tr.n_events, tr.n_sessions, n_rows], np.uint64).tofile(f)
            for a, dt in ((tr.t_ns, np.uint64), (tr.sid, np.uint32), (tr.info, np.uint32),
                          (tr.length, np.uint32), (tr.next_ns, np.uint64), (tr.tool, np.uint32),
                          (tr.kvb, np.uint32), (tr.turns, np.uint32)):
                np.ascontiguousarray(a, dtype=dt).tofile(f)
            for r in _rows(rng, n_rows):
                f.write(r)
    return sum(n for _, n in cases)


def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("no gcc")
    drv = tmp_path / "drv.c"
    drv.write_text(ORACLE_DRIVER)
    exe = tmp_path / "drv"
    subprocess.check_call(["gcc", "-std=gnu11", "-ffp-contract=off", "-I", os.path.dirname(ORACLE_C)]
                          + SAN + [str(drv), "-o", str(exe), "-lm"])
    data = tmp_path / "cases.bin"
    n_rows = _write_cases(str(data))
    r = subprocess.run([str(exe), str(data)], capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0 and "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, \
        r.stderr[-3000:]
    assert r.stdout.strip() == "ok %d" % n_rows


# ------------------------------------------------------- C ABI host side

HIP_STANDINS = r"""
// Stand-ins for the HIP runtime and the kernel launchers: "device" memory is
// host memory, copies are memcpy, launches do nothing.
#include <hip/hip_runtime.h>
#include <cstring>
#include "unison_device.h"

extern "C" {
void** __hipRegisterFatBinary(void*) { static void* h = nullptr; return &h; }
void __hipUnregisterFatBinary(void**) {}
void __hipRegisterVar(void**, char*, char*, const char*, int, size_t, int, int) {}
hipError_t hipGetDevice(int*) { return hipErrorNoDevice; }
const char* hipGetErrorString(hipError_t) { return "stand-in"; }
hipError_t hipGetSymbolAddress(void**, const void*) { return hipErrorNoDevice; }
hipError_t hipMemcpyAsync(void* d, const void* s, size_t n, hipMemcpyKind, hipStream_t) {
  std::memmove(d, s, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
FATBIN_DEFINITION
}

namespace unison {
hipError_t launch_sim(const SimArgs&, uint32_t, uint64_t, hipStream_t, int, int) { return hipSuccess; }
uint32_t sim_variant_capacity(int v) { return v >= 0 && v <= 14 && v != 6 ? (1u << 20) : 0u; }
int sim_auto_variant(uint32_t n, uint64_t) { return n <= 16 ? 5 : 10; }
uint64_t sim_variant_max_slots(int v) { return v == 13 ? 512u : v == 14 ? 4096u : (1u << 20); }
bool sim_variant_slots_ok(int v, uint64_t s) { return s <= sim_variant_max_slots(v); }
uint32_t sim_variant_lanes(int v) { return v == 5 ? 8u : 0u; }
hipError_t launch_hazard_counts(const uint32_t*, uint32_t, uint32_t*, uint32_t*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_eta_fit(uint64_t, const uint64_t*, const uint32_t*, const uint32_t*,
                          const uint64_t*, uint64_t*, hipStream_t) { return hipSuccess; }
hipError_t launch_max_time(const uint64_t* t, const uint64_t* next, uint64_t n, uint64_t* out,
                           hipStream_t) {
  uint64_t m = 0;
  for (uint64_t i = 0; i < n; ++i) {
    m = t[i] > m ? t[i] : m;
    m = (next[i] != ~0ull && next[i] > m) ? next[i] : m;
  }
  *out = m;
  return hipSuccess;
}
hipError_t launch_ema_replay(uint32_t, uint32_t, const uint64_t*, const uint8_t*, uint32_t, uint64_t,
                             float*, uint64_t*, hipStream_t) { return hipSuccess; }
hipError_t launch_score_fp32(uint32_t, const uint8_t*, const float*, const uint8_t*, const uint32_t*,
                             const uint32_t*, float, float*, hipStream_t) { return hipSuccess; }
hipError_t launch_score_fixed(uint32_t, const uint8_t*, const uint64_t*, const uint8_t*,
                              const uint32_t*, const uint32_t*, uint32_t, uint64_t, uint32_t,
                              uint64_t*, hipStream_t) { return hipSuccess; }
hipError_t launch_kendall(uint32_t, uint32_t, uint64_t, const float*, const uint64_t*, const uint32_t*,
                          uint64_t*, uint8_t*, hipStream_t) { return hipSuccess; }
uint32_t kendall_max_per() { return 4096; }
int kendall_barrier_after(uint32_t P, uint32_t step, uint32_t, uint32_t) {
  return P >= 256 && P <= 4096 && step <= 1 ? 1 : -1;
}
}  // namespace unison
"""

API_DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>
#include "unison.h"

#define CHECK(x) do { if (!(x)) { std::fprintf(stderr, "failed: %s (line %d)\n", #x, __LINE__); return 1; } } while (0)

struct Trace {
  std::vector<uint64_t> t, next;
  std::vector<uint32_t> sid, info, len, tool;
  void ev(uint64_t tt, uint32_t s, uint32_t kind, uint32_t turn, uint32_t l, uint32_t tl = 0) {
    t.push_back(tt); sid.push_back(s); info.push_back(kind << 24 | turn); len.push_back(l);
    next.push_back(~0ull); tool.push_back(tl);
  }
};

int main() {
  unison_dims d = {6, 3, 4, 2, 64, 1};
  size_t bytes = 0;
  CHECK(unison_workspace_size(&d, &bytes) == UNISON_OK && bytes > 0);
  unison_dims bad = d;
  bad.max_sessions = (1u << 20) + 1;
  CHECK(unison_workspace_size(&bad, &bytes) == UNISON_E_INVALID);
  bad = d; bad.n_sims = 0;
  CHECK(unison_workspace_size(&bad, &bytes) == UNISON_E_INVALID);
  CHECK(unison_workspace_size(&d, &bytes) == UNISON_OK);
  void* ws = std::aligned_alloc(256, (bytes + 255) / 256 * 256);
  std::memset(ws, 0, bytes);
  unison_ctx* ctx = nullptr;
  CHECK(unison_create(&ctx, &d, nullptr, (char*)ws + 1, bytes) == UNISON_E_INVALID);
  CHECK(unison_create(&ctx, &d, nullptr, ws, bytes - 1) == UNISON_E_INVALID);
  CHECK(unison_create(&ctx, &d, nullptr, ws, bytes) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, 0, 10) == UNISON_E_NOT_READY);
  unison_sim_params rows[6];
  std::memset(rows, 0, sizeof rows);
  CHECK(unison_set_params(ctx, rows) == UNISON_E_NOT_READY);

  // three traces: a good one, one whose fourth event ends a turn that never
  // began, one whose gap onset names tool class 16
  Trace a, b, c;
  a.ev(10, 0, 0, 0, 3); a.ev(20, 0, 1, 0, 0, 2); a.ev(30, 1, 0, 0, 4); a.ev(40, 1, 1, 0, 0, 1);
  a.ev(50, 0, 0, 1, 5); a.ev(60, 0, 2, 1, 0); a.ev(70, 1, 0, 1, 6); a.ev(80, 1, 2, 1, 0);
  a.next[1] = 50; a.next[3] = 70;
  b.ev(10, 0, 0, 0, 3); b.ev(20, 0, 1, 0, 0); b.ev(30, 1, 0, 0, 4); b.ev(40, 2, 1, 0, 0);
  c.ev(10, 0, 0, 0, 3); c.ev(20, 0, 1, 0, 0, 16); c.ev(30, 0, 0, 1, 4); c.ev(40, 0, 2, 1, 0);
  Trace all;
  std::vector<uint64_t> ev_off = {0}, ss_off = {0, 2, 5, 6};
  for (Trace* x : {&a, &b, &c}) {
    for (size_t i = 0; i < x->t.size(); ++i) {
      all.t.push_back(x->t[i]); all.sid.push_back(x->sid[i]); all.info.push_back(x->info[i]);
      all.len.push_back(x->len[i]); all.next.push_back(x->next[i]); all.tool.push_back(x->tool[i]);
    }
    ev_off.push_back(all.t.size());
  }
  std::vector<uint32_t> kvb(6, 1024);
  unison_trace_batch tb;
  std::memset(&tb, 0, sizeof tb);
  tb.n_traces = 3;
  tb.ev_offset = ev_off.data();
  tb.sess_offset = ss_off.data();
  CHECK(unison_load_traces(ctx, &tb) == UNISON_E_INVALID);      // null arrays
  tb.ev_t_ns = all.t.data(); tb.ev_sid = all.sid.data(); tb.ev_info = all.info.data();
  tb.ev_len = all.len.data(); tb.ev_next_ns = all.next.data(); tb.sess_kvb = kvb.data();
  tb.ev_tool = all.tool.data();
  tb.n_traces = 2;
  CHECK(unison_load_traces(ctx, &tb) == UNISON_E_INVALID);      // count differs from the dims
  tb.n_traces = 3;
  std::vector<uint64_t> big = ss_off;
  big[3] = 100;
  tb.sess_offset = big.data();
  CHECK(unison_load_traces(ctx, &tb) == UNISON_E_CAPACITY);
  tb.sess_offset = ss_off.data();
  CHECK(unison_load_traces(ctx, &tb) == UNISON_OK);
  tb.ev_tool = nullptr;
  CHECK(unison_load_traces(ctx, &tb) == UNISON_OK);
  tb.ev_tool = all.tool.data();
  CHECK(unison_load_traces(ctx, &tb) == UNISON_OK);

  uint32_t hd[51] = {0}, hn[51];
  for (int i = 0; i < 51; ++i) hn[i] = 1;
  CHECK(unison_set_hazard(ctx, 2, hd, hn) == UNISON_E_INVALID);
  CHECK(unison_set_hazard(ctx, 0, hd, hn) == UNISON_OK);
  CHECK(unison_set_hazard(ctx, 1, hd, hn) == UNISON_OK);
  uint64_t eta[16] = {5, 6, 7};
  CHECK(unison_set_eta(ctx, 3, eta) == UNISON_E_INVALID);
  for (uint32_t i = 0; i < 3; ++i) CHECK(unison_set_eta(ctx, i, eta) == UNISON_OK);
  for (int i = 0; i < 6; ++i) {
    rows[i].policy = (uint32_t)(i % 5); rows[i].tide = 1; rows[i].lut = (uint32_t)(i % 2);
    rows[i].trace = (uint32_t)(i % 3); rows[i].cap_sram_B = 4096; rows[i].cap_hbm_B = 1 << 20;
    rows[i].n_slots = 4; rows[i].dma_B_per_us = 1000; rows[i].ttl_ns = 100;
    rows[i].t_s_ns_per_B = 1e-4; rows[i].t_h_ns_per_B = 1e-3; rows[i].t_p_ns_per_tok = 5e4;
    rows[i].penalty_us = 5e8f; rows[i].b_h = 12; rows[i].b_g = 32; rows[i].tau_ns = 1000;
    rows[i].p_z = 500000000; rows[i].online_sessions = 3;
  }
  rows[5].score_mode = 1; rows[5].policy = 0; rows[5].recip_bits = 16; rows[4].dual_sync = 2;
  rows[3].hazard_online = 1;
  unison_sim_params keep = rows[2];
  rows[2].recip_bits = 33;
  CHECK(unison_set_params(ctx, rows) == UNISON_E_INVALID);
  rows[2] = keep; rows[2].policy = 5;
  CHECK(unison_set_params(ctx, rows) == UNISON_E_INVALID);
  rows[2] = keep; rows[2].penalty_us = -1.0f;
  CHECK(unison_set_params(ctx, rows) == UNISON_E_INVALID);
  rows[2] = keep;
  CHECK(unison_set_params(ctx, rows) == UNISON_OK);
  CHECK(unison_run(ctx, 9, 0, 10) == UNISON_E_INVALID);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, 64, 10) == UNISON_E_INVALID);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, UNISON_RUN_CONTINUE, 10) == UNISON_E_NOT_READY);
  CHECK(unison_debug_force_variant(ctx, 3) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, 0, 10) == UNISON_E_INVALID);  // dual rows need 11
  CHECK(unison_debug_force_variant(ctx, -1) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, UNISON_RUN_LOG | UNISON_RUN_LOG_VICTIM, ~0ull) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, UNISON_RUN_CONTINUE, 5) == UNISON_OK);
  rows[4].dual_sync = 0;
  CHECK(unison_set_params(ctx, rows) == UNISON_OK);
  for (uint32_t pol = 0; pol <= 4; ++pol) CHECK(unison_run(ctx, pol, 0, ~0ull) == UNISON_OK);
  CHECK(unison_debug_force_variant(ctx, 5) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, 0, ~0ull) == UNISON_OK);
  CHECK(unison_debug_force_variant(ctx, 6) == UNISON_OK);
  CHECK(unison_run(ctx, UNISON_POLICY_PARAMS, 0, ~0ull) == UNISON_E_CAPACITY);
  unison_counters cnt[6];
  CHECK(unison_read_counters(ctx, cnt, 4, 3) == UNISON_E_INVALID);
  CHECK(unison_read_counters(ctx, cnt, 0, 6) == UNISON_OK);
  const unison_counters* dev = nullptr;
  CHECK(unison_counters_device(ctx, &dev) == UNISON_OK && dev != nullptr);
  unison_record rec[64];
  uint64_t n_total = 0;
  CHECK(unison_read_log(ctx, 6, rec, 64, &n_total) == UNISON_E_INVALID);
  CHECK(unison_read_log(ctx, 1, rec, 64, &n_total) == UNISON_OK);
  uint32_t od[51], on[51];
  CHECK(unison_read_hazard(ctx, 3, od, on) == UNISON_OK);
  CHECK(unison_read_hazard(ctx, 0, od, on) == UNISON_OK);
  CHECK(unison_read_hazard(ctx, 9, od, on) == UNISON_E_INVALID);
  CHECK(unison_debug_cache_slots(ctx, -2) == UNISON_E_INVALID);
  CHECK(unison_set_stream(ctx, nullptr) == UNISON_OK);
  CHECK(unison_last_error(ctx) != nullptr);
  unison_destroy(ctx);

  // the allocation-free entry point finds no device here
  unison_ctx* st = nullptr;
  CHECK(unison_create_static(&st, &d, nullptr) == UNISON_E_HIP && st == nullptr);
  CHECK(std::strlen(unison_last_error(nullptr)) > 0);
  unison_dims huge = {1u << 20, 1, 1u << 20, 1, 0, 0};
  CHECK(unison_create_static(&st, &huge, nullptr) == UNISON_E_CAPACITY);

  // context-free entry points: argument checks and the barrier plan
  CHECK(unison_kendall(nullptr, 1, 1, 1, (float*)8, (uint64_t*)8, nullptr, (uint64_t*)8, (uint8_t*)8) ==
        UNISON_E_INVALID);
  CHECK(unison_score_fixed(nullptr, 1, (uint8_t*)8, (uint64_t*)8, (uint8_t*)8, hd, hn, 12, 0, 33,
                           (uint64_t*)8) == UNISON_E_INVALID);
  CHECK(unison_eta_fit(nullptr, 4, nullptr, nullptr, nullptr, nullptr, eta) == UNISON_E_INVALID);
  CHECK(unison_ema_replay(nullptr, 1, 0, (uint64_t*)8, (uint8_t*)8, 32, 1000, (float*)8, (uint64_t*)8) ==
        UNISON_E_INVALID);
  for (uint32_t P = 128; P <= 8192; P *= 2)
    for (uint32_t s = 0; s < 3; ++s) unison_debug_kendall_barrier(P, s, 8, 2);
  for (int code = 1; code >= -6; --code) CHECK(unison_strerror(code) != nullptr);
  std::free(ws);
  std::printf("ok\n");
  return 0;
}
"""


def test_api_host_side_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("no hipcc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.dirname(API_CPP)]
    host = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "--offload-host-only", "-std=c++17",
            "-fPIC"] + SAN
    api_o = tmp_path / "api.o"
    subprocess.check_call(host + inc + ["-c", API_CPP, "-o", str(api_o)],
                          stderr=subprocess.DEVNULL)
    syms = subprocess.run(["nm", "-u", str(api_o)], capture_output=True, text=True).stdout.split()
    fat = [s for s in syms if s.startswith("__hip_fatbin")]
    stand = tmp_path / "standins.cpp"
    stand.write_text(HIP_STANDINS.replace(
        "FATBIN_DEFINITION", "".join("char %s[16];\n" % s for s in fat)))
    stand_o = tmp_path / "standins.o"
    subprocess.check_call(host + inc + ["-c", str(stand), "-o", str(stand_o)],
                          stderr=subprocess.DEVNULL)
    drv = tmp_path / "drv.cpp"
    drv.write_text(API_DRIVER)
    exe = tmp_path / "drv"
    subprocess.check_call(["g++", "-std=c++17"] + SAN + inc +
                          [str(drv), str(api_o), str(stand_o), "-o", str(exe), "-lpthread"])
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0 and "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, \
        (r.stdout + r.stderr)[-3000:]
    assert r.stdout.strip() == "ok"
