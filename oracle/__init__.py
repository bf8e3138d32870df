"""TEST INFRASTRUCTURE -- the CPU oracle for the UNISON residency policy.

A ctypes wrapper over ``liboracle.so`` (built from ``unison_oracle.c`` with
gcc, no vectorisation, no FMA contraction).  Only ``tests/``, the package
smoke check and the benchmark's ``cpu_baseline`` leg may import this module;
the product path never does, and this module imports nothing from the
product package.

Inputs are duck-typed: a trace is any object with ``t_ns, sid, info, length,
next_ns, kvb`` numpy arrays (and optionally ``tool``, the tool class of each
gap onset); a parameter row is any numpy structured row with the field names
used below.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "unison_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

LUT_LEN = 51
ETA_CLASSES = 16
NONE_ID = 0xFFFFFFFF
OP_EVICT, OP_EXPIRE, OP_BYPASS, OP_PROMOTE, OP_SWAP, OP_VICTIM, OP_PLACE = 1, 2, 3, 4, 5, 6, 7
TIER_NONE, TIER_SRAM, TIER_HBM = 0, 1, 2


def build(force: bool = True) -> str:
    """Compiles liboracle.so in place."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=gnu11", "-Wall", "-ffp-contract=off", "-fno-fast-math",
               "-shared", "-fPIC", _SRC, "-o", _LIB + ".tmp", "-lm"]
        subprocess.check_call(cmd)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class Params(C.Structure):
    _fields_ = [
        ("policy", C.c_uint32), ("tide", C.c_uint32), ("score_mode", C.c_uint32),
        ("lut", C.c_uint32), ("cap_sram_B", C.c_uint64), ("cap_hbm_B", C.c_uint64),
        ("n_slots", C.c_uint64), ("dma_B_per_us", C.c_uint64), ("ttl_ns", C.c_uint64),
        ("t_s_ns_per_B", C.c_double), ("t_h_ns_per_B", C.c_double),
        ("t_p_ns_per_tok", C.c_double), ("penalty_us", C.c_float), ("b_h", C.c_uint32),
        ("b_g", C.c_uint32), ("hazard_online", C.c_uint32), ("online_sessions", C.c_uint32),
        ("pad0", C.c_uint32), ("tau_ns", C.c_uint64), ("p_z", C.c_uint64),
        ("dual_sync", C.c_uint32), ("recip_bits", C.c_uint32),
    ]


COUNTER_NAMES = (
    "requests", "hit_sram", "hit_hbm", "miss", "bypass", "evict", "expire", "promote", "swap",
    "dma_bytes", "tide_passes", "tokens_total", "tokens_computed", "extra_prefill_tok",
    "score_evals", "resident_evals", "digest", "victim_digest", "events", "error",
    "prefetch_hits", "vict_diff", "prom_diff",
)


class Counters(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in COUNTER_NAMES] + [
        ("amat_sum_ns", C.c_double), ("ttft_sum_ns", C.c_double)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


REC_DTYPE = np.dtype([("ev", np.uint32), ("op", np.uint32), ("a", np.uint32), ("b", np.uint32)])
STATE_DTYPE = np.dtype([
    ("used_sram", np.uint64), ("used_hbm", np.uint64), ("n_res", np.uint32),
    ("n_table", np.uint32), ("victim", np.uint32), ("tide_ran", np.uint32),
    ("tide_budget", np.uint64), ("tide_moved", np.uint64)])


def _p(a, ctype):
    return a.ctypes.data_as(C.POINTER(ctype)) if a is not None else None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = load_library(_LIB)
    return _lib


def compile_source(src_text, out_path):
    """Compiles oracle C source text (the oracle's own, or a test's altered
    copy of it) into a shared library at out_path, with the oracle's flags."""
    c_path = out_path + ".c"
    with open(c_path, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
                           "-shared", "-fPIC", c_path, "-o", out_path, "-lm"])
    return out_path


def source_text():
    with open(_SRC) as f:
        return f.read()


def load_library(path):
    """Loads a library built from the oracle source and declares its entry
    points."""
    L = C.CDLL(path)
    u32p, u64p, f32p, u8p = (C.POINTER(C.c_uint32), C.POINTER(C.c_uint64),
                             C.POINTER(C.c_float), C.POINTER(C.c_uint8))
    L.orc_run.restype = C.c_int
    L.orc_run.argtypes = [C.POINTER(Params), C.c_uint64, u64p, u32p, u32p, u32p, u64p,
                          C.c_uint32, u32p, u32p, u32p, C.c_uint64, C.POINTER(Counters),
                          C.c_void_p, C.c_uint32, u32p, C.c_void_p, C.c_void_p, u64p,
                          u32p, u64p]
    L.orc_eta_fit.argtypes = [C.c_uint64, u64p, u32p, u32p, u64p, u64p]
    L.orc_hazard_counts.argtypes = [u32p, C.c_uint32, u32p, u32p]
    L.orc_lut_f32.argtypes = [u32p, u32p, f32p]
    L.orc_lut_q.argtypes = [u32p, u32p, C.c_uint32, u64p]
    L.orc_score_f32.argtypes = [C.c_uint32, u8p, f32p, u8p, f32p, C.c_float, f32p]
    L.orc_score_fixed.restype = C.c_int
    L.orc_score_fixed.argtypes = [C.c_uint32, u8p, u64p, u8p, u64p, C.c_uint32,
                                  C.c_uint64, C.c_uint32, u64p]
    L.orc_ema_replay.argtypes = [C.c_uint32, C.c_uint32, u64p, u8p, C.c_uint32,
                                 C.c_uint64, f32p, u64p]
    L.orc_kendall.argtypes = [C.c_uint32, C.c_uint32, f32p, u64p, u32p, u64p, u8p]
    L.orc_run_batch.restype = C.c_int
    L.orc_run_batch.argtypes = [C.c_void_p, C.c_uint32, u32p, u32p, u64p, u64p, u64p, u32p,
                                u32p, u32p, u64p, u32p, u32p, u32p, C.c_uint64, C.c_void_p,
                                u64p, u32p, u64p]
    return L


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ hazard

def hazard_counts(turns):
    """eq. (hazard) counts d(t), n(t), t = 0..50, from a turn-count population."""
    T = _c(turns, np.uint32)
    d = np.zeros(LUT_LEN, np.uint32)
    n = np.zeros(LUT_LEN, np.uint32)
    lib().orc_hazard_counts(_p(T, C.c_uint32), T.shape[0], _p(d, C.c_uint32), _p(n, C.c_uint32))
    return d, n


def lut_f32(d, n):
    d, n = _c(d, np.uint32), _c(n, np.uint32)
    out = np.zeros(LUT_LEN, np.float32)
    lib().orc_lut_f32(_p(d, C.c_uint32), _p(n, C.c_uint32), _p(out, C.c_float))
    return out


def lut_q(d, n, b_h):
    d, n = _c(d, np.uint32), _c(n, np.uint32)
    out = np.zeros(LUT_LEN, np.uint64)
    lib().orc_lut_q(_p(d, C.c_uint32), _p(n, C.c_uint32), b_h, _p(out, C.c_uint64))
    return out


def luts_for(workload):
    """Hazard counts (d, n) [n_luts, 51] for every table of a workload."""
    n_l = len(workload.lut_pops)
    D = np.zeros((n_l, LUT_LEN), np.uint32)
    N = np.zeros((n_l, LUT_LEN), np.uint32)
    for i, pop in enumerate(workload.lut_pops):
        if pop is not None:
            D[i], N[i] = hazard_counts(pop)
    for (i, d, n) in getattr(workload, "flat_luts", []):
        D[i], N[i] = d, n
    return D, N


# ------------------------------------------------------------------ scores

def score_f32(turn, g, done, d, n, penalty):
    turn, g, done = _c(turn, np.uint8), _c(g, np.float32), _c(done, np.uint8)
    hf = lut_f32(d, n)
    out = np.zeros(turn.shape[0], np.float32)
    lib().orc_score_f32(turn.shape[0], _p(turn, C.c_uint8), _p(g, C.c_float),
                        _p(done, C.c_uint8), _p(hf, C.c_float), C.c_float(penalty),
                        _p(out, C.c_float))
    return out


def score_fixed(turn, gq, done, d, n, b_h, p_z, recip_bits=0):
    """Fixed-point scores; recip_bits 0: exact divider in eq. (t1), else a
    reciprocal table with that many fraction bits."""
    turn, gq, done = _c(turn, np.uint8), _c(gq, np.uint64), _c(done, np.uint8)
    hq = lut_q(d, n, b_h)
    out = np.zeros(turn.shape[0], np.uint64)
    rc = lib().orc_score_fixed(turn.shape[0], _p(turn, C.c_uint8), _p(gq, C.c_uint64),
                               _p(done, C.c_uint8), _p(hq, C.c_uint64), b_h, p_z, recip_bits,
                               _p(out, C.c_uint64))
    if rc != 0:
        raise ValueError("b_h %d or recip_bits %d out of range" % (b_h, recip_bits))
    return out


def ema_replay(gaps_ns, n_hist, b_g=32, tau_ns=1000):
    gaps = _c(gaps_ns, np.uint64)
    nh = _c(n_hist, np.uint8)
    n, mh = gaps.shape
    g = np.zeros(n, np.float32)
    gq = np.zeros(n, np.uint64)
    lib().orc_ema_replay(n, mh, _p(gaps, C.c_uint64), _p(nh, C.c_uint8), b_g, tau_ns,
                         _p(g, C.c_float), _p(gq, C.c_uint64))
    return g, gq


def kendall(x, y, idx=None, n_per=None):
    """Per-snapshot pair counts (C, D, ties x only, ties y only, ties both)
    and top-1 agreement.  With idx [n_snap, n_per] the snapshot entries are
    gathered from x and y; otherwise x and y are [n_snap, n_per]."""
    x = _c(x, np.float32)
    y = _c(y, np.uint64)
    if idx is not None:
        idx = _c(idx, np.uint32)
        n_snap, n_per = idx.shape
    else:
        n_snap, n_per = x.shape
    counts = np.zeros((n_snap, 5), np.uint64)
    top1 = np.zeros(n_snap, np.uint8)
    lib().orc_kendall(n_snap, n_per, _p(x, C.c_float), _p(y, C.c_uint64),
                      _p(idx, C.c_uint32) if idx is not None else None,
                      _p(counts, C.c_uint64), _p(top1, C.c_uint8))
    return counts, top1


def tau_b(counts):
    c, d, tx, ty, _ = [counts[..., i].astype(np.float64) for i in range(5)]
    den = np.sqrt((c + d + tx) * (c + d + ty))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(den > 0, (c - d) / den, np.nan)


# -------------------------------------------------------------- simulation

def _tool(trace):
    t = getattr(trace, "tool", None)
    return _c(t if t is not None else np.zeros(trace.t_ns.shape[0], np.uint32), np.uint32)


def eta_table(trace):
    """The ETA table fitted on a trace: mean wait (ns) per tool class."""
    t, info = _c(trace.t_ns, np.uint64), _c(trace.info, np.uint32)
    nxt, tool = _c(trace.next_ns, np.uint64), _tool(trace)
    out = np.zeros(ETA_CLASSES, np.uint64)
    lib().orc_eta_fit(t.shape[0], _p(t, C.c_uint64), _p(info, C.c_uint32), _p(tool, C.c_uint32),
                      _p(nxt, C.c_uint64), _p(out, C.c_uint64))
    return out


def params_struct(row):
    p = Params()
    for name, _ in Params._fields_:
        if name.startswith("pad"):
            continue
        v = row[name] if name in row.dtype.names else 0
        setattr(p, name, float(v) if name.startswith("t_") or name == "penalty_us" else int(v))
    return p


def run(trace, row, lut_d, lut_n, max_events=None, log_cap=0, states=False, counts=None,
        library=None, eta=None):
    """Runs one simulation. Returns (rc, counters dict, log or None, states or None,
    elapsed_ns of the event loop).  counts: optional uint32 array [2, 51] that
    receives the hazard counts d, n of the table at the end.  library: a
    library from load_library() to run instead of the oracle's own build.
    eta: the ETA table (default: fitted on the trace)."""
    L = lib() if library is None else library
    tool = _tool(trace)
    eta = _c(eta_table(trace) if eta is None else eta, np.uint64)
    p = params_struct(row)
    t_ns, sid = _c(trace.t_ns, np.uint64), _c(trace.sid, np.uint32)
    info, length = _c(trace.info, np.uint32), _c(trace.length, np.uint32)
    nxt, kvb = _c(trace.next_ns, np.uint64), _c(trace.kvb, np.uint32)
    d, n = _c(lut_d, np.uint32), _c(lut_n, np.uint32)
    n_ev = t_ns.shape[0]
    me = 0xFFFFFFFFFFFFFFFF if max_events is None else int(max_events)
    cnt = Counters()
    log = np.zeros(log_cap, REC_DTYPE) if log_cap else None
    log_len = np.zeros(1, np.uint32)
    n_st = min(n_ev, me)
    st = np.zeros(n_st, STATE_DTYPE) if states else None
    el = np.zeros(1, np.uint64)
    rc = L.orc_run(C.byref(p), n_ev, _p(t_ns, C.c_uint64), _p(sid, C.c_uint32),
                   _p(info, C.c_uint32), _p(length, C.c_uint32), _p(nxt, C.c_uint64),
                   kvb.shape[0], _p(kvb, C.c_uint32), _p(d, C.c_uint32), _p(n, C.c_uint32),
                   me, C.byref(cnt),
                   log.ctypes.data_as(C.c_void_p) if log is not None else None, log_cap,
                   _p(log_len, C.c_uint32),
                   st.ctypes.data_as(C.c_void_p) if st is not None else None,
                   counts.ctypes.data_as(C.c_void_p) if counts is not None else None,
                   _p(el, C.c_uint64), _p(tool, C.c_uint32), _p(eta, C.c_uint64))
    if log is not None:
        log = log[:min(int(log_len[0]), log_cap)]
        if int(log_len[0]) > log_cap:
            raise RuntimeError("oracle decision log overflow: %d > %d" % (log_len[0], log_cap))
    return rc, cnt.as_dict(), log, st, int(el[0])


class Batch:
    """A workload's traces, hazard counts and parameter rows marshalled once
    for orc_run_batch."""

    def __init__(self, workload):
        trs = workload.traces
        self.ev_off = np.zeros(len(trs) + 1, np.uint64)
        self.ss_off = np.zeros(len(trs) + 1, np.uint64)
        self.ev_off[1:] = np.cumsum([t.n_events for t in trs])
        self.ss_off[1:] = np.cumsum([t.n_sessions for t in trs])
        cat = lambda name, dt: np.ascontiguousarray(
            np.concatenate([getattr(t, name) for t in trs] + [np.zeros(1, dt)]), dtype=dt)
        self.t, self.sid = cat("t_ns", np.uint64), cat("sid", np.uint32)
        self.info, self.len = cat("info", np.uint32), cat("length", np.uint32)
        self.next, self.kvb = cat("next_ns", np.uint64), cat("kvb", np.uint32)
        self.tool = np.ascontiguousarray(np.concatenate([_tool(t) for t in trs] +
                                                        [np.zeros(1, np.uint32)]))
        self.eta = np.ascontiguousarray(np.stack([eta_table(t) for t in trs]), dtype=np.uint64)
        D, N = luts_for(workload)
        self.D, self.N = np.ascontiguousarray(D), np.ascontiguousarray(N)
        self.params = workload.params

    def prepare(self, sims):
        """The parameter rows of `sims` in the oracle's layout, to run more
        than once."""
        sims = list(sims)
        rows = (Params * max(len(sims), 1))()
        for k, i in enumerate(sims):
            rows[k] = params_struct(self.params[i])
        tr_idx = np.ascontiguousarray(self.params["trace"][sims], dtype=np.uint32)
        lut_idx = np.ascontiguousarray(self.params["lut"][sims], dtype=np.uint32)
        return sims, rows, tr_idx, lut_idx

    def run(self, sims, max_events=None):
        """Runs `sims` (a list, or what prepare() returned); returns (rc,
        counter dicts, summed event-loop ns)."""
        sims, rows, tr_idx, lut_idx = sims if isinstance(sims, tuple) else self.prepare(sims)
        n = len(sims)
        cnt = (Counters * max(n, 1))()
        el = np.zeros(1, np.uint64)
        me = 0xFFFFFFFFFFFFFFFF if max_events is None else int(max_events)
        rc = lib().orc_run_batch(
            C.cast(rows, C.c_void_p), n, _p(tr_idx, C.c_uint32), _p(lut_idx, C.c_uint32),
            _p(self.ev_off, C.c_uint64), _p(self.ss_off, C.c_uint64), _p(self.t, C.c_uint64),
            _p(self.sid, C.c_uint32), _p(self.info, C.c_uint32), _p(self.len, C.c_uint32),
            _p(self.next, C.c_uint64), _p(self.kvb, C.c_uint32), _p(self.D, C.c_uint32),
            _p(self.N, C.c_uint32), me, C.cast(cnt, C.c_void_p), _p(el, C.c_uint64),
            _p(self.tool, C.c_uint32), _p(self.eta, C.c_uint64))
        return rc, [cnt[k].as_dict() for k in range(n)], int(el[0])


def run_workload(workload, sims=None, max_events=None, batch=None):
    """Runs the listed simulations (default: all) of a workload.  Returns a
    list of counter dicts and the summed event-loop time in ns."""
    sims = range(workload.n_sims) if sims is None else sims
    b = Batch(workload) if batch is None else batch
    rc, out, total_ns = b.run(sims, max_events=max_events)
    if rc != 0:
        raise RuntimeError("oracle returned %d" % rc)
    return out, total_ns
