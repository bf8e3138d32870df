"""Python binding of libunison (argument marshalling only).

Every step of the simulation and of the ranking statistics runs in the HIP
library; PyTorch supplies device memory and the stream.  The binding raises
if the library has not been built or no GPU is present: there is no CPU path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libunison.so")

UNISON_OK, E_INVALID, E_BAD_TRACE, E_CAPACITY, E_HIP, E_NOT_READY = 0, -1, -2, -3, -4, -5
POLICY_PARAMS = 0xFF
RUN_CONTINUE, RUN_LOG = 1, 2
LUT_LEN = 51
ETA_CLASSES = 16
U64_MAX = 0xFFFFFFFFFFFFFFFF


class UnisonError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("unison error %d: %s" % (code, msg))
        self.code = code


class Dims(C.Structure):
    _fields_ = [("n_sims", C.c_uint32), ("n_traces", C.c_uint32), ("max_sessions", C.c_uint32),
                ("n_luts", C.c_uint32), ("log_cap", C.c_uint32), ("views", C.c_uint32)]


class SimParams(C.Structure):
    _fields_ = [
        ("policy", C.c_uint32), ("tide", C.c_uint32), ("score_mode", C.c_uint32),
        ("lut", C.c_uint32), ("trace", C.c_uint32), ("hazard_online", C.c_uint32),
        ("cap_sram_B", C.c_uint64), ("cap_hbm_B", C.c_uint64), ("n_slots", C.c_uint64),
        ("dma_B_per_us", C.c_uint64), ("ttl_ns", C.c_uint64),
        ("t_s_ns_per_B", C.c_double), ("t_h_ns_per_B", C.c_double),
        ("t_p_ns_per_tok", C.c_double), ("penalty_us", C.c_float), ("b_h", C.c_uint32),
        ("b_g", C.c_uint32), ("online_sessions", C.c_uint32), ("tau_ns", C.c_uint64),
        ("p_z", C.c_uint64), ("dual_sync", C.c_uint32), ("recip_bits", C.c_uint32),
    ]


COUNTER_FIELDS = (
    "requests", "hit_sram", "hit_hbm", "miss", "bypass", "evict", "expire", "promote", "swap",
    "dma_bytes", "tide_passes", "tokens_total", "tokens_computed", "extra_prefill_tok",
    "score_evals", "resident_evals", "digest", "victim_digest", "events", "error",
    "prefetch_hits", "vict_diff", "prom_diff",
)
COUNTERS_DTYPE = np.dtype([(n, np.uint64) for n in COUNTER_FIELDS] +
                          [("amat_sum_ns", np.float64), ("ttft_sum_ns", np.float64)])
RECORD_DTYPE = np.dtype([("ev", np.uint32), ("op", np.uint32), ("a", np.uint32), ("b", np.uint32)])


class TraceBatch(C.Structure):
    _fields_ = [("n_traces", C.c_uint32), ("pad0", C.c_uint32),
                ("ev_offset", C.POINTER(C.c_uint64)), ("sess_offset", C.POINTER(C.c_uint64)),
                ("ev_t_ns", C.c_void_p), ("ev_sid", C.c_void_p), ("ev_info", C.c_void_p),
                ("ev_len", C.c_void_p), ("ev_next_ns", C.c_void_p), ("sess_kvb", C.c_void_p),
                ("ev_tool", C.c_void_p)]


_lib = None


def lib():
    """Loads libunison.so; raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libunison.so is not built (run __graft_entry__.build())")
        L = C.CDLL(LIB_PATH)
        vp, i32, u32, u64 = C.c_void_p, C.c_int, C.c_uint32, C.c_uint64
        sig = {
            "unison_workspace_size": [C.POINTER(Dims), C.POINTER(C.c_size_t)],
            "unison_create": [C.POINTER(vp), C.POINTER(Dims), vp, vp, C.c_size_t],
            "unison_create_static": [C.POINTER(vp), C.POINTER(Dims), vp],
            "unison_load_traces": [vp, C.POINTER(TraceBatch)],
            "unison_hazard_counts": [vp, vp, u32, vp, vp],
            "unison_set_hazard": [vp, u32, vp, vp],
            "unison_eta_fit": [vp, u64, vp, vp, vp, vp, vp],
            "unison_set_eta": [vp, u32, vp],
            "unison_set_params": [vp, C.POINTER(SimParams)],
            "unison_run": [vp, u32, u32, u64],
            "unison_read_counters": [vp, vp, u32, u32],
            "unison_counters_device": [vp, C.POINTER(vp)],
            "unison_read_log": [vp, u32, vp, u32, C.POINTER(C.c_uint64)],
            "unison_read_hazard": [vp, u32, vp, vp],
            "unison_ema_replay": [vp, u32, u32, vp, vp, u32, u64, vp, vp],
            "unison_score_fp32": [vp, u32, vp, vp, vp, vp, vp, C.c_float, vp],
            "unison_score_fixed": [vp, u32, vp, vp, vp, vp, vp, u32, u64, u32, vp],
            "unison_kendall": [vp, u32, u32, u64, vp, vp, vp, vp, vp],
            "unison_debug_force_variant": [vp, i32],
            "unison_debug_cache_slots": [vp, i32],
            "unison_set_stream": [vp, vp],
            "unison_debug_kendall_barrier": [u32, u32, u32, u32],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = i32
        L.unison_destroy.argtypes = [vp]
        L.unison_destroy.restype = None
        L.unison_last_error.argtypes = [vp]
        L.unison_last_error.restype = C.c_char_p
        L.unison_strerror.argtypes = [i32]
        L.unison_strerror.restype = C.c_char_p
        L.unison_version.restype = u32
        _lib = L
    return _lib


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("libunison needs a ROCm GPU; torch.cuda.is_available() is False")
    return torch


def _stream():
    torch = _torch()
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _check(rc, ctx=None):
    if rc != UNISON_OK:
        L = lib()
        msg = (L.unison_last_error(ctx).decode() if ctx else L.unison_strerror(rc).decode())
        raise UnisonError(rc, msg)


def _dev(a, dtype=None):
    torch = _torch()
    a = np.ascontiguousarray(a if dtype is None else np.asarray(a, dtype=dtype))
    if a.dtype == np.uint64:
        t = torch.from_numpy(a.view(np.int64))
    elif a.dtype == np.uint32:
        t = torch.from_numpy(a.view(np.int32))
    else:
        t = torch.from_numpy(a)
    return t.to("cuda")


def _host(t, dtype):
    """Device tensor -> numpy array of `dtype` (reinterpreting the bytes)."""
    return t.cpu().numpy().view(dtype)


# -------------------------------------------------------------- simulation

class Simulator:
    """A batch of simulations on the GPU: traces, hazard tables and parameter
    rows of a workload (see paper_2609_09643_amd.synth.Workload)."""

    def __init__(self, workload, log_cap=0, variant=None, cache_slots=None, static=False):
        torch = _torch()
        L = lib()
        self.workload = workload
        traces = workload.traces
        ev_off = np.zeros(len(traces) + 1, np.uint64)
        ss_off = np.zeros(len(traces) + 1, np.uint64)
        ev_off[1:] = np.cumsum([t.n_events for t in traces])
        ss_off[1:] = np.cumsum([t.n_sessions for t in traces])
        self.ev_off, self.ss_off = ev_off, ss_off
        # one padding element keeps every device array non-empty
        cat = lambda name: np.concatenate([getattr(t, name) for t in traces] +
                                          [np.zeros(1, getattr(traces[0], name).dtype)])
        self.d_t = _dev(cat("t_ns"), np.uint64)
        self.d_sid = _dev(cat("sid"), np.uint32)
        self.d_info = _dev(cat("info"), np.uint32)
        self.d_len = _dev(cat("length"), np.uint32)
        self.d_next = _dev(cat("next_ns"), np.uint64)
        self.d_kvb = _dev(cat("kvb"), np.uint32)
        self.d_tool = _dev(cat("tool"), np.uint32)
        self.n_sims = workload.n_sims
        self.log_cap = int(log_cap)
        max_sess = max(t.n_sessions for t in traces)
        views = int(np.any(workload.params["dual_sync"] != 0))
        self.dims = Dims(self.n_sims, len(traces), max_sess, len(workload.lut_pops), self.log_cap,
                         views)
        nbytes = C.c_size_t()
        _check(L.unison_workspace_size(C.byref(self.dims), C.byref(nbytes)))
        self.ws_bytes = int(nbytes.value)
        self.ctx = C.c_void_p()
        if static:
            # the library's own static workspace: no device allocation
            self.ws = None
            rc = L.unison_create_static(C.byref(self.ctx), C.byref(self.dims), _stream())
            if rc != UNISON_OK:
                raise UnisonError(rc, L.unison_last_error(None).decode())
        else:
            self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device="cuda")
            base = self.ws.data_ptr()
            aligned = (base + 255) // 256 * 256
            _check(L.unison_create(C.byref(self.ctx), C.byref(self.dims), _stream(),
                                   C.c_void_p(aligned), C.c_size_t(self.ws_bytes)))
        if variant is not None:
            _check(L.unison_debug_force_variant(self.ctx, int(variant)), self.ctx)
        if cache_slots is not None:
            _check(L.unison_debug_cache_slots(self.ctx, int(cache_slots)), self.ctx)
        tb = TraceBatch()
        tb.n_traces = len(traces)
        self._ev_off_c = (C.c_uint64 * len(ev_off))(*[int(x) for x in ev_off])
        self._ss_off_c = (C.c_uint64 * len(ss_off))(*[int(x) for x in ss_off])
        tb.ev_offset = C.cast(self._ev_off_c, C.POINTER(C.c_uint64))
        tb.sess_offset = C.cast(self._ss_off_c, C.POINTER(C.c_uint64))
        tb.ev_t_ns, tb.ev_sid, tb.ev_info = (self.d_t.data_ptr(), self.d_sid.data_ptr(),
                                             self.d_info.data_ptr())
        tb.ev_len, tb.ev_next_ns, tb.sess_kvb = (self.d_len.data_ptr(), self.d_next.data_ptr(),
                                                 self.d_kvb.data_ptr())
        tb.ev_tool = self.d_tool.data_ptr()
        _check(L.unison_load_traces(self.ctx, C.byref(tb)), self.ctx)
        # the ETA table of each trace, fitted on the GPU from the trace's own gaps
        self.d_eta = torch.zeros((len(traces), ETA_CLASSES), dtype=torch.int64, device="cuda")
        for i, tr in enumerate(traces):
            b, n = int(ev_off[i]), int(tr.n_events)
            _check(L.unison_eta_fit(_stream(), n, C.c_void_p(self.d_t.data_ptr() + 8 * b),
                                    C.c_void_p(self.d_info.data_ptr() + 4 * b),
                                    C.c_void_p(self.d_tool.data_ptr() + 4 * b),
                                    C.c_void_p(self.d_next.data_ptr() + 8 * b), _ptr(self.d_eta[i])))
            _check(L.unison_set_eta(self.ctx, i, _ptr(self.d_eta[i])), self.ctx)
        # hazard tables: counted on the GPU from each population, or given counts
        self.d_lut_d = torch.zeros((len(workload.lut_pops), LUT_LEN), dtype=torch.int32, device="cuda")
        self.d_lut_n = torch.zeros_like(self.d_lut_d)
        flat = {i: (d, n) for (i, d, n) in getattr(workload, "flat_luts", [])}
        self._pops = []
        for i, pop in enumerate(workload.lut_pops):
            if pop is not None:
                dp = _dev(pop, np.uint32)
                self._pops.append(dp)
                _check(L.unison_hazard_counts(_stream(), _ptr(dp), int(dp.numel()),
                                              _ptr(self.d_lut_d[i]), _ptr(self.d_lut_n[i])))
            else:
                d, n = flat[i]
                self.d_lut_d[i].fill_(int(d))
                self.d_lut_n[i].fill_(int(n))
            _check(L.unison_set_hazard(self.ctx, i, _ptr(self.d_lut_d[i]), _ptr(self.d_lut_n[i])),
                   self.ctx)
        self.set_params(workload.params)

    def set_params(self, rows):
        arr = (SimParams * self.n_sims)()
        names = [f for f, _ in SimParams._fields_ if not f.startswith("pad")]
        for i in range(self.n_sims):
            r = rows[i]
            for f in names:
                v = r[f]
                setattr(arr[i], f, float(v) if f.startswith("t_") or f == "penalty_us" else int(v))
        self._params_c = arr
        _check(lib().unison_set_params(self.ctx, arr), self.ctx)

    def run(self, policy=POLICY_PARAMS, flags=0, max_events=None):
        me = U64_MAX if max_events is None else int(max_events)
        _check(lib().unison_run(self.ctx, policy, flags, me), self.ctx)

    def set_eta(self, trace, table):
        """Installs an ETA table (ns per tool class) for a trace in place of
        the one fitted on it."""
        t = _dev(np.asarray(table, np.uint64), np.uint64)
        self.d_eta[trace].copy_(t)
        _check(lib().unison_set_eta(self.ctx, trace, _ptr(self.d_eta[trace])), self.ctx)

    def eta_table(self, trace):
        """The ETA table fitted on the GPU for a trace (ns per tool class)."""
        return _host(self.d_eta[trace], np.uint64)

    def counters(self, check=True):
        out = np.zeros(self.n_sims, COUNTERS_DTYPE)
        rc = lib().unison_read_counters(self.ctx, out.ctypes.data_as(C.c_void_p), 0, self.n_sims)
        if check:
            _check(rc, self.ctx)
        return out

    def counters_device(self):
        p = C.c_void_p()
        _check(lib().unison_counters_device(self.ctx, C.byref(p)), self.ctx)
        return p.value

    def log(self, sim):
        cap = max(self.log_cap, 1)
        out = np.zeros(cap, RECORD_DTYPE)
        n = C.c_uint64()
        _check(lib().unison_read_log(self.ctx, sim, out.ctypes.data_as(C.c_void_p), cap,
                                     C.byref(n)), self.ctx)
        kept = min(int(n.value), self.log_cap)
        if int(n.value) > self.log_cap:
            raise RuntimeError("decision log overflow: %d > %d" % (n.value, self.log_cap))
        return out[:kept]

    def hazard(self, sim):
        """The hazard counts (d, n) [51] of simulation `sim`'s table after the
        latest run."""
        d = np.zeros(LUT_LEN, np.uint32)
        n = np.zeros(LUT_LEN, np.uint32)
        _check(lib().unison_read_hazard(self.ctx, sim, d.ctypes.data_as(C.c_void_p),
                                        n.ctypes.data_as(C.c_void_p)), self.ctx)
        return d, n

    def close(self):
        if self.ctx:
            lib().unison_destroy(self.ctx)
            self.ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------ ranking fidelity

def hazard_counts(turns_dev):
    torch = _torch()
    d = torch.zeros(LUT_LEN, dtype=torch.int32, device="cuda")
    n = torch.zeros(LUT_LEN, dtype=torch.int32, device="cuda")
    _check(lib().unison_hazard_counts(_stream(), _ptr(turns_dev), int(turns_dev.numel()), _ptr(d),
                                      _ptr(n)))
    return d, n


def ema_replay(gaps_dev, n_hist_dev, b_g=32, tau_ns=1000):
    """gaps_dev int64 [n, max_hist] (ns), n_hist_dev uint8 [n] ->
    (g float32 [n], gq int64 [n] holding uint64 values)."""
    torch = _torch()
    n, mh = gaps_dev.shape
    g = torch.empty(n, dtype=torch.float32, device="cuda")
    gq = torch.empty(n, dtype=torch.int64, device="cuda")
    _check(lib().unison_ema_replay(_stream(), n, mh, _ptr(gaps_dev), _ptr(n_hist_dev), b_g,
                                   tau_ns, _ptr(g), _ptr(gq)))
    return g, gq


def score_fp32(turn_dev, g_dev, done_dev, d_dev, n_dev, penalty_us):
    torch = _torch()
    out = torch.empty(turn_dev.numel(), dtype=torch.float32, device="cuda")
    _check(lib().unison_score_fp32(_stream(), int(turn_dev.numel()), _ptr(turn_dev), _ptr(g_dev),
                                   _ptr(done_dev), _ptr(d_dev), _ptr(n_dev),
                                   C.c_float(penalty_us), _ptr(out)))
    return out


def score_fixed(turn_dev, gq_dev, done_dev, d_dev, n_dev, b_h=12, p_z=500_000_000, recip_bits=0):
    torch = _torch()
    out = torch.empty(turn_dev.numel(), dtype=torch.int64, device="cuda")
    _check(lib().unison_score_fixed(_stream(), int(turn_dev.numel()), _ptr(turn_dev), _ptr(gq_dev),
                                    _ptr(done_dev), _ptr(d_dev), _ptr(n_dev), b_h, p_z, recip_bits,
                                    _ptr(out)))
    return out


def kendall(x_dev, y_dev, idx_dev=None, n_snap=None, n_per=None):
    """Pair counts [n_snap, 5] (int64 holding uint64) and top-1 flags [n_snap]."""
    torch = _torch()
    if idx_dev is not None:
        n_snap, n_per = idx_dev.shape
    counts = torch.empty((n_snap, 5), dtype=torch.int64, device="cuda")
    top1 = torch.empty(n_snap, dtype=torch.uint8, device="cuda")
    _check(lib().unison_kendall(_stream(), n_snap, n_per, int(x_dev.numel()), _ptr(x_dev),
                                _ptr(y_dev), _ptr(idx_dev), _ptr(counts), _ptr(top1)))
    return counts, top1
