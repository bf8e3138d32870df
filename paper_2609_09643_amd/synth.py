"""Seeded synthetic inputs shared by the HIP path, the oracle and the tests.

This module only draws data: session traces (arrival, gap-start and
completion events with their token lengths), per-simulation parameter rows
and raw populations (turn counts, gap histories) from which each side fits
its own hazard table and runs its own EMA.  It holds none of the policy's
arithmetic.

Workload shapes follow the paper's evaluation setup (Sec. V-A): agent
sessions whose prefix grows monotonically turn over turn (Sec. I), tool gaps
with medians of seconds and a 1 ms floor (Sec. VI-E), capacity envelopes in
tokens (Table VI) and 1,415 sessions / 33,596 turns in total (Sec. V-A).  The
paper's own traces are not available; these generators stand in for them.

Event encoding (the binary trace format both implementations read):
  t_ns     uint64  event time in nanoseconds, non-decreasing
  sid      uint32  session index within the trace
  info     uint32  kind << 24 | turn  (kind 0 ARRIVE, 1 GAP_START, 2 DONE)
  length   uint32  ARRIVE: resident KV length of the new turn in tokens, else 0
  next_ns  uint64  GAP_START: time of the session's next ARRIVE, else 2^64-1
  tool     uint32  GAP_START: the tool class of the gap that starts (0..4), else 0
Per session: kvb (uint32) KV bytes per token; turns (uint32) its turn count.

Tool classes.  A tool gap belongs to one of TOOL_CLASSES classes whose
medians spread around the gap distribution's median; a user wait is class
USER_CLASS.  The label of each drawn tool gap is sampled from its posterior
under that mixture (class c has log-median ln m + TOOL_OFFSETS[c] and log-
spread TOOL_SIGMA_W), with a generator seeded from the trace generator's
state without drawing from it, so labelling changes none of the trace's
other values.  The labels feed the tool-type arrival-table baseline (ETA).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

KIND_ARRIVE, KIND_GAP_START, KIND_DONE = 0, 1, 2
POLICY_SPEAR, POLICY_LRU, POLICY_TIMEOUT, POLICY_BELADY, POLICY_ETA = 0, 1, 2, 3, 4
POLICY_NAMES = ("spear_tide", "lru", "timeout", "belady", "eta")
# Tool-class labels of gaps: four tool classes around the tool-wait median and
# one class for user waits.  Offsets of the class log-medians (spread a, 3a
# around it with 1.25 a^2 + TOOL_SIGMA_W^2 = 1, the tool gaps' log-variance).
TOOL_SIGMA_W = 0.6
TOOL_OFFSETS = (-1.0733, -0.3578, 0.3578, 1.0733)
TOOL_CLASSES = len(TOOL_OFFSETS)
USER_CLASS = TOOL_CLASSES
ETA_CLASSES = 16                  # table entries of the ETA baseline
U64_MAX = np.uint64(0xFFFFFFFFFFFFFFFF)
KIB, MIB, GIB = 1024, 1024 ** 2, 1024 ** 3
NS = 1_000_000_000

# One row per simulation.  Each implementation copies these fields into its
# own argument layout.
SIM_PARAMS_DTYPE = np.dtype([
    ("policy", np.uint32), ("tide", np.uint32), ("score_mode", np.uint32),
    ("lut", np.uint32), ("trace", np.uint32), ("hazard_online", np.uint32),
    ("online_sessions", np.uint32), ("cap_sram_B", np.uint64), ("cap_hbm_B", np.uint64), ("n_slots", np.uint64),
    ("dma_B_per_us", np.uint64), ("ttl_ns", np.uint64),
    ("t_s_ns_per_B", np.float64), ("t_h_ns_per_B", np.float64),
    ("t_p_ns_per_tok", np.float64), ("penalty_us", np.float32),
    ("b_h", np.uint32), ("b_g", np.uint32), ("tau_ns", np.uint64), ("p_z", np.uint64),
    ("dual_sync", np.uint32), ("recip_bits", np.uint32),
])
DUAL_NONE, DUAL_EVERY, DUAL_EIGHT, DUAL_GAP = 0, 1, 2, 3


@dataclass
class Trace:
    t_ns: np.ndarray
    sid: np.ndarray
    info: np.ndarray
    length: np.ndarray
    next_ns: np.ndarray
    kvb: np.ndarray
    turns: np.ndarray
    tool: Optional[np.ndarray] = None   # per event (GAP_START: tool class), or None: all 0

    def __post_init__(self):
        if self.tool is None:
            self.tool = np.zeros(self.t_ns.shape[0], np.uint32)

    @property
    def n_events(self) -> int:
        return int(self.t_ns.shape[0])

    @property
    def n_sessions(self) -> int:
        return int(self.kvb.shape[0])

    @property
    def kind(self) -> np.ndarray:
        return (self.info >> 24).astype(np.uint32)

    @property
    def turn(self) -> np.ndarray:
        return (self.info & 0xFFFFFF).astype(np.uint32)

    def prefix(self, n: int) -> "Trace":
        return Trace(self.t_ns[:n], self.sid[:n], self.info[:n], self.length[:n],
                     self.next_ns[:n], self.kvb, self.turns, self.tool[:n])


@dataclass
class Workload:
    """A batch of simulations: traces, hazard-count populations and sims."""
    name: str
    traces: List[Trace]
    lut_pops: List[np.ndarray]          # turn-count population per hazard table
    params: np.ndarray                  # SIM_PARAMS_DTYPE, one row per simulation
    flat_luts: List[tuple] = field(default_factory=list)  # (index, d, n) constant tables

    @property
    def n_sims(self) -> int:
        return int(self.params.shape[0])


# ------------------------------------------------------------------ samplers

def _lognormal_s(rng, median_s, sigma, n, lo=None, hi=None):
    x = rng.lognormal(np.log(median_s), sigma, n)
    if lo is not None or hi is not None:
        x = np.clip(x, lo if lo is not None else -np.inf, hi if hi is not None else np.inf)
    return x


def gaps_single(rng, n):
    """lognormal(mu = ln 2 s, sigma = 1), at least 1 ms."""
    return _lognormal_s(rng, 2.0, 1.0, n, lo=1e-3)


def _gaps_single_parts(rng, n):
    return gaps_single(rng, n), np.zeros(n, bool)


gaps_single.parts = _gaps_single_parts
gaps_single.tool_median_s = 2.0


def _gaps_mixture_parts(rng, n):
    tool = _lognormal_s(rng, 4.0, 1.0, n, lo=0.5, hi=60.0)
    user = _lognormal_s(rng, 30.0, 1.0, n, lo=5.0, hi=300.0)
    is_tool = rng.random(n) < 0.8
    return np.where(is_tool, tool, user), ~is_tool


def gaps_mixture(rng, n):
    """80 % tool waits lognormal(ln 4 s, 1) in [0.5, 60] s, 20 % user waits
    lognormal(ln 30 s, 1) in [5, 300] s."""
    return _gaps_mixture_parts(rng, n)[0]


gaps_mixture.parts = _gaps_mixture_parts
gaps_mixture.tool_median_s = 4.0


def label_tools(lrng, gaps_s, is_user, tool_median_s):
    """Tool class of each gap: USER_CLASS for user waits; for tool waits a
    draw from the posterior over the TOOL_CLASSES classes (equal priors,
    class log-medians ln(tool_median_s) + TOOL_OFFSETS, log-spread
    TOOL_SIGMA_W) given the gap."""
    x = np.log(np.maximum(gaps_s, 1e-9)) - np.log(tool_median_s)
    d = x[:, None] - np.asarray(TOOL_OFFSETS)[None, :]
    w = np.exp(-0.5 * (d / TOOL_SIGMA_W) ** 2 - np.max(-0.5 * (d / TOOL_SIGMA_W) ** 2, axis=1,
                                                         keepdims=True))
    cdf = np.cumsum(w / w.sum(axis=1, keepdims=True), axis=1)
    u = lrng.random(gaps_s.shape[0])
    cls = np.minimum((u[:, None] > cdf).sum(axis=1), TOOL_CLASSES - 1)
    return np.where(is_user, USER_CLASS, cls).astype(np.uint32)


def _side_generator(rng):
    """A generator seeded from rng's current state, without drawing from rng."""
    st = int(rng.bit_generator.state["state"]["state"])
    return np.random.Generator(np.random.PCG64([st & (2 ** 64 - 1), st >> 64, 0x7001]))


def service_times(rng, n):
    """Turn service time lognormal(ln 1 s, 0.5) in [50 ms, 20 s]."""
    return _lognormal_s(rng, 1.0, 0.5, n, lo=0.05, hi=20.0)


def geometric_turns(rng, n_sessions, mean, total=None):
    t = rng.geometric(1.0 / mean, n_sessions).astype(np.int64)
    if total is not None:
        diff = int(total - t.sum())
        while diff != 0:
            i = int(rng.integers(n_sessions))
            if diff > 0:
                t[i] += 1
                diff -= 1
            elif t[i] > 1:
                t[i] -= 1
                diff += 1
    return t.astype(np.uint32)


def lognormal_turns(rng, n, median=15.0, sigma=0.8):
    """Turn counts T = 1 + floor(lognormal(ln median, sigma))."""
    return (1 + np.floor(rng.lognormal(np.log(median), sigma, n))).astype(np.uint32)


# ------------------------------------------------------------- trace builder

def build_trace(rng, turns, first_arrival_s, gap_fn, kvb, grow_lo=200, grow_hi=2000,
                max_len=131072) -> Trace:
    turns = np.asarray(turns, dtype=np.int64)
    n_sess = turns.shape[0]
    total = int(turns.sum())
    owner = np.repeat(np.arange(n_sess, dtype=np.int64), turns)
    starts = np.concatenate([[0], np.cumsum(turns)[:-1]])
    k = np.arange(total, dtype=np.int64) - starts[owner]

    svc_ns = np.rint(service_times(rng, total) * NS).astype(np.int64)
    parts = getattr(gap_fn, "parts", None)
    if parts is not None:
        gap_s, is_user = parts(rng, total)
    else:
        gap_s, is_user = gap_fn(rng, total), None
    gap_ns = np.rint(gap_s * NS).astype(np.int64)
    gap_ns[k == 0] = 0
    grow = rng.integers(grow_lo, grow_hi + 1, total).astype(np.int64)
    first_ns = np.rint(np.asarray(first_arrival_s) * NS).astype(np.int64)

    # a_{s,0} = first arrival; c_{s,k} = a_{s,k} + service; a_{s,k+1} = c_{s,k} + gap
    step = svc_ns + gap_ns                     # gap before turn k + service of turn k
    cum = np.cumsum(step)
    seg_base = np.concatenate([[0], cum[starts[1:] - 1]]) if n_sess > 1 else np.array([0])
    cum_in = cum - seg_base[owner]             # sum over turns 0..k of (gap + service)
    arrive = first_ns[owner] + cum_in - svc_ns
    complete = arrive + svc_ns
    lcum = np.cumsum(grow)
    lbase = np.concatenate([[0], lcum[starts[1:] - 1]]) if n_sess > 1 else np.array([0])
    length = np.minimum(lcum - lbase[owner], max_len)

    last = k == turns[owner] - 1
    next_arrive = np.empty(total, dtype=np.int64)
    next_arrive[:-1] = arrive[1:]
    next_arrive[-1] = -1
    # tool class of the gap that follows turn k (the gap before turn k + 1)
    if is_user is not None:
        cls = label_tools(_side_generator(rng), gap_s, is_user, gap_fn.tool_median_s)
    else:
        cls = np.zeros(total, np.uint32)
    next_cls = np.zeros(total, np.uint32)
    next_cls[:-1] = cls[1:]

    n_ev = 2 * total
    t = np.empty(n_ev, dtype=np.int64)
    sid = np.empty(n_ev, dtype=np.int64)
    kind = np.empty(n_ev, dtype=np.int64)
    turn = np.empty(n_ev, dtype=np.int64)
    ln = np.zeros(n_ev, dtype=np.int64)
    nxt = np.full(n_ev, -1, dtype=np.int64)
    t[0::2], t[1::2] = arrive, complete
    sid[0::2] = sid[1::2] = owner
    turn[0::2] = turn[1::2] = k
    kind[0::2] = KIND_ARRIVE
    kind[1::2] = np.where(last, KIND_DONE, KIND_GAP_START)
    ln[0::2] = length
    nxt[1::2] = np.where(last, -1, next_arrive)
    tool = np.zeros(n_ev, dtype=np.int64)
    tool[1::2] = np.where(last, 0, next_cls)
    rank = np.where(kind == KIND_ARRIVE, 1, 0)  # at equal times: ends before arrivals
    order = np.lexsort((sid, rank, t))
    nxt_u = nxt[order].astype(np.uint64)
    nxt_u[nxt[order] < 0] = U64_MAX
    return Trace(
        t_ns=t[order].astype(np.uint64),
        sid=sid[order].astype(np.uint32),
        info=((kind[order] << 24) | turn[order]).astype(np.uint32),
        length=ln[order].astype(np.uint32),
        next_ns=nxt_u,
        kvb=np.asarray(kvb, dtype=np.uint32),
        turns=turns.astype(np.uint32),
        tool=tool[order].astype(np.uint32),
    )


def poisson_arrivals(rng, n, rate_per_s):
    return np.cumsum(rng.exponential(1.0 / rate_per_s, n))


# ------------------------------------------------------------- parameter rows

def default_params(n):
    p = np.zeros(n, dtype=SIM_PARAMS_DTYPE)
    p["tide"] = 1
    p["n_slots"] = 64
    p["dma_B_per_us"] = 100_000          # 100 GB/s
    p["ttl_ns"] = 30 * NS
    p["t_s_ns_per_B"] = 1e-4
    p["t_h_ns_per_B"] = 1e-3
    p["t_p_ns_per_tok"] = 5e4
    p["penalty_us"] = np.float32(5e8)
    p["b_h"], p["b_g"], p["tau_ns"], p["p_z"] = 12, 32, 1000, 500_000_000
    p["online_sessions"] = 0xFFFFFFFF
    return p


def set_policy(p, policy, tide=None):
    """TIDE is on by default for SPEAR and Belady, off for the recency, timeout
    and ETA baselines."""
    p["policy"] = policy
    p["tide"] = (1 if policy in (POLICY_SPEAR, POLICY_BELADY) else 0) if tide is None else tide


# ------------------------------------------------------------------ workloads

def tiny_trace(seed=1, n_sessions=16, turns=12):
    rng = np.random.Generator(np.random.PCG64(seed))
    first = poisson_arrivals(rng, n_sessions, 5.0)
    return build_trace(rng, np.full(n_sessions, turns), first, gaps_single,
                       np.full(n_sessions, 128 * KIB))


def hazard_population(seed, n):
    rng = np.random.Generator(np.random.PCG64(seed))
    return lognormal_turns(rng, n)


# The constant hazard 1/23.7 written as counts: d = 10, n = 237 at every t.
FLAT_COUNTS = (10, 237)


def c1_tiny(seed=1) -> Workload:
    """16 sessions x 12 turns, 128 KiB/token, SRAM 64 MiB, HBM 2 GiB, DMA
    100 GB/s; SPEAR+TIDE and Belady on the same trace."""
    tr = tiny_trace(seed)
    p = default_params(2)
    set_policy(p[0:1], POLICY_SPEAR)
    set_policy(p[1:2], POLICY_BELADY)
    p["cap_sram_B"], p["cap_hbm_B"] = 64 * MIB, 2 * GIB
    return Workload("c1_tiny", [tr], [tr.turns], p)


C3_SRAM_MIB = (16, 24, 32, 48, 64, 96, 128, 256)
C3_HBM_GIB = (1, 2, 4, 8, 16, 24, 32, 64)
C3_TTL_S = (1, 2, 5, 10, 20, 30, 60, 120)
C3_PENALTY = (5e8, 5e7)


def c3_sweep(policies=(0, 1, 2, 3), n_seeds=8) -> Workload:
    """4,096 simulations per policy: 8 C1-shaped traces x 8 SRAM x 8 HBM
    capacities x 8 hazard variants (4 tables x 2 penalties; TTLs for the
    timeout policy).  Simulations that share (policy, trace) are contiguous."""
    traces = [tiny_trace(seed) for seed in range(1, n_seeds + 1)]
    pops = [tr.turns for tr in traces]
    pops.append(None)                       # placeholder: the flat table
    pops.append(hazard_population(1128, 128))
    pops.append(hazard_population(1496, 496))
    flat_idx = n_seeds
    rows = []
    for pol in policies:
        for ti in range(n_seeds):
            for si, s_mib in enumerate(C3_SRAM_MIB):
                for hi, h_gib in enumerate(C3_HBM_GIB):
                    for v in range(8):
                        rows.append((pol, ti, s_mib, h_gib, v))
    p = default_params(len(rows))
    arr = np.array(rows, dtype=np.int64)
    pol, ti, s_mib, h_gib, v = arr.T
    p["trace"] = ti
    p["cap_sram_B"] = s_mib.astype(np.uint64) * MIB
    p["cap_hbm_B"] = h_gib.astype(np.uint64) * GIB
    p["policy"] = pol
    p["tide"] = np.isin(pol, (POLICY_SPEAR, POLICY_BELADY)).astype(np.uint32)
    table = v // 2
    p["lut"] = np.where(table == 0, ti, np.where(table == 1, flat_idx, flat_idx + table - 1))
    pen = np.array(C3_PENALTY)[v % 2]
    p["penalty_us"] = pen.astype(np.float32)
    p["p_z"] = pen.astype(np.uint64)      # P_Z = P / tau with P in ns, tau = 1 us
    p["ttl_ns"] = np.where(pol == POLICY_TIMEOUT, np.array(C3_TTL_S)[v] * NS, 30 * NS).astype(np.uint64)
    return Workload("c3_sweep", traces, pops, p, flat_luts=[(flat_idx,) + FLAT_COUNTS])


def c2_paper_scale(seed=2) -> Workload:
    """1,415 sessions, 33,596 turns (geometric, mean 23.7), Poisson 5/s
    arrivals, mixture gaps, KV 64/128/160 KiB per token; a pool of 80K SRAM /
    400K HBM tokens at 128 KiB and 64 session slots; all four policies."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = 1415
    turns = geometric_turns(rng, n, 23.7, total=33596)
    first = poisson_arrivals(rng, n, 5.0)
    kvb = np.array([64, 128, 160], dtype=np.uint32)[rng.permutation(n) % 3] * KIB
    tr = build_trace(rng, turns, first, gaps_mixture, kvb)
    p = default_params(4)
    for q in range(4):
        set_policy(p[q:q + 1], q)
    # The Edge-Tight envelope (10K / 50K tokens, Table VI) scaled by 8: this
    # trace keeps ~530 sessions live at once, about 8x the paper's traces.
    p["cap_sram_B"] = 8 * 10_000 * 128 * KIB
    p["cap_hbm_B"] = 8 * 50_000 * 128 * KIB
    p["n_slots"] = 64
    return Workload("c2_paper_scale", [tr], [tr.turns], p)


def c4_large(n_traces=8, n_sessions=65536, total_turns=2_000_000, seed0=100) -> Workload:
    """65,536 concurrently live sessions, 2M turns, prefixes up to 128K
    tokens at 160 KiB/token, SRAM 512 MiB, HBM 288 GiB; 8 traces x 8 hazard
    variants of SPEAR+TIDE."""
    traces = []
    for i in range(n_traces):
        rng = np.random.Generator(np.random.PCG64(seed0 + i))
        turns = geometric_turns(rng, n_sessions, total_turns / n_sessions, total=total_turns)
        first = np.sort(rng.uniform(0.0, 60.0, n_sessions))
        traces.append(build_trace(rng, turns, first, gaps_mixture,
                                  np.full(n_sessions, 160 * KIB)))
    pops = [tr.turns for tr in traces]
    pops.append(None)
    pops.append(hazard_population(2128, 128))
    pops.append(hazard_population(2496, 496))
    flat_idx = n_traces
    p = default_params(n_traces * 8)
    set_policy(p, POLICY_SPEAR)
    p["trace"] = np.repeat(np.arange(n_traces), 8)
    v = np.tile(np.arange(8), n_traces)
    table = v // 2
    p["lut"] = np.where(table == 0, p["trace"], np.where(table == 1, flat_idx, flat_idx + table - 1))
    pen = np.array(C3_PENALTY)[v % 2]
    p["penalty_us"] = pen.astype(np.float32)
    p["p_z"] = pen.astype(np.uint64)
    p["cap_sram_B"] = 512 * MIB
    p["cap_hbm_B"] = 288 * GIB
    # N_sess = 4,096 register slots: the traces never hold more than 2,048
    # residents, so the bound never binds (the decisions of the whole trace
    # are those of N_sess = 65,536)
    p["n_slots"] = 4096
    return Workload("c4_large", traces, pops, p, flat_luts=[(flat_idx,) + FLAT_COUNTS])


@dataclass
class RankingSet:
    """Register-file snapshots for the ranking-fidelity study: a pool of
    session states (turn index, completion flag, raw gap history) and, per
    snapshot, the pool entries resident at that moment."""
    turn: np.ndarray       # uint8 [pool]
    done: np.ndarray       # uint8 [pool]
    gaps_ns: np.ndarray    # uint64 [pool, max_hist]
    n_hist: np.ndarray     # uint8 [pool]
    idx: np.ndarray        # uint32 [n_snap, n_per]
    lut_pop: np.ndarray    # turn counts the hazard table is fitted on

    @property
    def n_snap(self):
        return int(self.idx.shape[0])

    @property
    def n_per(self):
        return int(self.idx.shape[1])


def c5_ranking(n_snap=10000, n_per=4096, pool=65536, max_hist=8, seed=5) -> RankingSet:
    """Turn indices from 23.7-mean geometric sessions capped at 60, a gap
    history of min(t, 8) mixture gaps per session, 2 % completed sessions,
    and a hazard table fitted on 128 lognormal(ln 15, 0.8) turn counts."""
    rng = np.random.Generator(np.random.PCG64(seed))
    turn = np.minimum(rng.geometric(1 / 23.7, pool) - 1, 60).astype(np.uint8)
    done = (rng.random(pool) < 0.02).astype(np.uint8)
    n_hist = np.minimum(turn, max_hist).astype(np.uint8)
    gaps = np.rint(gaps_mixture(rng, pool * max_hist) * NS).astype(np.uint64).reshape(pool, max_hist)
    gaps[np.arange(max_hist)[None, :] >= n_hist[:, None]] = 0
    idx = np.empty((n_snap, n_per), dtype=np.uint32)
    for s in range(n_snap):
        idx[s] = rng.choice(pool, size=n_per, replace=False)
    lut_pop = lognormal_turns(np.random.Generator(np.random.PCG64(seed + 1000)), 128)
    return RankingSet(turn, done, gaps, n_hist, idx, lut_pop)


# ------------------------------------------------- fixed-point format sweep

# Sec. IV-C: the pre-registered grid of hazard bits b_h, gap-register bits
# b_g and time divisor tau (exact divider, b_s = 64), and the locked point of
# eq. (lock).
FORMAT_BH = (8, 10, 12)
FORMAT_BG = (24, 32, 64)
FORMAT_TAU_NS = (1, 1000, 1_000_000)
LOCKED_FORMAT = (12, 32, 1000)
# The divider type of eq. (t1): 0 is the exact divider; W > 0 a reciprocal
# table of depth Lambda whose entries hold W fraction bits (the entry width is
# not given: it is swept).
FORMAT_DIVIDERS = (0, 12, 16, 20, 24)

# Six traces of 128..496 sessions, 1,415 sessions and 33,596 turns in all
# (Sec. V-A); three capacity envelopes of Table VI in tokens at 128 KiB/token:
# Edge-Tight (10K SRAM / 50K HBM) and its HBM-100K and SRAM-20K neighbours.
FIDELITY_SESSIONS = (128, 160, 192, 215, 224, 496)
FIDELITY_ENVELOPES = ((10_000, 50_000), (10_000, 100_000), (20_000, 50_000))
FIDELITY_TURNS = 33_596


def format_grid():
    """The 27 (b_h, b_g, tau_ns) points of the format sweep."""
    return [(bh, bg, tau) for bh in FORMAT_BH for bg in FORMAT_BG for tau in FORMAT_TAU_NS]


def format_grid_dividers(dividers=FORMAT_DIVIDERS):
    """The sweep with its divider-type axis: (b_h, b_g, tau_ns, W) for every
    grid point and divider (W = 0 exact, else reciprocal-table bits)."""
    return [(bh, bg, tau, w) for (bh, bg, tau) in format_grid() for w in dividers]


def fix_total(rng, t, total, lo=1):
    """Adds or removes single turns at random sessions until sum(t) = total."""
    t = np.asarray(t, dtype=np.int64).copy()
    diff = int(total - t.sum())
    while diff != 0:
        i = int(rng.integers(t.shape[0]))
        if diff > 0:
            t[i] += 1
            diff -= 1
        elif t[i] > lo:
            t[i] -= 1
            diff += 1
    return t.astype(np.uint32)


def fidelity_traces(seed=300, rate_per_s=0.2):
    """The six stand-in traces: turn counts 1 + floor(lognormal(ln 16.5,
    0.8)) (mean about 23.7, a hazard that rises with the turn index) fixed up
    to 33,596 turns in all; Poisson arrivals at 0.2 sessions/s, which keeps
    about 50 sessions live at once (the paper's traces stay at or below 64);
    mixture gaps; KV 64/128/160 KiB per token in thirds."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n_all = sum(FIDELITY_SESSIONS)
    turns = fix_total(rng, lognormal_turns(rng, n_all, median=16.5), FIDELITY_TURNS)
    traces, at = [], 0
    for n in FIDELITY_SESSIONS:
        first = poisson_arrivals(rng, n, rate_per_s)
        kvb = np.array([64, 128, 160], dtype=np.uint32)[rng.permutation(n) % 3] * KIB
        traces.append(build_trace(rng, turns[at:at + n], first, gaps_mixture, kvb))
        at += n
    return traces


FORMAT_META_DTYPE = np.dtype([("trace", np.uint32), ("envelope", np.uint32), ("fmt", np.int32)])


def format_sweep(traces=None, envelopes=FIDELITY_ENVELOPES, formats=None, penalty_us=5e8):
    """SPEAR+TIDE on every (trace, envelope) cell, once with the fp32 score
    and once per fixed-point format.  Returns the workload and, per
    simulation, its (trace, envelope, format index; -1 for fp32).  P_Z is the
    penalty in units of tau: P_Z = P / tau (eq. (lock)).  A format is (b_h,
    b_g, tau_ns) with the exact divider, or (b_h, b_g, tau_ns, W) with W the
    reciprocal table's fraction bits (0: exact)."""
    traces = fidelity_traces() if traces is None else traces
    formats = format_grid() if formats is None else list(formats)
    rows, meta = [], []
    for ti in range(len(traces)):
        for ei in range(len(envelopes)):
            for fi in range(-1, len(formats)):
                rows.append((ti, ei, fi))
    p = default_params(len(rows))
    set_policy(p, POLICY_SPEAR)
    m = np.zeros(len(rows), dtype=FORMAT_META_DTYPE)
    for r, (ti, ei, fi) in enumerate(rows):
        s_tok, h_tok = envelopes[ei]
        p[r]["trace"] = ti
        p[r]["lut"] = ti
        p[r]["cap_sram_B"] = s_tok * 128 * KIB
        p[r]["cap_hbm_B"] = h_tok * 128 * KIB
        p[r]["penalty_us"] = np.float32(penalty_us)
        if fi >= 0:
            bh, bg, tau = formats[fi][:3]
            p[r]["score_mode"] = 1
            p[r]["b_h"], p[r]["b_g"], p[r]["tau_ns"] = bh, bg, tau
            p[r]["recip_bits"] = formats[fi][3] if len(formats[fi]) > 3 else 0
            p[r]["p_z"] = int(round(penalty_us * 1000 / tau))
        m[r] = (ti, ei, fi)
    w = Workload("format_sweep", list(traces), [tr.turns for tr in traces], p)
    return w, m


def fidelity_snapshots(n_snap=7265, n_per=64, seed=6) -> RankingSet:
    """Eviction-snapshot stand-ins for the format sweep's ranking gate: the
    C5 session pool drawn into 7,265 snapshots of 64 live sessions (the
    paper's traces keep at most 64 live)."""
    return c5_ranking(n_snap=n_snap, n_per=n_per, seed=seed)


ATTAIN_META_DTYPE = np.dtype([("trace", np.uint32), ("kind", np.uint32), ("n", np.uint32)])
ATTAIN_LRU, ATTAIN_OFFLINE, ATTAIN_ONLINE, ATTAIN_PREFIX = 0, 1, 2, 3


def completion_order(tr):
    """Session ids in the order their DONE events occur."""
    return tr.sid[tr.kind == KIND_DONE]


def attainment_workload(traces=None, envelope=FIDELITY_ENVELOPES[0], points=None):
    """Per trace: LRU; SPEAR+TIDE with the table fitted on the whole trace;
    and, for n in `points` (default 0, 1, 2, 4, ... and the trace's session
    count), SPEAR+TIDE whose table starts empty and counts the first n
    completions as they happen (ATTAIN_ONLINE), and SPEAR+TIDE with a fixed
    table fitted on the turn counts of the first n sessions to complete
    (ATTAIN_PREFIX)."""
    traces = fidelity_traces() if traces is None else traces
    rows, pops = [], [tr.turns for tr in traces]
    for ti, tr in enumerate(traces):
        N = tr.n_sessions
        pts = points if points is not None else sorted({0, N} | {1 << k for k in range(20) if (1 << k) < N})
        order = completion_order(tr)
        rows.append((ti, ATTAIN_LRU, 0, ti))
        rows.append((ti, ATTAIN_OFFLINE, N, ti))
        for n in pts:
            rows.append((ti, ATTAIN_ONLINE, int(n), ti))
            pops.append(tr.turns[order[:int(n)]])
            rows.append((ti, ATTAIN_PREFIX, int(n), len(pops) - 1))
    p = default_params(len(rows))
    meta = np.zeros(len(rows), ATTAIN_META_DTYPE)
    for r, (ti, kind, n, lut) in enumerate(rows):
        set_policy(p[r:r + 1], POLICY_LRU if kind == ATTAIN_LRU else POLICY_SPEAR)
        p[r]["trace"] = ti
        p[r]["lut"] = lut
        p[r]["cap_sram_B"] = envelope[0] * 128 * KIB
        p[r]["cap_hbm_B"] = envelope[1] * 128 * KIB
        if kind == ATTAIN_ONLINE:
            p[r]["hazard_online"] = 1
            p[r]["online_sessions"] = n
        meta[r] = (ti, kind, n)
    return Workload("attainment", list(traces), pops, p), meta


# ---------------------------------------------- ablations and capacity sweep

# Six SRAM/HBM envelopes (tokens at 128 KiB) along the axes of Table VI.
ABLATION_ENVELOPES = ((10_000, 30_000), (10_000, 50_000), (10_000, 100_000), (10_000, 200_000),
                      (20_000, 50_000), (40_000, 50_000))
# scoring x tiering: (policy, tide); the tool-type arrival table (ETA) is the
# third evictor, with and without TIDE
COMPONENTS = (("lru", POLICY_LRU, 0), ("lru+tide", POLICY_LRU, 1), ("spear", POLICY_SPEAR, 0),
              ("spear+tide", POLICY_SPEAR, 1), ("eta", POLICY_ETA, 0), ("eta+tide", POLICY_ETA, 1))
ASE_SLOTS = (4, 8, 16, 32, 64, 128, 256)
STUDY_META_DTYPE = np.dtype([("trace", np.uint32), ("envelope", np.uint32), ("arm", np.uint32)])


def _study_rows(traces, cells):
    """cells: list of (trace, envelope (sram_tok, hbm_tok), arm, dict of
    parameter overrides)."""
    p = default_params(len(cells))
    meta = np.zeros(len(cells), STUDY_META_DTYPE)
    for r, (ti, env, ei, arm, over) in enumerate(cells):
        p[r]["trace"], p[r]["lut"] = ti, ti
        p[r]["cap_sram_B"] = env[0] * 128 * KIB
        p[r]["cap_hbm_B"] = env[1] * 128 * KIB
        for k, v in over.items():
            p[r][k] = v
        meta[r] = (ti, ei, arm)
    return Workload("study", list(traces), [tr.turns for tr in traces], p), meta


def dual_ablation(traces=None, envelope=FIDELITY_ENVELOPES[0]):
    """Sec. IV-B / Table V: SPEAR+TIDE with the unified register file (arm 0)
    and with dual copies refreshed after every request and gap (1), every 8
    requests (2) or at gap onsets (3), per trace."""
    traces = fidelity_traces() if traces is None else traces
    cells = [(ti, envelope, 0, sync, {"policy": POLICY_SPEAR, "tide": 1, "dual_sync": sync})
             for ti in range(len(traces)) for sync in (DUAL_NONE, DUAL_EVERY, DUAL_EIGHT, DUAL_GAP)]
    return _study_rows(traces, cells)


def component_ablation(traces=None, envelopes=ABLATION_ENVELOPES):
    """Scoring x tiering (the ablation beside Table IV): LRU, LRU+TIDE, SPEAR,
    SPEAR+TIDE, ETA, ETA+TIDE (arm = index in COMPONENTS) per trace and
    envelope."""
    traces = fidelity_traces() if traces is None else traces
    cells = [(ti, env, ei, a, {"policy": pol, "tide": tide})
             for ti in range(len(traces)) for ei, env in enumerate(envelopes)
             for a, (_, pol, tide) in enumerate(COMPONENTS)]
    return _study_rows(traces, cells)


def slot_sweep(traces=None, envelope=FIDELITY_ENVELOPES[0], slots=ASE_SLOTS):
    """eq. (ase): SPEAR+TIDE with N session slots (arm = index in slots) per
    trace."""
    traces = fidelity_traces() if traces is None else traces
    cells = [(ti, envelope, 0, a, {"policy": POLICY_SPEAR, "tide": 1, "n_slots": n})
             for ti in range(len(traces)) for a, n in enumerate(slots)]
    return _study_rows(traces, cells)
