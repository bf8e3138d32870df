"""Pins of the oracle's ETA baseline (a tool-type arrival table: every session
that calls a tool is expected back after that tool's mean wait): the table
fitted by hand, a hand-worked trace on which the predicted and the true
returns disagree, its reduction to Belady when every tool has a single
latency, and the order it evicts in with a single tool class.  No GPU."""
import collections

import numpy as np
import pytest

import eta_cases
import oracle
from paper_2609_09643_amd import synth
from paper_2609_09643_amd.synth import (KIND_ARRIVE, KIND_DONE, KIND_GAP_START, POLICY_BELADY,
                                         POLICY_ETA)
from tracekit import single_tier_params, trace_from_events

H0 = (np.zeros(51, np.uint32), np.ones(51, np.uint32))


def run(tr, p, eta=None, log_cap=10000):
    rc, cnt, log, st, _ = oracle.run(tr, p[0], H0[0], H0[1], log_cap=log_cap, states=True, eta=eta)
    return rc, cnt, log, st


def decisions(log):
    return [(int(r["ev"]), int(r["op"]), int(r["a"]), int(r["b"])) for r in log]


def test_eta_table_fit_by_hand():
    """Class 0 gaps of 10 us and 20 us: mean 15,000 ns.  Class 1 gaps of 7, 8
    and 8 ns: floor(23 / 3) = 7.  Class 2: no gap, 0.  A DONE carries no gap."""
    A, G, D = KIND_ARRIVE, KIND_GAP_START, KIND_DONE
    ev = [(0, 0, A, 0, 1), (1000, 0, G, 0, 0), (11000, 0, A, 1, 1), (12000, 0, G, 1, 0),
          (32000, 0, A, 2, 1), (33000, 0, D, 2, 0),
          (40000, 1, A, 0, 1), (40001, 1, G, 0, 0), (40008, 1, A, 1, 1), (40010, 1, G, 1, 0),
          (40018, 1, A, 2, 1), (40020, 1, G, 2, 0), (40028, 1, A, 3, 1), (40030, 1, D, 3, 0)]
    tools = [0, 0, 0, 0, 0, 9, 0, 1, 0, 1, 0, 1, 0, 9]
    tr = trace_from_events(ev, 2, tools=tools)
    want = np.zeros(16, np.uint64)
    want[0], want[1] = 15000, 7
    assert np.array_equal(oracle.eta_table(tr), want)


@pytest.mark.parametrize("policy", ["eta", "belady"])
def test_predicted_and_true_returns_disagree(policy):
    tr, rows, want = eta_cases.predicted_and_true_returns_disagree()
    p = rows(POLICY_ETA if policy == "eta" else POLICY_BELADY)
    rc, cnt, log, _ = run(tr, p, eta=np.array(eta_cases.ETA_TABLE, np.uint64))
    assert rc == 0
    want_log, (req, miss, hits) = want[policy]
    assert decisions(log) == want_log
    assert (cnt["requests"], cnt["miss"], cnt["hit_hbm"]) == (req, miss, hits)


def fixed_latency_trace(rng, n_sess, turns, lat_ns):
    """Sessions whose every gap takes exactly its tool's latency; service times
    and first arrivals at random."""
    events, tools = [], []
    for s in range(n_sess):
        t = int(rng.integers(0, 50_000))
        for k in range(turns):
            t += 1
            events.append((t, s, KIND_ARRIVE, k, 1 + k))
            tools.append(0)
            t += int(rng.integers(100, 5000))
            last = k == turns - 1
            c = int(rng.integers(0, len(lat_ns)))
            events.append((t, s, KIND_DONE if last else KIND_GAP_START, k, 0))
            tools.append(0 if last else c)
            t += 0 if last else lat_ns[c] - 1
    order = sorted(range(len(events)), key=lambda i: (events[i][0], events[i][2] == KIND_ARRIVE,
                                                      events[i][1]))
    return trace_from_events([events[i] for i in order], n_sess, tools=[tools[i] for i in order])


@pytest.mark.parametrize("seed", range(6))
def test_eta_is_belady_when_every_tool_has_one_latency(seed):
    """When each tool class always takes the same time, the table's mean is
    that time and every predicted return is the true one: ETA's keys are
    Belady's, so every decision, hit and both digests agree (one tier or two,
    with TIDE or without)."""
    rng = np.random.default_rng(40 + seed)
    lat = [int(x) for x in rng.integers(1000, 400_000, 3)]
    tr = fixed_latency_trace(rng, int(rng.integers(3, 12)), int(rng.integers(2, 7)), lat)
    if seed % 2:
        p = single_tier_params(POLICY_ETA, int(rng.integers(1, 4)))
    else:
        p = synth.default_params(1)
        p["cap_sram_B"], p["cap_hbm_B"], p["n_slots"], p["dma_B_per_us"] = 8, 30, 6, 1000
        p["tide"] = 1
    fit = oracle.eta_table(tr)
    assert all(int(fit[c]) == lat[c] for c in range(3) if np.any(tr.tool[tr.kind == 1] == c))
    p["policy"] = POLICY_ETA
    rc_e, ce, le, _ = run(tr, p)
    p["policy"] = POLICY_BELADY
    rc_b, cb, lb, _ = run(tr, p)
    assert rc_e == rc_b == 0
    assert decisions(le) == decisions(lb)
    assert ce == cb


@pytest.mark.parametrize("seed", range(6))
def test_one_tool_class_evicts_the_latest_gap_onset(seed):
    """With one tool class every gap is predicted to last the same time, so
    the predicted return orders the sessions by their gap onset: ETA evicts a
    completed session first, else the evictable session whose gap began last
    (ties to the smaller id) -- the reverse of LRU among idle sessions."""
    rng = np.random.default_rng(70 + seed)
    n_sess = int(rng.integers(3, 8))
    m = int(rng.integers(1, n_sess))
    reqs = [int(x) for x in rng.integers(0, n_sess, 60)]
    from tracekit import trace_from_requests
    tr = trace_from_requests(reqs, n_sess, dt=int(rng.integers(2, 30)) * 1000)
    rc, cnt, log, _ = run(tr, single_tier_params(POLICY_ETA, m))
    assert rc == 0
    onset, done, res, pinned = {}, set(), set(), set()
    by_ev = collections.defaultdict(list)
    for r in log:
        by_ev[int(r["ev"])].append((int(r["op"]), int(r["a"])))
    checked = 0
    for e in range(tr.n_events):
        s, kind, now = int(tr.sid[e]), int(tr.kind[e]), int(tr.t_ns[e])
        if kind == KIND_ARRIVE:
            pinned.add(s)
            res.discard(s)
        else:
            pinned.discard(s)
            onset[s] = now
            if kind == KIND_DONE:
                done.add(s)
        for op, a in by_ev[e]:
            if op == oracle.OP_EVICT:
                cands = sorted(q for q in res if q not in pinned)
                if any(q in done for q in cands):
                    want = min(q for q in cands if q in done)
                else:
                    latest = max(onset[q] for q in cands)
                    want = min(q for q in cands if onset[q] == latest)
                assert a == want
                res.discard(a)
                checked += 1
            elif op == oracle.OP_PLACE:
                res.add(a)
    assert checked > 5


def test_tool_class_beyond_the_table_breaks_the_trace():
    A, G = KIND_ARRIVE, KIND_GAP_START
    ev = [(10, 0, A, 0, 1), (20, 0, G, 0, 0), (30, 0, A, 1, 1), (40, 0, G, 1, 0)]
    tr = trace_from_events(ev, 1, tools=[0, 3, 0, 16])
    rc, cnt, _, _ = run(tr, single_tier_params(POLICY_ETA, 2))
    assert rc == -2 and cnt["error"] == 4
