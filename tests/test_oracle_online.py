"""The oracle's online hazard table (the convergence study beside
eq. (attainment)): pinned to the offline counts of eq. (hazard), to the
completion order read off the trace, and to the zero table it starts from."""
import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth

ZERO = np.zeros(51, np.uint32)


def row_for(policy=synth.POLICY_SPEAR, online=1, k=0xFFFFFFFF, score_mode=0):
    p = synth.default_params(1)
    synth.set_policy(p, policy)
    p["cap_sram_B"], p["cap_hbm_B"] = 64 * synth.MIB, 2 * synth.GIB
    p["hazard_online"], p["online_sessions"], p["score_mode"] = online, k, score_mode
    return p[0]


def done_order(tr):
    """Session ids in the order their DONE events occur."""
    return tr.sid[tr.kind == synth.KIND_DONE]


@pytest.fixture(scope="module")
def tr():
    return synth.fidelity_traces()[0]


def run_counts(tr, row, lut=(ZERO, ZERO), max_events=None):
    counts = np.zeros((2, 51), np.uint32)
    rc, cnt, _, _, _ = oracle.run(tr, row, lut[0], lut[1], counts=counts, max_events=max_events)
    assert rc == 0
    return cnt, counts


@pytest.mark.parametrize("score_mode", [0, 1])
def test_full_trace_counts_equal_the_offline_counts(tr, score_mode):
    _, counts = run_counts(tr, row_for(score_mode=score_mode))
    d, n = oracle.hazard_counts(tr.turns)
    assert np.array_equal(counts[0], d) and np.array_equal(counts[1], n)


@pytest.mark.parametrize("k", [1, 7, 40, 127])
def test_first_k_completions_are_counted(tr, k):
    _, counts = run_counts(tr, row_for(k=k))
    first = done_order(tr)[:k]
    d, n = oracle.hazard_counts(tr.turns[first])
    assert np.array_equal(counts[0], d) and np.array_equal(counts[1], n)
    assert counts[1][0] == k


def test_zero_sessions_is_the_zero_table(tr):
    on, _ = run_counts(tr, row_for(k=0))
    off, _ = run_counts(tr, row_for(online=0), lut=(ZERO, ZERO))
    assert on == off


def test_before_the_first_completion_the_online_run_is_the_zero_table(tr):
    first_done = int(np.nonzero(tr.kind == synth.KIND_DONE)[0][0])
    on, _ = run_counts(tr, row_for(), max_events=first_done)
    off, _ = run_counts(tr, row_for(online=0), max_events=first_done)
    assert on == off
    # one event later the table holds one session and the runs may part
    on1, c1 = run_counts(tr, row_for(), max_events=first_done + 1)
    assert c1[1][0] == 1


def test_offline_runs_report_their_own_table(tr):
    d, n = oracle.hazard_counts(tr.turns)
    _, counts = run_counts(tr, row_for(online=0), lut=(d, n))
    assert np.array_equal(counts[0], d) and np.array_equal(counts[1], n)


def test_attainment_arithmetic():
    from paper_2609_09643_amd import fidelity
    from paper_2609_09643_amd.unison import COUNTERS_DTYPE
    meta = np.zeros(4, synth.ATTAIN_META_DTYPE)
    meta[:] = [(0, synth.ATTAIN_LRU, 0), (0, synth.ATTAIN_OFFLINE, 9),
               (0, synth.ATTAIN_ONLINE, 0), (0, synth.ATTAIN_ONLINE, 9)]
    c = np.zeros(4, COUNTERS_DTYPE)
    c["requests"] = 100
    c["hit_hbm"] = [40, 60, 45, 60]          # LRU 0.40, offline 0.60
    curves, ref = fidelity.attainment(c, meta)
    assert ref[0] == (0.4, 0.6)
    assert [(n, round(a, 12)) for n, a, _ in curves[0]["online"]] == [(0, 0.25), (9, 1.0)]


def test_oracle_attainment_on_the_smallest_trace():
    """A(n) from oracle trajectories: one finite point per requested n for
    both tables, and the prefix table fitted on every completion is the
    offline table, so its point is exactly A = 1."""
    from paper_2609_09643_amd import fidelity
    from paper_2609_09643_amd.unison import COUNTERS_DTYPE
    trs = synth.fidelity_traces()[:1]
    w, meta = synth.attainment_workload(trs, points=[0, 32, 128])
    res, _ = oracle.run_workload(w)
    c = np.zeros(len(res), COUNTERS_DTYPE)
    for i, r in enumerate(res):
        for k, v in r.items():
            c[i][k] = v
    curves, ref = fidelity.attainment(c, meta)
    lru, off = ref[0]
    assert off != lru
    for kind in ("online", "prefix"):
        assert [n for n, _, _ in curves[0][kind]] == [0, 32, 128]
        assert all(np.isfinite(a) for _, a, _ in curves[0][kind])
    assert curves[0]["prefix"][-1][1] == 1.0
    # the prefix table over all sessions has the offline counts
    order = synth.completion_order(trs[0])
    assert sorted(order.tolist()) == list(range(trs[0].n_sessions))
