"""The fixed-point format sweep (Sec. IV-C): its grid and workloads, the drift
and Kendall arithmetic of the sweep driver, and the oracle's trajectories
at grid points other than the locked one (CPU only)."""
import numpy as np
import pytest
from scipy import stats

import oracle
from paper_2609_09643_amd import fidelity, synth
from paper_2609_09643_amd.unison import COUNTERS_DTYPE


def test_grid_has_27_distinct_points_and_the_locked_one():
    g = synth.format_grid()
    assert len(g) == 27 and len(set(g)) == 27
    assert synth.LOCKED_FORMAT in g
    assert {p[0] for p in g} == {8, 10, 12}
    assert {p[1] for p in g} == {24, 32, 64}
    assert {p[2] for p in g} == {1, 1000, 1_000_000}


def test_divider_axis_crosses_every_point_with_every_divider():
    g = synth.format_grid_dividers()
    assert len(g) == 27 * len(synth.FORMAT_DIVIDERS) and len(set(g)) == len(g)
    assert synth.LOCKED_FORMAT + (0,) in g
    w, meta = synth.format_sweep(traces=synth.fidelity_traces()[:1], formats=g)
    fixed = meta["fmt"] >= 0
    assert np.all(w.params["recip_bits"][~fixed] == 0)
    assert [int(r) for r in w.params["recip_bits"][fixed][:len(g)]] == [f[3] for f in g]


def test_reciprocal_divider_trajectories_are_consistent():
    """The oracle replays a whole trace with the reciprocal-table divider at
    each width: the counts that the trace fixes hold, and at W = 32 the
    decisions equal the exact divider's on this trace (every reciprocal then
    sits within 2^-33 of 1 / sigma_q)."""
    tr = synth.fidelity_traces()[0]
    fmts = [(12, 32, 1000, w) for w in (0, 12, 24, 32)]
    w, meta = synth.format_sweep(traces=[tr], envelopes=synth.FIDELITY_ENVELOPES[:1], formats=fmts)
    res, _ = oracle.run_workload(w)
    req = int(tr.turns.sum())
    for r in res:
        assert r["requests"] == req == r["hit_sram"] + r["hit_hbm"] + r["miss"]
    exact, w32 = res[1], res[4]
    assert exact["digest"] == w32["digest"] and exact["victim_digest"] == w32["victim_digest"]


def test_fidelity_traces_match_the_corpus_totals():
    trs = synth.fidelity_traces()
    assert [t.n_sessions for t in trs] == list(synth.FIDELITY_SESSIONS)
    assert sum(t.n_sessions for t in trs) == 1415
    assert sum(int(t.turns.sum()) for t in trs) == 33596
    for t in trs:
        assert t.n_events == 2 * int(t.turns.sum())
        assert np.all(np.diff(t.t_ns.astype(np.int64)) >= 0)


def test_sweep_rows_scale_the_penalty_by_tau():
    trs = synth.fidelity_traces()[:1]
    w, meta = synth.format_sweep(traces=trs)
    assert w.n_sims == len(synth.FIDELITY_ENVELOPES) * 28
    p = w.params
    fp32 = meta["fmt"] < 0
    assert np.all(p["score_mode"][fp32] == 0) and np.all(p["score_mode"][~fp32] == 1)
    grid = synth.format_grid()
    for r, m in zip(p, meta):
        s_tok, h_tok = synth.FIDELITY_ENVELOPES[int(m["envelope"])]
        assert int(r["cap_sram_B"]) == s_tok * 128 * 1024
        assert int(r["cap_hbm_B"]) == h_tok * 128 * 1024
        if int(m["fmt"]) >= 0:
            bh, bg, tau = grid[int(m["fmt"])]
            assert (int(r["b_h"]), int(r["b_g"]), int(r["tau_ns"])) == (bh, bg, tau)
            # P = 5e8 us = 5e11 ns; P_Z = P / tau
            assert int(r["p_z"]) * tau == 500_000_000_000


def test_drift_arithmetic():
    # two cells, one format: fp32 hit rates 0.5 and 0.25, score_q 0.502 and 0.25
    meta = np.zeros(4, synth.FORMAT_META_DTYPE)
    meta[:] = [(0, 0, -1), (0, 0, 0), (1, 0, -1), (1, 0, 0)]
    c = np.zeros(4, COUNTERS_DTYPE)
    c["requests"] = 1000
    c["hit_sram"] = [100, 102, 50, 50]
    c["hit_hbm"] = [400, 400, 200, 200]
    c["amat_sum_ns"] = [1e6, 1.01e6, 2e6, 2e6]
    d_hr, d_am, cells = fidelity.trajectory_drift(c, meta, 1)
    assert cells == [(0, 0), (1, 0)]
    assert np.allclose(d_hr[0], [0.2, 0.0])
    assert np.allclose(d_am[0], [1.0, 0.0])


def test_tau_b_from_pair_counts_matches_scipy():
    rng = np.random.default_rng(3)
    for n in (5, 17, 64):
        x = rng.integers(0, 6, n).astype(np.float32)
        y = (x + rng.integers(0, 3, n)).astype(np.uint64)
        counts, _ = oracle.kendall(x.reshape(1, n), y.reshape(1, n))
        want = stats.kendalltau(x, y.astype(np.float64), variant="b").statistic
        assert abs(fidelity.tau_b(counts)[0] - want) < 1e-12


@pytest.mark.parametrize("fmt", [(8, 24, 1), (10, 64, 1_000_000), (12, 32, 1000)])
def test_oracle_fixed_trajectories_at_grid_points(fmt):
    """The oracle's score_q trajectory at a grid point: decisions are
    complete and consistent (every request is a hit, a miss, or bypassed
    after a miss), and the locked point stays close to fp32 on this cell."""
    tr = synth.fidelity_traces()[0]
    w, meta = synth.format_sweep(traces=[tr], envelopes=synth.FIDELITY_ENVELOPES[:1], formats=[fmt])
    res, _ = oracle.run_workload(w)
    for r in res:
        assert r["error"] == 0
        assert r["requests"] == r["hit_sram"] + r["hit_hbm"] + r["miss"]
        assert r["bypass"] <= r["miss"]
        assert r["events"] == tr.n_events
    c = np.zeros(len(res), COUNTERS_DTYPE)
    for i, r in enumerate(res):
        for k, v in r.items():
            c[i][k] = v
    d_hr, _, _ = fidelity.trajectory_drift(c, meta, 1)
    assert np.all(np.isfinite(d_hr))
    if fmt == synth.LOCKED_FORMAT:
        assert abs(d_hr[0, 0]) <= 1.0
