"""GPU parity of the fixed-point format sweep (Sec. IV-C): score_q
trajectories at all 27 grid points and the fp32 reference against the
oracle (every counter), and the sweep's ranking statistics against the
oracle's scorers and pair counts."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import fidelity, synth
from parity import compare_counters, oracle_counters

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def test_all_formats_on_the_smallest_trace_match_the_oracle():
    tr = synth.fidelity_traces()[0]
    w, meta = synth.format_sweep(traces=[tr])
    say("format sweep parity: %d sims x %d events" % (w.n_sims, tr.n_events))
    from paper_2609_09643_amd.unison import Simulator
    s = Simulator(w)
    s.run()
    got = s.counters()
    compare_counters(got, oracle_counters(w), label="format sweep")
    d_hr, _, cells = fidelity.trajectory_drift(got, meta, 27)
    assert len(cells) == len(synth.FIDELITY_ENVELOPES) and np.all(np.isfinite(d_hr))


def test_ranking_statistics_match_the_oracle():
    rs = synth.fidelity_snapshots(n_snap=300)
    fmts = [(8, 24, 1), (10, 32, 1_000_000), (12, 32, 1000), (12, 64, 1)]
    say("ranking fidelity parity: %d snapshots x %d, %d formats" % (rs.n_snap, rs.n_per, len(fmts)))
    got = fidelity.ranking_fidelity(rs, fmts)
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, _ = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    x = oracle.score_f32(rs.turn, g, rs.done, d, n, 5e8)
    for (bh, bg, tau), (mtau, ptau, top1) in zip(fmts, got):
        _, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist, bg, tau)
        y = oracle.score_fixed(rs.turn, gq, rs.done, d, n, bh, 500_000_000_000 // tau)
        counts, t1 = oracle.kendall(x, y, rs.idx)
        tb = fidelity.tau_b(counts)
        assert mtau == pytest.approx(float(np.nanmean(tb)), rel=0, abs=0)
        assert ptau == pytest.approx(float(fidelity.tau_b(counts.sum(axis=0, keepdims=True))[0]),
                                     rel=0, abs=0)
        assert top1 == float((t1 == 1).mean())


def test_reciprocal_dividers_on_the_smallest_trace_match_the_oracle():
    """The divider-type axis: every grid point with each reciprocal-table
    width, whole-trace SPEAR+TIDE trajectories, every counter."""
    tr = synth.fidelity_traces()[0]
    fmts = [f for f in synth.format_grid_dividers() if f[3] != 0]
    w, meta = synth.format_sweep(traces=[tr], formats=fmts)
    say("divider sweep parity: %d sims x %d events" % (w.n_sims, tr.n_events))
    from paper_2609_09643_amd.unison import Simulator
    s = Simulator(w)
    s.run()
    compare_counters(s.counters(), oracle_counters(w), label="divider sweep")


def test_ranking_statistics_with_reciprocal_dividers_match_the_oracle():
    rs = synth.fidelity_snapshots(n_snap=300)
    fmts = [(12, 32, 1000, 12), (12, 32, 1000, 24), (8, 64, 1, 16)]
    got = fidelity.ranking_fidelity(rs, fmts)
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, _ = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    x = oracle.score_f32(rs.turn, g, rs.done, d, n, 5e8)
    for (bh, bg, tau, wb), (mtau, ptau, top1) in zip(fmts, got):
        _, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist, bg, tau)
        y = oracle.score_fixed(rs.turn, gq, rs.done, d, n, bh, 500_000_000_000 // tau, recip_bits=wb)
        counts, t1 = oracle.kendall(x, y, rs.idx)
        assert mtau == float(np.nanmean(fidelity.tau_b(counts)))
        assert top1 == float((t1 == 1).mean())
