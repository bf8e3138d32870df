"""GPU parity of the ranking-fidelity kernels (EMA replay, fp32 and fixed-point
scorers, Kendall tau-b pair counts) against the oracle: bit-exact."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def U():
    from paper_2609_09643_amd import unison
    return unison


@pytest.fixture(scope="module")
def rs():
    return synth.c5_ranking(n_snap=2000)


def dev(U, a, dt=None):
    return U._dev(a, dt)


def test_hazard_counts(U, rs):
    for pop in (rs.lut_pop, np.full(16, 12, np.uint32), np.arange(0, 300, dtype=np.uint32)):
        d, n = U.hazard_counts(dev(U, pop, np.uint32))
        od, on = oracle.hazard_counts(pop)
        assert np.array_equal(U._host(d, np.uint32), od)
        assert np.array_equal(U._host(n, np.uint32), on)


@pytest.mark.parametrize("b_g,tau", [(32, 1000), (24, 1000), (64, 1), (32, 1_000_000)])
def test_ema_replay_bit_exact(U, rs, b_g, tau):
    say("ema replay: %d sessions" % rs.turn.shape[0])
    g, gq = U.ema_replay(dev(U, rs.gaps_ns, np.uint64), dev(U, rs.n_hist), b_g, tau)
    og, ogq = oracle.ema_replay(rs.gaps_ns, rs.n_hist, b_g, tau)
    assert np.array_equal(U._host(g, np.uint32), og.view(np.uint32))
    assert np.array_equal(U._host(gq, np.uint64), ogq)


@pytest.mark.parametrize("penalty", [5e8, 5e7, 0.0])
def test_score_fp32_bit_exact(U, rs, penalty):
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, _ = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    out = U.score_fp32(dev(U, rs.turn), dev(U, g), dev(U, rs.done), dev(U, d, np.uint32),
                       dev(U, n, np.uint32), penalty)
    want = oracle.score_f32(rs.turn, g, rs.done, d, n, penalty)
    assert np.array_equal(U._host(out, np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("b_h,p_z", [(12, 500_000_000), (16, 500_000_000), (8, 50_000_000),
                                     (12, 1 << 50)])
def test_score_fixed_exact(U, rs, b_h, p_z):
    d, n = oracle.hazard_counts(rs.lut_pop)
    _, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    gq = gq.copy()
    gq[:64] = np.uint64(2 ** 64 - 1) - np.arange(64, dtype=np.uint64)   # u128 path
    out = U.score_fixed(dev(U, rs.turn), dev(U, gq, np.uint64), dev(U, rs.done),
                        dev(U, d, np.uint32), dev(U, n, np.uint32), b_h, p_z)
    want = oracle.score_fixed(rs.turn, gq, rs.done, d, n, b_h, p_z)
    assert np.array_equal(U._host(out, np.uint64), want)


@pytest.mark.parametrize("b_h,recip", [(12, 12), (12, 16), (12, 24), (16, 32), (8, 20), (10, 1)])
def test_score_fixed_reciprocal_divider_exact(U, rs, b_h, recip):
    d, n = oracle.hazard_counts(rs.lut_pop)
    _, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    gq = gq.copy()
    gq[:64] = np.uint64(2 ** 64 - 1) - np.arange(64, dtype=np.uint64)   # saturating products
    out = U.score_fixed(dev(U, rs.turn), dev(U, gq, np.uint64), dev(U, rs.done),
                        dev(U, d, np.uint32), dev(U, n, np.uint32), b_h, 500_000_000, recip)
    want = oracle.score_fixed(rs.turn, gq, rs.done, d, n, b_h, 500_000_000, recip_bits=recip)
    assert np.array_equal(U._host(out, np.uint64), want)


@pytest.mark.parametrize("n_per", [2, 3, 64, 65, 255, 257, 1000])
def test_kendall_small_with_ties(U, n_per):
    rng = np.random.default_rng(n_per)
    n_snap = 7
    x = rng.integers(0, max(2, n_per // 3), (n_snap, n_per)).astype(np.float32)
    y = rng.integers(0, max(2, n_per // 4), (n_snap, n_per)).astype(np.uint64)
    x[0] = np.inf
    y[1] = 2 ** 64 - 1
    c, t = U.kendall(dev(U, x.ravel()), dev(U, y.ravel(), np.uint64), None, n_snap, n_per)
    oc, ot = oracle.kendall(x, y)
    assert np.array_equal(U._host(c, np.uint64), oc)
    assert np.array_equal(t.cpu().numpy(), ot)


def test_kendall_ranking_snapshots(U, rs):
    """Snapshots of 4,096 resident sessions: fp32 scores against the locked
    fixed-point format; counts exact on a sample of snapshots."""
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    x = oracle.score_f32(rs.turn, g, rs.done, d, n, 5e8)
    y = oracle.score_fixed(rs.turn, gq, rs.done, d, n, 12, 500_000_000)
    say("kendall: %d snapshots x %d" % (rs.n_snap, rs.n_per))
    c, t = U.kendall(dev(U, x), dev(U, y, np.uint64), dev(U, rs.idx, np.uint32))
    c = U._host(c, np.uint64)
    t = t.cpu().numpy()
    assert np.all(c.sum(axis=1) == rs.n_per * (rs.n_per - 1) // 2)
    sample = np.arange(0, rs.n_snap, rs.n_snap // 24)
    oc, ot = oracle.kendall(x, y, idx=rs.idx[sample])
    assert np.array_equal(c[sample], oc)
    assert np.array_equal(t[sample], ot)


def test_kendall_ranking_snapshots_in_the_wide_form(U, rs):
    """The same snapshots with every fixed-point score other than 2^64 - 1
    shifted up 33 bits: order and ties are unchanged, so are tau-b's counts
    and the top-1 flags, but no snapshot packs into one 64-bit key.  Every
    snapshot must match the packed form's result, and a sample the oracle."""
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    x = oracle.score_f32(rs.turn, g, rs.done, d, n, 5e8)
    y = oracle.score_fixed(rs.turn, gq, rs.done, d, n, 12, 500_000_000).astype(np.uint64)
    top = np.uint64(2 ** 64 - 1)
    assert int(y[y != top].max()) < 2 ** 31
    yw = np.where(y == top, top, y << np.uint64(33)).astype(np.uint64)
    ys = yw[rs.idx]
    assert np.all(((ys != top) & (ys >= np.uint64(2 ** 32))).any(axis=1)), "a snapshot would pack"
    say("kendall, wide form: %d snapshots x %d" % (rs.n_snap, rs.n_per))
    idx = dev(U, rs.idx, np.uint32)
    cn, tn = U.kendall(dev(U, x), dev(U, y, np.uint64), idx)
    cw, tw = U.kendall(dev(U, x), dev(U, yw, np.uint64), idx)
    cw = U._host(cw, np.uint64)
    tw = tw.cpu().numpy()
    assert np.array_equal(cw, U._host(cn, np.uint64))
    assert np.array_equal(tw, tn.cpu().numpy())
    sample = np.arange(3, rs.n_snap, rs.n_snap // 12)
    oc, ot = oracle.kendall(x, yw, idx=rs.idx[sample])
    assert np.array_equal(cw[sample], oc)
    assert np.array_equal(tw[sample], ot)


@pytest.mark.parametrize("n_per", [256, 257, 1000, 2048, 4095, 4096])
def test_kendall_sorted_path_heavy_ties(U, n_per):
    """From 256 entries the counts come from sorting: few distinct values, the
    extremes of both scores, -0 beside +0, and padding to a power of two."""
    rng = np.random.default_rng(1000 + n_per)
    n_snap = 5
    x = rng.integers(0, 6, (n_snap, n_per)).astype(np.float32)
    y = rng.integers(0, 5, (n_snap, n_per)).astype(np.uint64)
    x[0, ::7] = np.inf
    x[1, ::5] = -0.0
    x[1, 1::5] = 0.0
    y[2, ::3] = 2 ** 64 - 1
    x[3] = rng.standard_normal(n_per).astype(np.float32)       # all distinct, both signs
    y[3] = rng.integers(0, 2 ** 63, n_per).astype(np.uint64)
    x[4] = 1.0                                                  # one x value
    c, t = U.kendall(dev(U, x.ravel()), dev(U, y.ravel(), np.uint64), None, n_snap, n_per)
    oc, ot = oracle.kendall(x, y)
    assert np.array_equal(U._host(c, np.uint64), oc)
    assert np.array_equal(t.cpu().numpy(), ot)


@pytest.mark.parametrize("n_per", [300, 4096])
def test_kendall_sorted_path_at_the_32_bit_key_boundary(U, n_per):
    """A snapshot packs (x, y) into one 64-bit key only while every y other
    than 2^64 - 1 lies below 2^32 - 1 (2^64 - 1 then stands in as 2^32 - 1):
    y values at 2^32 - 2, 2^32 - 1 and 2^32 beside 2^64 - 1, each snapshot on
    its side of the boundary, with ties in both scores."""
    rng = np.random.default_rng(7 + n_per)
    n_snap = 4
    x = rng.integers(0, 9, (n_snap, n_per)).astype(np.float32)
    top = np.array([2 ** 32 - 2, 2 ** 32 - 1, 2 ** 32, 2 ** 64 - 1], np.uint64)
    y = rng.integers(0, 6, (n_snap, n_per)).astype(np.uint64)
    y[0, ::4] = top[0]                      # narrow: the largest packed value
    y[0, 1::4] = top[3]
    y[1, ::4] = top[1]                      # wide: 2^32 - 1 is a real value
    y[1, 1::4] = top[3]
    y[2, ::3] = top[2]                      # wide
    y[2, 1::3] = top[0]
    y[3, ::5] = top[3]                      # narrow, only the done value above
    c, t = U.kendall(dev(U, x.ravel()), dev(U, y.ravel(), np.uint64), None, n_snap, n_per)
    oc, ot = oracle.kendall(x, y)
    assert np.array_equal(U._host(c, np.uint64), oc)
    assert np.array_equal(t.cpu().numpy(), ot)


def test_kendall_rejects_out_of_range_index(U):
    x = np.arange(10, dtype=np.float32)
    y = np.arange(10, dtype=np.uint64)
    idx = np.array([[0, 1, 2], [3, 4, 99]], np.uint32)
    c, t = U.kendall(dev(U, x), dev(U, y, np.uint64), dev(U, idx))
    assert t.cpu().numpy().tolist() == [1, 255]


def test_every_c5_snapshot_in_the_bench_pipeline(U):
    """The whole ranking-fidelity pass as bench.py times it (hazard counts,
    both EMA replays, both scorers, the sorted Kendall kernel) on all 10,000
    snapshots of 4,096 sessions, at b_h = 16 and 12: every snapshot's five
    pair counts and top-1 flag equal the oracle's, through the digests that
    tests/golden/make_c5_golden.py wrote with the oracle."""
    import os
    import sys as _sys
    here = os.path.dirname(os.path.abspath(__file__))
    _sys.path.insert(0, os.path.join(here, "golden"))
    import make_c5_golden as G
    gold = np.load(os.path.join(here, "golden", "c5_kendall.npz"))
    full = synth.c5_ranking()
    assert tuple(int(v) for v in gold["shape"]) == (full.n_snap, full.n_per)
    say("kendall: all %d snapshots x %d, two formats" % (full.n_snap, full.n_per))
    pop = dev(U, full.lut_pop, np.uint32)
    d, n = U.hazard_counts(pop)
    g, gq = U.ema_replay(dev(U, full.gaps_ns, np.uint64), dev(U, full.n_hist))
    x = U.score_fp32(dev(U, full.turn), g, dev(U, full.done), d, n, G.P_US)
    idx = dev(U, full.idx, np.uint32)
    for bh in G.FORMATS:
        y = U.score_fixed(dev(U, full.turn), gq, dev(U, full.done), d, n, bh, G.P_Z)
        c, t = U.kendall(x, y, idx)
        c = U._host(c, np.uint64)
        t = t.cpu().numpy()
        assert np.array_equal(c.sum(axis=0, dtype=np.uint64), gold["sum_bh%d" % bh])
        assert int(t.astype(np.uint64).sum()) == int(gold["top1_bh%d" % bh][0])
        bad = np.nonzero(G.snapshot_digests(c, t) != gold["digest_bh%d" % bh])[0]
        assert len(bad) == 0, "b_h %d: snapshots %s differ from the oracle" % (bh, bad[:8].tolist())
