"""The policy studies' arithmetic (Table V shifts, the scoring x tiering
ablation, eq. (ase)) on hand-made counters, and their workloads run through
the oracle (CPU only)."""
import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import studies, synth
from paper_2609_09643_amd.unison import COUNTERS_DTYPE


def counters(rows):
    c = np.zeros(len(rows), COUNTERS_DTYPE)
    for i, r in enumerate(rows):
        for k, v in r.items():
            c[i][k] = v
    return c


def test_dual_table_shifts():
    meta = np.zeros(2, synth.STUDY_META_DTYPE)
    meta[:] = [(0, 0, synth.DUAL_NONE), (0, 0, synth.DUAL_EIGHT)]
    c = counters([
        dict(requests=100, hit_sram=20, hit_hbm=30, tokens_total=1000, tokens_computed=600,
             amat_sum_ns=1000.0, evict=10),
        dict(requests=100, hit_sram=18, hit_hbm=30, tokens_total=1000, tokens_computed=650,
             amat_sum_ns=1100.0, evict=12, vict_diff=3, promote=3, swap=1, prom_diff=2)])
    (r,) = studies.dual_table(c, meta)
    assert r["sync"] == synth.DUAL_EIGHT
    assert r["vict_ne_pct"] == 25.0 and r["prom_ne_pct"] == 50.0
    assert r["d_hr_pp"] == pytest.approx(-2.0) and r["d_sram_pp"] == pytest.approx(-2.0)
    assert r["d_pre_pp"] == pytest.approx(-5.0) and r["d_amat_pct"] == pytest.approx(10.0)


def test_component_table():
    n_arms = len(synth.COMPONENTS)
    meta = np.zeros(n_arms, synth.STUDY_META_DTYPE)
    meta[:] = [(0, 0, a) for a in range(n_arms)]
    c = counters([dict(requests=10, hit_hbm=2, amat_sum_ns=100.0, tokens_total=10, tokens_computed=9)]
                 + [dict(requests=10, hit_hbm=4, amat_sum_ns=50.0, tokens_total=10, tokens_computed=5,
                         promote=4, swap=0, prefetch_hits=1)] * (n_arms - 1))
    t = studies.component_table(c, meta)
    assert t["lru"]["amat_over_lru"] == 1.0 and t["lru"]["prefetch_accuracy"] is None
    assert t["spear+tide"]["amat_over_lru"] == pytest.approx(0.5)
    assert t["lru+tide"]["prefetch_accuracy"] == 0.25
    assert t["spear"]["prefetch_accuracy"] is None          # no TIDE, no prefetch
    assert t["spear+tide"]["hr"] == pytest.approx(0.4) and t["lru"]["prered"] == pytest.approx(0.1)
    assert t["eta"]["prefetch_accuracy"] is None and t["eta+tide"]["prefetch_accuracy"] == 0.25


def test_ase_is_one_where_every_metric_peaks():
    slots = (8, 64)
    meta = np.zeros(4, synth.STUDY_META_DTYPE)
    meta[:] = [(d, 0, a) for d in range(2) for a in range(2)]
    # at N = 64 each trace has the higher hit rate and the lower AMAT and TTFT
    c = counters([dict(requests=10, hit_hbm=3, amat_sum_ns=200.0, ttft_sum_ns=400.0),
                  dict(requests=10, hit_hbm=6, amat_sum_ns=100.0, ttft_sum_ns=100.0)] * 2)
    (n8, a8), (n64, a64) = studies.ase(c, meta, slots)
    assert (n8, n64) == (8, 64) and a64 == pytest.approx(1.0)
    # (0.5 * 0.5 * 0.25)^(6/6) over the two traces' three ratios each
    assert a8 == pytest.approx((0.5 * 0.5 * 0.25) ** (2 / 6))


def oracle_counters(w):
    res, _ = oracle.run_workload(w)
    return counters(res)


def test_study_workloads_through_the_oracle():
    trs = synth.fidelity_traces()[:1]
    w, meta = synth.component_ablation(trs, synth.ABLATION_ENVELOPES[:2])
    c = oracle_counters(w)
    t = studies.component_table(c, meta)
    assert t["lru+tide"]["moves"] > 0 and t["spear+tide"]["moves"] > 0
    assert t["lru"]["moves"] == 0 and t["spear"]["moves"] == 0
    assert np.all(c["prefetch_hits"] <= c["promote"] + c["swap"])
    assert np.all(c["prefetch_hits"] <= c["hit_sram"])
    w, meta = synth.slot_sweep(trs, slots=(8, 64))
    pts = studies.ase(oracle_counters(w), meta, (8, 64))
    assert all(0 < v <= 1 for _, v in pts)
    w, meta = synth.dual_ablation(trs)
    rows = studies.dual_table(oracle_counters(w), meta)
    assert [r["sync"] for r in rows] == [1, 2, 3]
