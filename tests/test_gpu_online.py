"""GPU parity of the online hazard table (the convergence study beside
eq. (attainment)) against the oracle: every counter, and the counts each
simulation's table holds at the end, over register-table, LDS-table and
streamed-table kernels and across a CONTINUE split."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth
from parity import compare_counters

pytestmark = pytest.mark.gpu

CAPS = (0, 1, 3, 8, 0xFFFFFFFF)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def Sim(*a, **k):
    from paper_2609_09643_amd.unison import Simulator
    return Simulator(*a, **k)


def online(w, sims=None):
    p = (w.params if sims is None else w.params[np.asarray(sims)]).copy()
    p["hazard_online"] = 1
    p["online_sessions"] = np.array(CAPS, np.uint32)[np.arange(len(p)) % len(CAPS)]
    return synth.Workload(w.name + "_online", w.traces, w.lut_pops, p, w.flat_luts)


def oracle_with_counts(w, max_events=None):
    D, N = oracle.luts_for(w)
    cnts, counts = [], []
    for i in range(w.n_sims):
        row = w.params[i]
        c = np.zeros((2, 51), np.uint32)
        rc, cnt, _, _, _ = oracle.run(w.traces[int(row["trace"])], row, D[int(row["lut"])],
                                      N[int(row["lut"])], counts=c, max_events=max_events)
        assert rc == 0
        cnts.append(cnt)
        counts.append(c)
    return cnts, counts


def check(s, w, label, max_events=None):
    want, counts = oracle_with_counts(w, max_events)
    compare_counters(s.counters(), want, label=label)
    for i in range(w.n_sims):
        d, n = s.hazard(i)
        assert np.array_equal(d, counts[i][0]) and np.array_equal(n, counts[i][1]), \
            "%s sim %d: hazard counts differ" % (label, i)


@pytest.mark.parametrize("variant", [None, 0, 4, 7, 3, 9, 12, 10, 13, 14])
def test_c3_online_tables(variant):
    c3 = synth.c3_sweep()
    w = online(c3, list(range(0, c3.n_sims, 97)))
    say("online c3: %d sims, variant %s" % (w.n_sims, variant))
    s = Sim(w, variant=variant)
    s.run()
    check(s, w, "online c3 variant %s" % variant)


def test_paper_shaped_trace_online_all_policies_and_both_scores():
    tr = synth.fidelity_traces()[0]
    p = synth.default_params(10)
    for i in range(10):
        synth.set_policy(p[i:i + 1], i % 4)
    p["score_mode"][8:] = 1
    p["policy"][8:] = synth.POLICY_SPEAR
    p["tide"][8:] = 1
    p["cap_sram_B"], p["cap_hbm_B"] = 10_000 * 128 * 1024, 50_000 * 128 * 1024
    p["hazard_online"] = 1
    p["online_sessions"] = [0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 16, 16, 16, 16, 40,
                            0xFFFFFFFF]
    w = synth.Workload("online_fid", [tr], [tr.turns], p)
    say("online paper-shaped trace: %d sims x %d events" % (w.n_sims, tr.n_events))
    s = Sim(w)
    s.run()
    check(s, w, "online paper-shaped")
    d, n = oracle.hazard_counts(tr.turns)
    gd, gn = s.hazard(0)
    assert np.array_equal(gd, d) and np.array_equal(gn, n)


@pytest.mark.parametrize("variant", [None, 9, 12, 13, 14])
def test_online_table_survives_continue(variant):
    tr = synth.fidelity_traces()[1]
    w0 = synth.format_sweep(traces=[tr], envelopes=synth.FIDELITY_ENVELOPES[:1],
                            formats=[synth.LOCKED_FORMAT])[0]
    w = online(w0)
    first_done = int(np.nonzero(tr.kind == synth.KIND_DONE)[0][0])
    split = first_done + 500
    say("online continue: %d sims, split at event %d of %d" % (w.n_sims, split, tr.n_events))
    s = Sim(w, variant=variant)
    s.run(max_events=split)
    check(s, w, "online prefix", max_events=split)
    s.run(flags=1)
    check(s, w, "online resumed")


def test_fixed_tables_report_their_counts():
    w = synth.c1_tiny()
    s = Sim(w)
    s.run()
    d, n = oracle.hazard_counts(w.traces[0].turns)
    for i in range(w.n_sims):
        gd, gn = s.hazard(i)
        assert np.array_equal(gd, d) and np.array_equal(gn, n)


def test_attainment_batch_matches_the_oracle():
    from paper_2609_09643_amd import fidelity
    trs = synth.fidelity_traces()[:2]
    (curves, ref, c, w) = fidelity.run_attainment(trs)
    say("attainment parity: %d sims" % w.n_sims)
    want, _ = oracle_with_counts(w)
    compare_counters(c, want, label="attainment")
    assert set(curves) == {0, 1}
