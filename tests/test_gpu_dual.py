"""GPU parity of the dual register-file design (eq. (rf), eq. (stale)) against
the oracle: every counter (Vict!= and Prom!= included) and decision logs, on
the hand-worked trace, a paper-shaped trace with TIDE and a C3 subset, across
a CONTINUE split; and the launcher's routing to streamed-table kernels."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth
from parity import compare_counters, oracle_counters, oracle_log, same_log
from test_oracle_dual import EVENTS
from tracekit import single_tier_params, trace_from_events

pytestmark = pytest.mark.gpu

SYNCS = (synth.DUAL_NONE, synth.DUAL_EVERY, synth.DUAL_EIGHT, synth.DUAL_GAP)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def Sim(*a, **k):
    from paper_2609_09643_amd.unison import Simulator
    return Simulator(*a, **k)


def test_hand_worked_trace_all_organisations():
    tr = trace_from_events(EVENTS, 3)
    p = np.concatenate([single_tier_params(synth.POLICY_SPEAR, slots=2) for _ in SYNCS])
    p["dual_sync"] = SYNCS
    zero = np.zeros(51, np.uint32)
    w = synth.Workload("dual_hand", [tr], [None], p, flat_luts=[(0, 0, 0)])
    s = Sim(w, log_cap=64)
    s.run(flags=2)
    compare_counters(s.counters(), oracle_counters(w), label="dual hand-worked")
    for i in range(w.n_sims):
        assert same_log(s.log(i), oracle_log(w, i, log_cap=64)), "sync %d log" % SYNCS[i]
    assert [int(x) for x in s.counters()["vict_diff"]] == [0, 1, 0, 1]


def paper_shaped_rows(n_traces=1):
    rows = []
    for ti in range(n_traces):
        for pol in (synth.POLICY_SPEAR, synth.POLICY_LRU, synth.POLICY_BELADY):
            for sync in SYNCS:
                p = synth.default_params(1)
                synth.set_policy(p, pol, tide=1)
                p["trace"], p["lut"] = ti, ti
                p["cap_sram_B"], p["cap_hbm_B"] = 10_000 * 128 * 1024, 50_000 * 128 * 1024
                p["dual_sync"] = sync
                rows.append(p[0])
    return np.array(rows, dtype=synth.SIM_PARAMS_DTYPE)


@pytest.mark.parametrize("variant", [None, 11])
def test_paper_shaped_trace_with_tide(variant):
    trs = synth.fidelity_traces()[:2]
    w = synth.Workload("dual_fid", trs, [t.turns for t in trs], paper_shaped_rows(2))
    say("dual paper-shaped: %d sims, variant %s" % (w.n_sims, variant))
    s = Sim(w, variant=variant)
    s.run()
    got = s.counters()
    compare_counters(got, oracle_counters(w), label="dual paper-shaped")
    assert int(got["vict_diff"].sum()) > 0 and int(got["prom_diff"].sum()) > 0


def test_c3_subset_and_continue():
    c3 = synth.c3_sweep()
    sims = list(range(0, c3.n_sims, 101))
    p = c3.params[np.asarray(sims)].copy()
    p["dual_sync"] = np.array(SYNCS, np.uint32)[np.arange(len(sims)) % 4]
    w = synth.Workload("dual_c3", c3.traces, c3.lut_pops, p, c3.flat_luts)
    say("dual c3: %d sims" % w.n_sims)
    s = Sim(w)
    s.run(max_events=150)
    compare_counters(s.counters(), oracle_counters(w, max_events=150), label="dual c3 prefix")
    s.run(flags=1)
    compare_counters(s.counters(), oracle_counters(w), label="dual c3 resumed")


def test_register_variants_refuse_dual_rows():
    from paper_2609_09643_amd.unison import E_INVALID, UnisonError
    tr = synth.tiny_trace()
    p = synth.default_params(1)
    p["cap_sram_B"], p["cap_hbm_B"] = 64 * synth.MIB, 2 * synth.GIB
    p["dual_sync"] = synth.DUAL_EVERY
    w = synth.Workload("dual_refuse", [tr], [tr.turns], p)
    s = Sim(w, variant=5)
    with pytest.raises(UnisonError) as e:
        s.run()
    assert e.value.code == E_INVALID
