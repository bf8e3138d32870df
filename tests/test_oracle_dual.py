"""The oracle's dual register files (eq. (rf), eq. (stale)): a hand-worked
trace on which the eviction engine's stale copy misses a completion, and
the identities that hold for any trace."""
import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth
from paper_2609_09643_amd.synth import KIND_ARRIVE as A, KIND_DONE as D, KIND_GAP_START as G
from tracekit import single_tier_params, trace_from_events

ZERO = np.zeros(51, np.uint32)
OP_EVICT = 1

# Two slots, one unbounded tier, h = 0 (score = gap EMA in us).
#   A and B each serve a first turn; A returns after a 5 ms gap (g = 1500),
#   B after a 9 ms gap (g = 2700) and opens a new gap; then A completes and C
#   arrives needing a slot.  The live file scores the completed A at S_max and
#   evicts it; a copy last refreshed before A's completion still sees A in
#   service with score 1500 < 2700 and evicts B, which then misses on return
#   and evicts A in turn.
EVENTS = [
    (1_000, 0, A, 0, 1), (2_000, 0, G, 0, 0),
    (3_000, 1, A, 0, 1), (4_000, 1, G, 0, 0),
    (5_002_000, 0, A, 1, 1),
    (9_004_000, 1, A, 1, 1), (9_005_000, 1, G, 1, 0),
    (9_006_000, 0, D, 1, 0),
    (9_007_000, 2, A, 0, 1), (9_008_000, 2, D, 0, 0),
    (12_000_000, 1, A, 2, 1), (12_001_000, 1, D, 2, 0),
]


def run(tr, row, log_cap=64):
    rc, cnt, log, _, _ = oracle.run(tr, row, ZERO, ZERO, log_cap=log_cap)
    assert rc == 0
    return cnt, log


@pytest.fixture(scope="module")
def tr():
    return trace_from_events(EVENTS, 3)


def row(sync):
    p = single_tier_params(synth.POLICY_SPEAR, slots=2)
    p["dual_sync"] = sync
    return p[0]


def evictions(log):
    return [(int(r["ev"]), int(r["a"])) for r in log if r["op"] == OP_EVICT]


def test_live_file_evicts_the_completed_session(tr):
    cnt, log = run(tr, row(synth.DUAL_NONE))
    assert evictions(log) == [(8, 0)]
    assert (cnt["requests"], cnt["hit_hbm"], cnt["miss"]) == (6, 3, 3)
    assert cnt["vict_diff"] == 0


@pytest.mark.parametrize("sync", [synth.DUAL_EVERY, synth.DUAL_GAP])
def test_stale_copy_evicts_the_other_session(tr, sync):
    cnt, log = run(tr, row(sync))
    # B's return then misses and takes A's slot (the live and the copied
    # choice agree there: A is completed, or outranks the never-copied C)
    assert evictions(log) == [(8, 1), (10, 0)]
    assert (cnt["requests"], cnt["hit_hbm"], cnt["miss"]) == (6, 2, 4)
    assert cnt["vict_diff"] == 1 and cnt["evict"] == 2


def test_never_synced_copy_ties_to_the_smallest_id(tr):
    # six requests: the every-8 copy is still the empty file, every score is
    # equal, and the tie goes to the smaller id -- here the live choice
    cnt, log = run(tr, row(synth.DUAL_EIGHT))
    assert evictions(log) == [(8, 0)]
    assert cnt["vict_diff"] == 0


@pytest.mark.parametrize("policy", [synth.POLICY_SPEAR, synth.POLICY_LRU, synth.POLICY_BELADY])
@pytest.mark.parametrize("sync", [synth.DUAL_EVERY, synth.DUAL_EIGHT, synth.DUAL_GAP])
def test_identities_on_a_random_trace(policy, sync):
    """Differing decisions are a subset of the decisions; the scan counts do
    not depend on the organisation; every request is still classified."""
    tr = synth.tiny_trace(seed=11, n_sessions=16, turns=12)
    p = synth.default_params(1)
    synth.set_policy(p, policy)
    p["cap_sram_B"], p["cap_hbm_B"] = 32 * synth.MIB, 2 * synth.GIB
    d, n = oracle.hazard_counts(tr.turns)
    live = oracle.run(tr, p[0], d, n)[1]
    p["dual_sync"] = sync
    rc, dual, _, _, _ = oracle.run(tr, p[0], d, n)
    assert rc == 0
    assert dual["vict_diff"] <= dual["evict"]
    assert dual["prom_diff"] <= dual["promote"] + dual["swap"]
    assert dual["requests"] == dual["hit_sram"] + dual["hit_hbm"] + dual["miss"]
    assert dual["requests"] == live["requests"] and dual["events"] == live["events"]
    assert live["vict_diff"] == 0 and live["prom_diff"] == 0
