"""Host replay of the register-table kernels' global index arithmetic (no GPU).

For every register-table shape -- G lanes per simulation and EPL sessions per
lane, the retired 64 x 24 included -- and the batches the GPU tests run
(the randomised batches as drawn before and after the ETA baseline existed,
and a subset of the sweep), this rebuilds what each thread of the launch
would touch: its lane group's simulation through the lane-group map, the
table rows tb + s of its sessions s = j G + lane and their KV sizes at
sb + s, its trace's events, and every session id the simulation reads at an
event or through a decision (victims, migrants, swaps), taken from the
oracle's decision logs.  Each index must lie inside its buffer and each
session id inside the lane/slot grid, as the kernel assumes."""
import numpy as np
import pytest

import oracle
from paper_2609_09643_amd import synth

SHAPES = {0: (16, 1), 1: (64, 1), 2: (64, 4), 4: (4, 4), 5: (8, 2), 6: (64, 24), 7: (16, 4),
          8: (32, 8)}
NONE = 0xFFFFFFFF
BLOCK = 256


def lane_group_map(params, lanes, policy_override=0xFF):
    """The launcher's lane-group -> simulation map: simulations sorted by
    (policy, score form, trace), a new wavefront where that changes, empty
    groups in between; None for the identity map."""
    n = params.shape[0]
    gpw = 64 // lanes
    if gpw == 1:
        return None
    pol = params["policy"] if policy_override == 0xFF else np.full(n, policy_override)
    mode = np.where(pol == synth.POLICY_SPEAR, params["score_mode"], 0)
    key = (pol.astype(np.int64) << 40) | (mode.astype(np.int64) << 32) | params["trace"].astype(np.int64)
    order = np.argsort(key, kind="stable")
    slots = []
    for j, i in enumerate(order):
        if j and key[i] != key[order[j - 1]]:
            while len(slots) % gpw:
                slots.append(NONE)
        slots.append(int(i))
    if len(slots) == n and all(s == k for k, s in enumerate(slots)):
        return None
    return np.array(slots, np.int64)


def replay(w, G, EPL, check_logs=True):
    n_sims = w.n_sims
    max_sess = max(t.n_sessions for t in w.traces)
    total_sess = sum(t.n_sessions for t in w.traces)
    ev_off = np.concatenate([[0], np.cumsum([t.n_events for t in w.traces])])
    ss_off = np.concatenate([[0], np.cumsum([t.n_sessions for t in w.traces])])
    slots = lane_group_map(w.params, G)
    n_slots = n_sims if slots is None else len(slots)
    blocks = (n_slots + BLOCK // G - 1) // (BLOCK // G)
    gtid = np.arange(blocks * BLOCK, dtype=np.int64)
    slot = gtid // G
    lane = gtid % G
    if slots is None:
        sim = slot
    else:
        sim = np.where(slot < n_slots, slots[np.minimum(slot, n_slots - 1)], NONE)
    live = sim < n_sims
    assert live.sum() == n_sims * G, "every simulation gets one lane group"
    for t_idx in range(n_sims):
        assert np.count_nonzero(sim == t_idx) == G
    held = 0
    for g_sim, g_lane in zip(sim[live], lane[live]):
        P = w.params[g_sim]
        tr = int(P["trace"])
        n_sess = w.traces[tr].n_sessions
        if n_sess > G * EPL:
            continue                     # the kernel flags the simulation instead
        tb = int(g_sim) * max_sess
        sb = int(ss_off[tr])
        s = np.arange(EPL, dtype=np.int64) * G + int(g_lane)
        s = s[s < n_sess]
        assert np.all(tb + s < n_sims * max_sess)
        assert np.all(sb + s < total_sess)
        held += s.size
        assert int(P["lut"]) < len(w.lut_pops) and tr + 1 < len(ev_off)
    assert held == sum(w.traces[int(p["trace"])].n_sessions for p in w.params
                       if w.traces[int(p["trace"])].n_sessions <= G * EPL)
    if not check_logs:
        return
    D, N = oracle.luts_for(w)
    for i in range(n_sims):
        P = w.params[i]
        tr = w.traces[int(P["trace"])]
        if tr.n_sessions > G * EPL:
            continue
        rc, _, log, _, _ = oracle.run(tr, P, D[int(P["lut"])], N[int(P["lut"])], log_cap=1 << 16)
        ids = np.concatenate([tr.sid, log["a"][log["a"] != NONE],
                              log["b"][(log["op"] == oracle.OP_SWAP)]]).astype(np.int64)
        assert np.all(ids < tr.n_sessions)
        assert np.all(ids // G < EPL) and np.all(ids % G < G)


def random_batch(seed, lo, hi, n_policies):
    import test_gpu_random as R
    return R.batch(seed, lo, hi, n_policies=n_policies)


@pytest.mark.parametrize("variant", sorted(SHAPES))
@pytest.mark.parametrize("name,seed,lo,hi", [("small", 71, 1, 16), ("medium", 72, 17, 64),
                                              ("large", 73, 65, 300)])
@pytest.mark.parametrize("n_policies", [4, 5])
def test_random_batches_stay_in_bounds(variant, name, seed, lo, hi, n_policies):
    G, EPL = SHAPES[variant]
    w = random_batch(seed, lo, hi, n_policies)
    if max(t.n_sessions for t in w.traces) > G * EPL and variant != 6:
        pytest.skip("the variant does not hold these traces")
    replay(w, G, EPL, check_logs=(variant == 6 and name == "large"))


@pytest.mark.parametrize("variant", sorted(SHAPES))
def test_sweep_subset_stays_in_bounds(variant):
    G, EPL = SHAPES[variant]
    c3 = synth.c3_sweep()
    sims = np.arange(0, c3.n_sims, 29)
    w = synth.Workload("c3", c3.traces, c3.lut_pops, c3.params[sims].copy(), c3.flat_luts)
    replay(w, G, EPL, check_logs=False)
