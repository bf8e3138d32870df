"""Pins of the oracle's event simulation (Algorithm 1 with SPEAR, TIDE and the
baselines) against things fixed outside it: textbook LRU and Belady MIN in
the single-tier, uniform-size setting; brute force over every eviction
choice; a hand-worked two-tier TIDE example; invariants checked by an
independent replay of the decision log.  No GPU."""
import collections
import itertools

import numpy as np
import pytest

import oracle
from oracle import OP_BYPASS, OP_EVICT, OP_EXPIRE, OP_PLACE, OP_PROMOTE, OP_SWAP
from paper_2609_09643_amd import synth
from paper_2609_09643_amd.synth import (KIND_ARRIVE, KIND_DONE, KIND_GAP_START, POLICY_BELADY,
                                         POLICY_LRU, POLICY_SPEAR, POLICY_TIMEOUT)
from tracekit import single_tier_params, trace_from_events, trace_from_requests

H0 = (np.zeros(51, np.uint32), np.ones(51, np.uint32))        # h = 0 everywhere


def run(trace, p, lut=H0, log_cap=10000, states=True, max_events=None):
    rc, cnt, log, st, _ = oracle.run(trace, p[0], lut[0], lut[1], log_cap=log_cap,
                                     states=states, max_events=max_events)
    return rc, cnt, log, st


def evictions(log):
    return [int(r["a"]) for r in log if r["op"] == OP_EVICT]


def random_requests(rng, n_sess, n_req):
    return [int(x) for x in rng.integers(0, n_sess, n_req)]


# ------------------------------------------------- textbook reductions

def lru_reference(reqs, m):
    cache, hits, victims = collections.OrderedDict(), 0, []
    for s in reqs:
        if s in cache:
            hits += 1
            cache.move_to_end(s)
        else:
            if len(cache) == m:
                victims.append(cache.popitem(last=False)[0])
            cache[s] = True
    return hits, victims


def min_reference(reqs, m):
    """Belady (1966): on a fault with a full cache evict the page whose next
    use is farthest away (never used again = infinitely far; ties to the
    smallest id)."""
    cache, hits, victims = set(), 0, []
    for i, s in enumerate(reqs):
        if s in cache:
            hits += 1
            continue
        if len(cache) == m:
            def nxt(q):
                for j in range(i + 1, len(reqs)):
                    if reqs[j] == q:
                        return j
                return float("inf")
            v = max(sorted(cache), key=lambda q: (nxt(q), -q))
            cache.remove(v)
            victims.append(v)
        cache.add(s)
    return hits, victims


@pytest.mark.parametrize("seed", range(12))
def test_lru_is_textbook_lru(seed):
    rng = np.random.default_rng(seed)
    n_sess, m = int(rng.integers(2, 8)), int(rng.integers(1, 5))
    reqs = random_requests(rng, n_sess, 60)
    rc, cnt, log, _ = run(trace_from_requests(reqs, n_sess), single_tier_params(POLICY_LRU, m))
    hits, victims = lru_reference(reqs, m)
    assert rc == 0
    assert cnt["hit_hbm"] == hits and cnt["hit_sram"] == 0
    assert evictions(log) == victims


@pytest.mark.parametrize("seed", range(12))
def test_belady_is_textbook_min(seed):
    rng = np.random.default_rng(100 + seed)
    n_sess, m = int(rng.integers(2, 8)), int(rng.integers(1, 5))
    reqs = random_requests(rng, n_sess, 60)
    rc, cnt, log, _ = run(trace_from_requests(reqs, n_sess), single_tier_params(POLICY_BELADY, m))
    hits, victims = min_reference(reqs, m)
    assert rc == 0
    assert cnt["hit_hbm"] == hits
    assert evictions(log) == victims


def brute_force_max_hits(reqs, m):
    best = 0

    def rec(i, cache, hits):
        nonlocal best
        if hits + (len(reqs) - i) <= best:
            return
        if i == len(reqs):
            best = max(best, hits)
            return
        s = reqs[i]
        if s in cache:
            rec(i + 1, cache, hits + 1)
        elif len(cache) < m:
            rec(i + 1, cache | {s}, hits)
        else:
            for v in sorted(cache):
                rec(i + 1, (cache - {v}) | {s}, hits)

    rec(0, frozenset(), 0)
    return best


@pytest.mark.parametrize("seed", range(10))
def test_no_policy_beats_brute_force_and_belady_reaches_it(seed):
    rng = np.random.default_rng(200 + seed)
    n_sess, m = int(rng.integers(3, 6)), int(rng.integers(1, 3))
    reqs = random_requests(rng, n_sess, 16)
    best = brute_force_max_hits(reqs, m)
    tr = trace_from_requests(reqs, n_sess, dt=int(rng.integers(5, 50)) * 1000)
    got = {}
    for pol in (POLICY_SPEAR, POLICY_LRU, POLICY_TIMEOUT, POLICY_BELADY):
        p = single_tier_params(pol, m)
        p["ttl_ns"] = 40_000
        rc, cnt, _, _ = run(tr, p)
        assert rc == 0
        got[pol] = cnt["hit_hbm"]
    assert got[POLICY_BELADY] == best
    assert all(v <= best for v in got.values())


def test_spear_h0_evicts_largest_gap_average():
    """With h = 0 the SPEAR score is the gap EMA itself (eq. (esp)), so the
    victim must be the evictable session with the largest EMA of its gaps,
    here recomputed in float64 from the trace times."""
    rng = np.random.default_rng(7)
    n_sess, m = 6, 3
    reqs = random_requests(rng, n_sess, 80)
    # irregular spacing so that the gaps differ
    events, t = [], 1000
    turn, last_end, ema, last_req = {}, {}, {}, {}
    for i, s in enumerate(reqs):
        last_req[s] = i
    for i, s in enumerate(reqs):
        t += int(rng.integers(1, 100)) * 1_000_000
        k = turn.get(s, 0)
        turn[s] = k + 1
        events.append((t, s, KIND_ARRIVE, k, 1))
        events.append((t + 1000, s, KIND_DONE if last_req[s] == i else KIND_GAP_START, k, 0))
        t += 1000
    tr = trace_from_events(events, n_sess)
    rc, cnt, log, _ = run(tr, single_tier_params(POLICY_SPEAR, m))
    assert rc == 0
    # replay to know the EMA and residency at each eviction
    by_ev = collections.defaultdict(list)
    for r in log:
        by_ev[int(r["ev"])].append(r)
    res, done = set(), set()
    checked = 0
    for e in range(tr.n_events):
        s, kind = int(tr.sid[e]), int(tr.kind[e])
        now = int(tr.t_ns[e])
        if kind == KIND_ARRIVE:
            if s in last_end:
                gap_us = (now - last_end[s]) / 1000.0
                ema[s] = 0.3 * gap_us + 0.7 * ema.get(s, 0.0)
            else:
                ema[s] = 0.0
        else:
            last_end[s] = now
            if kind == KIND_DONE:
                done.add(s)
        for r in by_ev[e]:
            a = int(r["a"])
            if r["op"] == OP_EVICT:
                cands = [q for q in res if q != s]
                if any(q in done for q in cands):
                    assert a in done
                else:
                    vals = sorted((ema[q] for q in cands), reverse=True)
                    if len(vals) < 2 or vals[0] - vals[1] > 1e-4 * vals[0]:
                        assert ema[a] == vals[0]
                        checked += 1
                res.discard(a)
            elif r["op"] == OP_PLACE:
                res.add(a)
            elif r["op"] == OP_BYPASS:
                res.discard(a)
    assert checked > 10


# ------------------------------------------------- hand-worked example

def test_tide_and_accounting_worked_example():
    """Three sessions, SRAM 10 B, HBM 100 B, 1 B/token, DMA 1 B/us, Belady
    keys (time of the next arrival).  Worked by hand:
      e0  s0 arrives (8)  miss, SRAM            e1 gap: EMA 0 -> budget 0
      e2  s1 arrives (5)  miss, SRAM full -> HBM
      e4  s2 arrives (3)  miss, 8+3 > 10 -> HBM
      e6  s1 returns (6)  HBM hit, gap 46 us -> EMA 13.8 us
      e7  s1 gap: budget 13 B.  p = s2 (next 60 us) cannot join SRAM alone;
          d = s0 (next 900 us): 60 < 900, 3+8 <= 13 -> swap; left 2 B.
          Then p = s0, d = s2: 900 < 60 fails -> stop.  DMA busy 11 us.
      e8  s2 returns (4)  SRAM hit              e9 gap at 61 us: DMA busy
      e10 s0 returns (9)  HBM hit   e12 s1 (7) HBM hit   e14 s2 (5) SRAM hit
    Costs t_s = 1, t_h = 10 ns/B, t_p = 100 ns/token (eq. (hr-amat)):
      AMAT sum 800+500+300+60+4+90+70+5 = 1829
      TTFT sum 800+500+300+150+103+180+160+104 = 2297"""
    A, G, D = KIND_ARRIVE, KIND_GAP_START, KIND_DONE
    ev = [(1000, 0, A, 0, 8), (2000, 0, G, 0, 0), (3000, 1, A, 0, 5), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 3), (6000, 2, G, 0, 0), (50000, 1, A, 1, 6), (51000, 1, G, 1, 0),
          (60000, 2, A, 1, 4), (61000, 2, G, 1, 0), (900000, 0, A, 1, 9), (901000, 0, D, 1, 0),
          (2000000, 1, A, 2, 7), (2001000, 1, D, 2, 0), (3000000, 2, A, 2, 5),
          (3001000, 2, D, 2, 0)]
    tr = trace_from_events(ev, 3)
    p = synth.default_params(1)
    p["policy"], p["tide"] = POLICY_BELADY, 1
    p["cap_sram_B"], p["cap_hbm_B"], p["n_slots"], p["dma_B_per_us"] = 10, 100, 10, 1
    p["t_s_ns_per_B"], p["t_h_ns_per_B"], p["t_p_ns_per_tok"] = 1.0, 10.0, 100.0
    rc, cnt, log, st = run(tr, p)
    assert rc == 0
    S, H = oracle.TIER_SRAM, oracle.TIER_HBM
    want = [(0, OP_PLACE, 0, S), (2, OP_PLACE, 1, H), (4, OP_PLACE, 2, H), (6, OP_PLACE, 1, H),
            (7, OP_SWAP, 2, 0), (8, OP_PLACE, 2, S), (10, OP_PLACE, 0, H),
            (12, OP_PLACE, 1, H), (14, OP_PLACE, 2, S)]
    assert [(int(r["ev"]), int(r["op"]), int(r["a"]), int(r["b"])) for r in log] == want
    assert (cnt["requests"], cnt["miss"], cnt["hit_sram"], cnt["hit_hbm"]) == (8, 3, 2, 3)
    assert (cnt["swap"], cnt["promote"], cnt["dma_bytes"], cnt["tide_passes"]) == (1, 0, 11, 4)
    assert int(st[7]["tide_budget"]) == 13 and int(st[7]["tide_moved"]) == 11
    assert st[9]["tide_ran"] == 0
    assert cnt["amat_sum_ns"] == 1829.0 and cnt["ttft_sum_ns"] == 2297.0
    assert (cnt["tokens_total"], cnt["tokens_computed"], cnt["extra_prefill_tok"]) == (47, 21, 0)
    # the scan covers the table: 1,1,2,2,3,3,3,... entries; residents are counted apart
    assert cnt["score_evals"] == 1 + 1 + 2 + 2 + 3 * 12
    assert cnt["events"] == 16


def test_bypass_oversized_without_eviction():
    A, G = KIND_ARRIVE, KIND_GAP_START
    ev = [(10, 0, A, 0, 50), (20, 0, G, 0, 0), (30, 1, A, 0, 500), (40, 1, G, 0, 0)]
    p = synth.default_params(1)
    p["policy"], p["tide"] = POLICY_LRU, 0
    p["cap_sram_B"], p["cap_hbm_B"] = 10, 100
    rc, cnt, log, _ = run(trace_from_events(ev, 2), p)
    assert rc == 0 and cnt["bypass"] == 1 and cnt["evict"] == 0
    assert [int(r["op"]) for r in log] == [OP_PLACE, OP_BYPASS]


def test_miss_after_loss_counts_extra_prefill():
    A, G, D = KIND_ARRIVE, KIND_GAP_START, KIND_DONE
    ev = [(10, 0, A, 0, 50), (20, 0, G, 0, 0), (30, 1, A, 0, 60), (40, 1, G, 0, 0),
          (50, 0, A, 1, 70), (60, 0, D, 1, 0)]
    p = single_tier_params(POLICY_LRU, 1)
    p["t_p_ns_per_tok"] = 2.0
    rc, cnt, log, _ = run(trace_from_events(ev, 2), p)
    # s0 is evicted for s1, then misses again and re-prefills its 50-token prefix
    assert evictions(log) == [0, 1]
    assert cnt["miss"] == 3 and cnt["extra_prefill_tok"] == 50
    assert cnt["tokens_computed"] == 50 + 60 + 70 and cnt["amat_sum_ns"] == 2.0 * 180


def test_timeout_expires_idle_sessions():
    A, G, D = KIND_ARRIVE, KIND_GAP_START, KIND_DONE
    ev = [(0, 0, A, 0, 1), (10, 0, G, 0, 0), (20, 1, A, 0, 1), (30, 1, G, 0, 0),
          (5011, 2, A, 0, 1), (5020, 2, D, 0, 0), (9000, 1, A, 1, 1), (9010, 1, D, 1, 0)]
    p = single_tier_params(POLICY_TIMEOUT, 10)
    p["ttl_ns"] = 5000
    rc, cnt, log, _ = run(trace_from_events(ev, 3), p)
    # at t=5011 s0 (idle since 10) has waited 5001 > 5000; s1 (since 30) has not
    expired = [(int(r["ev"]), int(r["a"])) for r in log if r["op"] == OP_EXPIRE]
    assert expired == [(4, 0), (6, 1)]
    assert cnt["expire"] == 2 and cnt["miss"] == 4 and cnt["hit_hbm"] == 0


def test_slot_limit_binds():
    A, G = KIND_ARRIVE, KIND_GAP_START
    ev = [(10, 0, A, 0, 1), (20, 0, G, 0, 0), (30, 1, A, 0, 1), (40, 1, G, 0, 0)]
    p = single_tier_params(POLICY_SPEAR, 1)
    rc, cnt, log, st = run(trace_from_events(ev, 2), p)
    assert evictions(log) == [0] and max(st["n_res"]) == 1


def test_pinned_sessions_are_never_victims():
    # both sessions are in service when s2 arrives: nothing can be evicted
    A, G = KIND_ARRIVE, KIND_GAP_START
    ev = [(10, 0, A, 0, 1), (20, 1, A, 0, 1), (30, 2, A, 0, 1), (40, 0, G, 0, 0),
          (50, 1, G, 0, 0), (60, 2, G, 0, 0)]
    rc, cnt, log, _ = run(trace_from_events(ev, 3), single_tier_params(POLICY_LRU, 2))
    assert cnt["bypass"] == 1 and cnt["evict"] == 0


@pytest.mark.parametrize("bad", ["sid", "turn", "time", "double_start", "end_without_arrive"])
def test_bad_traces_are_rejected(bad):
    A, G = KIND_ARRIVE, KIND_GAP_START
    ev = [(10, 0, A, 0, 1), (20, 0, G, 0, 0), (30, 0, A, 1, 2), (40, 0, G, 1, 0)]
    if bad == "sid":
        ev[2] = (30, 5, A, 1, 2)
    elif bad == "turn":
        ev[2] = (30, 0, A, 2, 2)
    elif bad == "time":
        ev[2] = (15, 0, A, 1, 2)
    elif bad == "double_start":
        ev[2] = (30, 0, A, 0, 2)
    else:
        ev[1] = (20, 1, G, 0, 0)
    tr = trace_from_events(ev, 2)
    rc, cnt, _, _ = run(tr, single_tier_params(POLICY_LRU, 4))
    assert rc == -2 and cnt["error"] > 0


# ---------------------------------------------- invariants by replay

def replay_check(tr, p, log, st, cnt):
    """Re-applies the logged decisions to an independent residency model and
    checks eq. (cap), pinning, TIDE legality and the bookkeeping."""
    C_S, C_H, slots = int(p["cap_sram_B"]), int(p["cap_hbm_B"]), int(p["n_slots"])
    kvb = tr.kvb.astype(np.int64)
    tier, size, length = {}, {}, {}
    pinned, done = set(), set()
    by_ev = collections.defaultdict(list)
    for r in log:
        by_ev[int(r["ev"])].append((int(r["op"]), int(r["a"]), int(r["b"])))
    req = hit = miss = 0
    for e in range(len(st)):
        s, kind = int(tr.sid[e]), int(tr.kind[e])
        ops = by_ev[e]
        for op, a, b in ops:                      # TTL timers fire before the event
            if op == OP_EXPIRE:
                assert a in tier and a not in pinned
                del tier[a]
        if kind == KIND_ARRIVE:
            pinned.add(s)
        else:
            pinned.discard(s)
            if kind == KIND_DONE:
                done.add(s)
        # this event's scan result: an evictable resident, or none when all are pinned
        v = int(st[e]["victim"])
        if v != oracle.NONE_ID:
            assert v in tier and v not in pinned
        else:
            assert all(q in pinned for q in tier)
        if kind == KIND_ARRIVE:
            req += 1
            if s in tier:
                hit += 1
                del tier[s]
            else:
                miss += 1
            length[s] = int(tr.length[e])
        for op, a, b in ops:
            if op == OP_PLACE:
                assert kind == KIND_ARRIVE and a == s and b in (1, 2) and a not in tier
                tier[a], size[a] = b, length[a] * int(kvb[a])
            elif op == OP_BYPASS:
                assert kind == KIND_ARRIVE and a == s and a not in tier
            elif op == OP_EVICT:
                assert a in tier and a not in pinned
                del tier[a]
            elif op == OP_PROMOTE:
                assert kind == KIND_GAP_START and tier.get(a) == 2 and a not in pinned
                tier[a] = 1
            elif op == OP_SWAP:
                assert kind == KIND_GAP_START and tier.get(a) == 2 and tier.get(b) == 1
                assert a not in pinned and b not in pinned and a not in done
                tier[a], tier[b] = 1, 2
        if kind == KIND_ARRIVE:
            assert sum(1 for op, a, _ in ops if a == s and op in (OP_PLACE, OP_BYPASS)) == 1
        used_s = sum(size[q] for q, t in tier.items() if t == 1)
        used_h = sum(size[q] for q, t in tier.items() if t == 2)
        assert used_s <= C_S and used_h <= C_H and len(tier) <= slots
        assert (used_s, used_h, len(tier)) == (int(st[e]["used_sram"]), int(st[e]["used_hbm"]),
                                              int(st[e]["n_res"]))
        assert int(st[e]["tide_moved"]) <= int(st[e]["tide_budget"])
    assert req == cnt["requests"] and hit == cnt["hit_sram"] + cnt["hit_hbm"]
    assert miss == cnt["miss"]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("policy", [POLICY_SPEAR, POLICY_LRU, POLICY_TIMEOUT, POLICY_BELADY])
def test_invariants_random_two_tier(seed, policy):
    rng = np.random.default_rng(1000 + seed)
    tr = synth.tiny_trace(seed=50 + seed, n_sessions=int(rng.integers(3, 20)),
                          turns=int(rng.integers(1, 9)))
    p = synth.default_params(1)
    p["policy"] = policy
    p["tide"] = int(rng.integers(0, 2))
    p["cap_sram_B"] = int(rng.choice([0, 64, 256, 1024])) * synth.MIB
    p["cap_hbm_B"] = int(rng.choice([1, 2, 4, 16])) * synth.GIB
    p["n_slots"] = int(rng.integers(1, 12))
    p["ttl_ns"] = int(rng.choice([1, 3, 10])) * synth.NS
    p["dma_B_per_us"] = int(rng.choice([1000, 100_000, 10_000_000]))
    d, n = oracle.hazard_counts(synth.hazard_population(seed, 64))
    rc, cnt, log, st = run(tr, p, lut=(d, n), log_cap=100000)
    assert rc == 0
    assert cnt["requests"] == int(tr.turns.sum()) == cnt["hit_sram"] + cnt["hit_hbm"] + cnt["miss"]
    assert cnt["miss"] - tr.n_sessions <= cnt["evict"] + cnt["expire"] + cnt["bypass"]
    replay_check(tr, p[0], log, st, cnt)


def test_digest_covers_decisions_and_is_deterministic():
    w = synth.c1_tiny()
    D, N = oracle.luts_for(w)
    a = oracle.run(w.traces[0], w.params[0], D[0], N[0], log_cap=5000)
    b = oracle.run(w.traces[0], w.params[0], D[0], N[0], log_cap=5000)
    assert a[1] == b[1]
    c = oracle.run(w.traces[0], w.params[1], D[0], N[0], log_cap=5000)
    assert c[1]["digest"] != a[1]["digest"]


def test_prefix_runs_agree_with_full_run():
    w = synth.c1_tiny()
    D, N = oracle.luts_for(w)
    _, full, flog, fst, _ = oracle.run(w.traces[0], w.params[0], D[0], N[0], log_cap=5000,
                                       states=True)
    _, pre, plog, pst, _ = oracle.run(w.traces[0], w.params[0], D[0], N[0], log_cap=5000,
                                      states=True, max_events=100)
    assert pre["events"] == 100
    assert np.array_equal(pst, fst[:100])
    assert np.array_equal(plog, flog[flog["ev"] < 100])
