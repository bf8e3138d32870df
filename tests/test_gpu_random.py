"""Randomised GPU parity against the oracle: seeded random traces (1 to 300
sessions, one to eight turns, per-session KV sizes, arrival rates from
sparse to crowded) under random parameter rows (every policy, TIDE on or
off, both score forms at random grid formats, tiny to ample capacities, slot
limits, TTLs, DMA rates, fixed or online hazard tables), each batch run on
every kernel variant that holds it.  Every counter must match."""
import sys

import numpy as np
import pytest

from paper_2609_09643_amd import synth
from parity import compare_counters, oracle_counters

pytestmark = pytest.mark.gpu

KIB, MIB, GIB = synth.KIB, synth.MIB, synth.GIB


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def Sim(*a, **k):
    from paper_2609_09643_amd.unison import Simulator
    return Simulator(*a, **k)


def random_trace(rng, n_sess):
    turns = rng.geometric(0.35, n_sess).clip(max=8)
    rate = float(rng.choice([0.5, 5.0, 50.0]))
    first = synth.poisson_arrivals(rng, n_sess, rate)
    gap_fn = synth.gaps_single if rng.random() < 0.5 else synth.gaps_mixture
    kvb = rng.choice(np.array([1, 64, 128, 160]) * KIB, n_sess)
    return synth.build_trace(rng, turns, first, gap_fn, kvb,
                             grow_lo=int(rng.integers(1, 200)), grow_hi=int(rng.integers(200, 3000)))


def random_rows(rng, n_traces, per_trace, n_luts, n_policies=5):
    formats = synth.format_grid()
    rows = []
    for ti in range(n_traces):
        for _ in range(per_trace):
            p = synth.default_params(1)
            pol = int(rng.integers(0, n_policies))
            synth.set_policy(p, pol, tide=int(rng.integers(0, 2)))
            p["trace"] = ti
            p["lut"] = int(rng.integers(0, n_luts))
            if pol == synth.POLICY_SPEAR and rng.random() < 0.4:
                bh, bg, tau = formats[int(rng.integers(len(formats)))]
                p["score_mode"], p["b_h"], p["b_g"], p["tau_ns"] = 1, bh, bg, tau
                p["p_z"] = int(round(5e8 * 1000 / tau))
            p["penalty_us"] = float(rng.choice([0.0, 5e7, 5e8]))
            p["cap_sram_B"] = int(rng.choice([0, 1, 16, 64, 512])) * MIB
            p["cap_hbm_B"] = int(rng.choice([0, 1, 4, 16, 64])) * GIB
            p["n_slots"] = int(rng.choice([1, 3, 16, 64, 1 << 20]))
            p["dma_B_per_us"] = int(rng.choice([1, 1000, 100_000, 10_000_000]))
            p["ttl_ns"] = int(rng.choice([1, 100, 2000, 30_000])) * 1_000_000
            if rng.random() < 0.25:
                p["hazard_online"] = 1
                p["online_sessions"] = int(rng.choice([0, 1, 5, 0xFFFFFFFF]))
            rows.append(p[0])
    return np.array(rows, dtype=synth.SIM_PARAMS_DTYPE)


def batch(seed, lo, hi, n_traces=24, per_trace=12, n_policies=5):
    """A randomised batch; n_policies = 4 draws the rows as before the ETA
    baseline existed (the batches the retired variant ran on)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    sizes = np.clip(np.floor(np.exp(rng.uniform(np.log(lo), np.log(hi + 1), n_traces))), lo, hi).astype(int)
    traces = [random_trace(rng, int(n)) for n in sizes]
    # the traces' own tables, a flat table and one fitted elsewhere
    pops = [t.turns for t in traces] + [None, synth.hazard_population(seed + 7, 128)]
    rows = random_rows(rng, len(traces), per_trace, len(pops), n_policies)
    flat = len(traces)
    return synth.Workload("random_%d" % seed, traces, pops, rows, flat_luts=[(flat,) + synth.FLAT_COUNTS])


BATCHES = {
    "small": (71, 1, 16, (None, 0, 4, 1, 3, 9, 12, 10)),
    "medium": (72, 17, 64, (None, 8, 2, 9, 12, 3)),
    "large": (73, 65, 300, (None, 9, 12, 10, 3)),
}
# Variant 6 (64 x 24) faulted the GPU on the large batch; it is retired and
# the library refuses it, so the case stays here, skipped.
RETIRED_LARGE = 6


@pytest.fixture(scope="module", params=sorted(BATCHES))
def case(request):
    seed, lo, hi, variants = BATCHES[request.param]
    w = batch(seed, lo, hi)
    say("random %s: %d traces of %d..%d sessions, %d sims, %d events" % (
        request.param, len(w.traces), lo, hi, w.n_sims, sum(t.n_events for t in w.traces)))
    return request.param, w, oracle_counters(w), variants


def test_random_batches_on_every_variant(case):
    name, w, want, variants = case
    for v in variants:
        say("random %s: variant %s" % (name, v))
        s = Sim(w, variant=v)
        s.run()
        compare_counters(s.counters(), want, label="random %s variant %s" % (name, v))
        del s


def test_random_batches_split_by_continue(case):
    """The same batches in three launches cut at uneven event counts, on
    the automatic choice and the streamed kernel: a resumed run is the
    uninterrupted one."""
    name, w, want, _ = case
    longest = max(t.n_events for t in w.traces)
    cuts = [max(1, longest // 7), max(1, longest // 3)]
    for v in (None, 10):
        say("random %s split %s: variant %s" % (name, cuts, v))
        s = Sim(w, variant=v)
        s.run(max_events=cuts[0])
        s.run(flags=1, max_events=cuts[1])
        s.run(flags=1)
        compare_counters(s.counters(), want, label="random %s split, variant %s" % (name, v))
        del s


def test_random_batches_with_few_cache_slots(case):
    """The streamed kernels with zero and one resident-cache slot per
    thread, across a CONTINUE: every thread with residents reads the table
    or refills its slot."""
    name, w, want, _ = case
    longest = max(t.n_events for t in w.traces)
    for v in (3, 10):
        for slots in (0, 1):
            say("random %s: variant %s, %d cache slots" % (name, v, slots))
            s = Sim(w, variant=v, cache_slots=slots)
            s.run(max_events=max(1, longest // 3))
            s.run(flags=1)
            compare_counters(s.counters(), want, label="random %s variant %s, %d slots" % (name, v, slots))
            del s


def test_random_batches_under_a_policy_override(case):
    """One policy for every row (unison_run's override), then the rows' own
    policies again on the same context: the register-table kernels regroup
    their simulations by policy, score form and trace for each."""
    import copy
    name, w, want, _ = case
    s = Sim(w)
    for pol in (synth.POLICY_LRU, synth.POLICY_BELADY, synth.POLICY_SPEAR):
        say("random %s: override %d" % (name, pol))
        w2 = copy.copy(w)
        w2.params = w.params.copy()
        w2.params["policy"] = pol
        s.run(policy=pol)
        compare_counters(s.counters(), oracle_counters(w2), label="random %s override %d" % (name, pol))
    s.run()
    compare_counters(s.counters(), want, label="random %s after overrides" % name)


def test_random_decision_logs(case):
    """Full ordered decision logs of a few simulations of each batch."""
    from parity import oracle_log, same_log
    name, w, _, _ = case
    s = Sim(w, log_cap=1 << 14)
    s.run(flags=2)
    for i in range(0, w.n_sims, 37):
        assert same_log(s.log(i), oracle_log(w, i, log_cap=1 << 14)), "random %s sim %d log" % (name, i)


@pytest.mark.skip(reason="variant 6 (64 x 24) is retired after a GPU fault on this batch; "
                         "no cause was found and the library refuses the variant")
def test_random_large_batch_on_the_retired_variant():
    seed, lo, hi, _ = BATCHES["large"]
    w = batch(seed, lo, hi)
    s = Sim(w, variant=RETIRED_LARGE)
    s.run()
    compare_counters(s.counters(), oracle_counters(w), label="random large variant 6")


@pytest.mark.parametrize("name", sorted(BATCHES))
def test_random_batches_on_the_slot_kernel(name):
    """The slot kernel holds residents in VGPR slots sized by N_sess (at
    most 512): the batches with N_sess capped there, in one launch and split
    by CONTINUE."""
    seed, lo, hi, _ = BATCHES[name]
    w = batch(seed, lo, hi)
    w.params["n_slots"] = np.minimum(w.params["n_slots"], 512)
    want = oracle_counters(w)
    say("random %s on the slot kernel: %d sims" % (name, w.n_sims))
    s = Sim(w, variant=13)
    s.run()
    compare_counters(s.counters(), want, label="random %s slot kernel" % name)
    longest = max(t.n_events for t in w.traces)
    s.run(max_events=max(1, longest // 5))
    s.run(flags=1)
    compare_counters(s.counters(), want, label="random %s slot kernel split" % name)


@pytest.mark.parametrize("name", sorted(BATCHES))
def test_random_batches_on_the_wide_kernel(name):
    """The wide-table kernel (table in the workspace, residents in LDS slots,
    the next entry loaded one event ahead): every batch, in one launch and
    split by CONTINUE."""
    seed, lo, hi, _ = BATCHES[name]
    w = batch(seed, lo, hi)
    want = oracle_counters(w)
    say("random %s on the wide kernel: %d sims" % (name, w.n_sims))
    s = Sim(w, variant=14)
    s.run()
    compare_counters(s.counters(), want, label="random %s wide kernel" % name)
    longest = max(t.n_events for t in w.traces)
    s.run(max_events=max(1, longest // 7))
    s.run(flags=1)
    compare_counters(s.counters(), want, label="random %s wide kernel split" % name)


def test_random_dual_rows():
    w = batch(74, 1, 120, n_traces=6, per_trace=8)
    rng = np.random.Generator(np.random.PCG64(75))
    w.params["dual_sync"] = rng.integers(0, 4, w.n_sims)
    say("random dual: %d sims" % w.n_sims)
    s = Sim(w)
    s.run()
    compare_counters(s.counters(), oracle_counters(w), label="random dual rows")
