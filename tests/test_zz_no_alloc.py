"""The allocation-free entry point, unison_create_static, against
unison_create on the same inputs: two calls in a row, the second smaller,
each with every counter (both digests included) and the decision logs equal
to those of a context over a caller-allocated workspace; a context that a
later call superseded is refused; dims beyond the static array are refused
without creating anything."""
import sys

import numpy as np
import pytest

from paper_2609_09643_amd import synth
from parity import compare_counters, same_log

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def subset(w, sims):
    return synth.Workload(w.name, w.traces, w.lut_pops, w.params[np.asarray(sims)].copy(),
                          w.flat_luts)


def as_dicts(rows):
    return [{f: (float(r[f]) if f in ("amat_sum_ns", "ttft_sum_ns") else int(r[f]))
             for f in rows.dtype.names} for r in rows]


def both(w, log_cap=0, flags=0):
    from paper_2609_09643_amd.unison import Simulator
    ref = Simulator(w, log_cap=log_cap)
    ref.run(flags=flags)
    want = ref.counters().copy()
    logs = [ref.log(i).copy() for i in range(w.n_sims)] if log_cap else None
    ref.close()
    st = Simulator(w, log_cap=log_cap, static=True)
    st.run(flags=flags)
    return st, want, logs


def test_static_workspace_matches_the_allocated_one_twice_in_a_row():
    from paper_2609_09643_amd.unison import E_INVALID, UnisonError
    c3 = synth.c3_sweep()
    big = subset(c3, list(range(0, c3.n_sims, 2)))        # 8,192 simulations, 11.6 MiB
    say("static workspace: call 1, %d simulations" % big.n_sims)
    s1, want1, _ = both(big)
    compare_counters(s1.counters(), as_dicts(want1), label="static call 1")
    small = synth.c1_tiny()                               # 2 simulations, with logs
    say("static workspace: call 2, %d simulations" % small.n_sims)
    s2, want2, logs2 = both(small, log_cap=4096, flags=2)
    compare_counters(s2.counters(), as_dicts(want2), label="static call 2")
    for i in range(small.n_sims):
        assert same_log(s2.log(i), logs2[i]), "static call 2 sim %d log" % i
    # the first context's array now belongs to the second: it is refused
    with pytest.raises(UnisonError) as e:
        s1.run()
    assert e.value.code == E_INVALID and "superseded" in str(e.value)
    s2.run(flags=2)                                       # the live one still runs
    compare_counters(s2.counters(), as_dicts(want2), label="static call 2 again")
    s1.close()
    s2.close()


def test_static_workspace_refuses_dims_beyond_its_size():
    from paper_2609_09643_amd.unison import E_CAPACITY, Simulator, UnisonError
    c3 = synth.c3_sweep()
    w = subset(c3, [i % c3.n_sims for i in range(24_000)])  # 34 MiB of workspace
    with pytest.raises(UnisonError) as e:
        Simulator(w, static=True)
    assert e.value.code == E_CAPACITY and "static workspace" in str(e.value)
