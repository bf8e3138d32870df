"""GPU parity on the hand-worked TIDE traces (tests/tide_cases.py): every
kernel variant reproduces the decision list worked out by hand (and so the
oracle's), with its counters."""
import sys

import pytest

import tide_cases
from paper_2609_09643_amd import synth

pytestmark = pytest.mark.gpu

VARIANTS = (None, 0, 1, 2, 3, 4, 5, 7, 8, 9, 10, 11, 12, 13, 14)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("name", sorted(tide_cases.CASES))
def test_tide_worked_example_on_every_variant(name):
    from paper_2609_09643_amd.unison import Simulator
    tr, p, want_log, want, _ = tide_cases.CASES[name]()
    w = synth.Workload("tide_" + name, [tr], [None], p, flat_luts=[(0, 0, 1)])
    for v in VARIANTS:
        say("tide case %s, variant %s" % (name, v))
        s = Simulator(w, log_cap=256, variant=v)
        s.run(flags=2)
        c = s.counters()[0]
        got = [(int(r["ev"]), int(r["op"]), int(r["a"]), int(r["b"])) for r in s.log(0)]
        assert got == want_log, (name, v)
        for k, val in want.items():
            assert int(c[k]) == val, (name, v, k, int(c[k]), val)
        s.close()
