"""GPU parity of the policy-study workloads (dual register files, scoring x
tiering, the session-capacity sweep) against the oracle: every counter."""
import sys

import pytest

from paper_2609_09643_amd import studies, synth
from parity import compare_counters, oracle_counters

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("study", ["dual_ablation", "component_ablation", "slot_sweep"])
def test_study_matches_the_oracle(study):
    trs = synth.fidelity_traces()[:2]
    w, meta = getattr(synth, study)(trs)
    print("%s: %d sims" % (study, w.n_sims), file=sys.stderr, flush=True)
    c = studies.run(w)
    compare_counters(c, oracle_counters(w), label=study)
