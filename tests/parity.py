"""Helpers that compare the HIP path with the oracle (test infrastructure)."""
import numpy as np

import oracle

# Floating-point counters: the oracle adds one f64 product per request in event
# order, the GPU rounds the products of exact integer totals once at the end.
# Both are the same real-valued sums; 1e-6 relative is the agreed bound.
FLOAT_FIELDS = ("amat_sum_ns", "ttft_sum_ns")
REL_TOL = 1e-6


def oracle_counters(workload, sims=None, max_events=None):
    res, _ = oracle.run_workload(workload, sims=sims, max_events=max_events)
    return res


def compare_counters(got_rows, want, sims=None, label=""):
    """got_rows: numpy COUNTERS_DTYPE rows; want: list of oracle dicts."""
    sims = list(range(len(want))) if sims is None else list(sims)
    bad = []
    for k, i in enumerate(sims):
        g, w = got_rows[i], want[k]
        for f, v in w.items():
            if f in FLOAT_FIELDS:
                gv = float(g[f])
                if abs(gv - v) > REL_TOL * max(1.0, abs(v)):
                    bad.append((i, f, gv, v))
            elif int(g[f]) != int(v):
                bad.append((i, f, int(g[f]), int(v)))
        if len(bad) > 20:
            break
    assert not bad, "%s: %d mismatches, first: %s" % (label, len(bad), bad[:8])


def oracle_log(workload, sim, log_cap=1 << 16, max_events=None):
    D, N = oracle.luts_for(workload)
    row = workload.params[sim]
    rc, _, log, _, _ = oracle.run(workload.traces[int(row["trace"])], row, D[int(row["lut"])],
                                  N[int(row["lut"])], log_cap=log_cap, max_events=max_events)
    return log


def same_log(a, b):
    return np.array_equal(np.asarray(a).view(np.uint32).reshape(-1, 4),
                          np.asarray(b).view(np.uint32).reshape(-1, 4))
