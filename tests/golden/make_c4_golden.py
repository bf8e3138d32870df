"""Writes c4_prefix.json: the oracle's counters (both decision digests
included) for two simulations of the large-live-set workload (65,536
sessions, 160 KiB per token, SRAM 512 MiB, HBM 288 GiB, N_sess = 4,096)
after the first 100,000, 200,000, 300,000 and 400,000 events of its first
trace.  By 400,000 events about 63,000 sessions have arrived and the register
file holds about 57,000 entries.

Everything comes from oracle/ on the seeded trace of
paper_2609_09643_amd.synth (which draws data only).  The file also keeps a
SHA-256 of the trace's arrays, so that a changed generator is noticed before
any comparison.  Run from the repository root (about two minutes on eight
cores):

    python tests/golden/make_c4_golden.py
"""
import concurrent.futures as cf
import hashlib
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2609_09643_amd import synth  # noqa: E402

OUT = os.path.join(HERE, "c4_prefix.json")
SIMS = (0, 3)            # trace-fitted table with P = 5e8 us; flat table with P = 5e7 us
CHECKPOINTS = (100_000, 200_000, 300_000, 400_000)


def workload():
    return synth.c4_large(n_traces=1)


def trace_sha(tr):
    h = hashlib.sha256()
    for a in (tr.t_ns, tr.sid, tr.info, tr.length, tr.next_ns, tr.kvb):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def main():
    w = workload()
    tr = w.traces[0]
    D, N = oracle.luts_for(w)

    def one(job):
        sim, n = job
        row = w.params[sim]
        rc, cnt, _, st, _ = oracle.run(tr, row, D[int(row["lut"])], N[int(row["lut"])],
                                       max_events=n, states=True)
        assert rc == 0
        return sim, n, cnt, int(st[-1]["n_table"]), int(st[-1]["n_res"])

    jobs = [(s, n) for n in CHECKPOINTS[::-1] for s in SIMS]
    with cf.ThreadPoolExecutor(len(jobs)) as ex:     # the oracle releases the GIL
        res = list(ex.map(one, jobs))
    out = {"workload": "c4_large(n_traces=1): 65,536 sessions, %d events" % tr.n_events,
           "trace_sha256": trace_sha(tr), "sims": list(SIMS), "checkpoints": list(CHECKPOINTS),
           "counters": {}, "table_entries": {}, "residents": {}}
    for sim, n, cnt, n_table, n_res in sorted(res, key=lambda r: (r[1], r[0])):
        key = str(n)
        out["counters"].setdefault(key, []).append(
            {k: (float(v) if isinstance(v, float) else int(v)) for k, v in cnt.items()})
        out["table_entries"].setdefault(key, []).append(n_table)
        out["residents"].setdefault(key, []).append(n_res)
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", OUT, "table entries at the checkpoints:", out["table_entries"])


if __name__ == "__main__":
    main()
