"""Writes c5_kendall.npz: the oracle's Kendall pair counts and top-1 flags for
every snapshot of the ranking-fidelity workload (10,000 snapshots of 4,096
sessions), fp32 score against the fixed-point score at b_h = 16 and at the
locked b_h = 12 (eq. (lock)).

Everything here comes from oracle/ (hazard counts, both EMAs, both scores,
the pair counts) on the seeded inputs of paper_2609_09643_amd.synth, which
draws data only.  Per snapshot the file keeps an 8-byte BLAKE2b digest of its
five counts and its top-1 flag, plus the sums of each count over all
snapshots.  Run from the repository root:

    python tests/golden/make_c5_golden.py
"""
import concurrent.futures as cf
import hashlib
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2609_09643_amd import synth  # noqa: E402

OUT = os.path.join(HERE, "c5_kendall.npz")
FORMATS = (16, 12)
P_US, P_Z = 5e8, 500_000_000


def snapshot_digests(counts, top1):
    """8-byte BLAKE2b of each snapshot's 5 little-endian u64 counts and its
    top-1 byte, as uint64."""
    c = np.ascontiguousarray(counts, dtype="<u8")
    t = np.ascontiguousarray(top1, dtype=np.uint8)
    out = np.empty(c.shape[0], np.uint64)
    for s in range(c.shape[0]):
        h = hashlib.blake2b(c[s].tobytes() + t[s:s + 1].tobytes(), digest_size=8)
        out[s] = np.frombuffer(h.digest(), "<u8")[0]
    return out


def main(threads=os.cpu_count() or 1):
    rs = synth.c5_ranking()
    d, n = oracle.hazard_counts(rs.lut_pop)
    g, gq = oracle.ema_replay(rs.gaps_ns, rs.n_hist)
    x = oracle.score_f32(rs.turn, g, rs.done, d, n, P_US)
    res = {}
    for bh in FORMATS:
        y = oracle.score_fixed(rs.turn, gq, rs.done, d, n, bh, P_Z)
        blocks = np.array_split(np.arange(rs.n_snap), max(1, rs.n_snap // 100))
        with cf.ThreadPoolExecutor(threads) as ex:   # the oracle releases the GIL
            parts = list(ex.map(lambda b: oracle.kendall(x, y, idx=rs.idx[b]), blocks))
        counts = np.concatenate([p[0] for p in parts])
        top1 = np.concatenate([p[1] for p in parts])
        res["digest_bh%d" % bh] = snapshot_digests(counts, top1)
        res["sum_bh%d" % bh] = counts.sum(axis=0, dtype=np.uint64)
        res["top1_bh%d" % bh] = np.array([int(top1.sum())], np.uint64)
        print("b_h = %d: mean tau-b %.6f, top-1 %.4f" % (
            bh, float(np.nanmean(oracle.tau_b(counts))), float(top1.mean())), flush=True)
    res["shape"] = np.array([rs.n_snap, rs.n_per], np.uint64)
    np.savez(OUT, **res)
    print("wrote", OUT)


if __name__ == "__main__":
    main()
