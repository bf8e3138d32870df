"""Policy studies on the batched simulation: the unified-versus-dual register
file ablation (Sec. IV-B, Table V), the scoring x tiering ablation with
prefetch accuracy, and Agent Serving Effectiveness over the session capacity
(eq. (ase)).  Each study is one launch of libunison; this module turns the
counters into the paper's rates.
"""
from __future__ import annotations

import numpy as np

from . import synth
from . import unison as U
from .fidelity import hit_rate, mean_amat


def sram_rate(c):
    return c["hit_sram"].astype(np.float64) / np.maximum(c["requests"].astype(np.float64), 1)


def prefill_reduction(c):
    """eq. (prered): 1 - tokens prefilled / tokens requested."""
    return 1.0 - c["tokens_computed"].astype(np.float64) / np.maximum(
        c["tokens_total"].astype(np.float64), 1)


def mean_ttft(c):
    return c["ttft_sum_ns"] / np.maximum(c["requests"].astype(np.float64), 1)


def prefetch_accuracy(c):
    """Share of TIDE's moves into SRAM that its session's next request finds
    there; nan without moves."""
    moves = (c["promote"] + c["swap"]).astype(np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(moves > 0, c["prefetch_hits"].astype(np.float64) / moves, np.nan)


def run(workload):
    sim = U.Simulator(workload)
    sim.run()
    return sim.counters()


def dual_table(c, meta):
    """Per trace and dual schedule (1, 2, 3): Vict!= and Prom!= (% of the dual
    run's evictions / TIDE moves), and the shifts against the unified run:
    hit rate, SRAM hit rate and prefill reduction in pp, AMAT in %."""
    hr, sr, pre, am = hit_rate(c), sram_rate(c), prefill_reduction(c), mean_amat(c)
    base = {int(m["trace"]): i for i, m in enumerate(meta) if int(m["arm"]) == synth.DUAL_NONE}
    rows = []
    for i, m in enumerate(meta):
        arm = int(m["arm"])
        if arm == synth.DUAL_NONE:
            continue
        b = base[int(m["trace"])]
        moves = int(c["promote"][i] + c["swap"][i])
        rows.append({"trace": int(m["trace"]), "sync": arm,
                     "vict_ne_pct": 100.0 * int(c["vict_diff"][i]) / max(int(c["evict"][i]), 1),
                     "prom_ne_pct": 100.0 * int(c["prom_diff"][i]) / max(moves, 1),
                     "d_hr_pp": 100.0 * (hr[i] - hr[b]), "d_sram_pp": 100.0 * (sr[i] - sr[b]),
                     "d_pre_pp": 100.0 * (pre[i] - pre[b]),
                     "d_amat_pct": 100.0 * (am[i] - am[b]) / am[b] if am[b] else 0.0})
    return rows


def component_table(c, meta):
    """Per component (LRU, LRU+TIDE, SPEAR, SPEAR+TIDE, ETA, ETA+TIDE): hit rate and prefill
    reduction averaged over traces and envelopes, AMAT relative to LRU as a
    geometric mean of per-cell ratios, and the prefetch accuracy of the
    TIDE arms over all their moves."""
    hr, pre, am = hit_rate(c), prefill_reduction(c), mean_amat(c)
    lru = {(int(m["trace"]), int(m["envelope"])): i for i, m in enumerate(meta) if int(m["arm"]) == 0}
    out = {}
    for a, (name, _, tide) in enumerate(synth.COMPONENTS):
        idx = [i for i, m in enumerate(meta) if int(m["arm"]) == a]
        ratios = [am[i] / am[lru[(int(meta[i]["trace"]), int(meta[i]["envelope"]))]] for i in idx]
        moves = int(sum(int(c["promote"][i] + c["swap"][i]) for i in idx))
        hits = int(sum(int(c["prefetch_hits"][i]) for i in idx))
        out[name] = {"hr": float(np.mean(hr[idx])), "prered": float(np.mean(pre[idx])),
                     "amat_over_lru": float(np.exp(np.mean(np.log(ratios)))),
                     "prefetch_accuracy": (hits / moves) if (tide and moves) else None,
                     "moves": moves}
    return out


def ase(c, meta, slots=synth.ASE_SLOTS):
    """eq. (ase): ASE(N) = (prod over traces d of HR_d / max HR_d *
    min AMAT_d / AMAT_d * min TTFT_d / TTFT_d)^(1 / (3 * traces)), the
    extremes taken over the capacity sweep.  Returns [(N, ASE(N))]."""
    hr, am, tt = hit_rate(c), mean_amat(c), mean_ttft(c)
    traces = sorted({int(m["trace"]) for m in meta})
    grid = {(int(m["trace"]), int(m["arm"])): i for i, m in enumerate(meta)}
    logs = np.zeros(len(slots))
    for d in traces:
        ii = [grid[(d, a)] for a in range(len(slots))]
        h, a_, t = hr[ii], am[ii], tt[ii]
        logs += np.log(h / h.max()) + np.log(a_.min() / a_) + np.log(t.min() / t)
    val = np.exp(logs / (3 * len(traces)))
    return [(int(n), float(v)) for n, v in zip(slots, val)]
