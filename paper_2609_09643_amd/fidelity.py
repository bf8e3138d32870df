"""The fixed-point format sweep (Sec. IV-C) with its two hard gates, and the
online convergence of the hazard table (eq. (attainment)).

For every (b_h, b_g, tau) point of the pre-registered grid (exact divider,
b_s = 64, P_Z = P / tau) this measures, on the GPU:

* end-to-end drift: SPEAR+TIDE replayed over whole traces once with the fp32
  score (eq. (esp)) and once with score_q (eq. (scoreq)); per (trace,
  capacity envelope) cell the hit-rate difference in percentage points and
  the relative AMAT difference (eq. (hr-amat)).  Gate: the worst cell stays
  within 0.20 pp.
* ranking fidelity on register-file snapshots: both EMAs replayed over each
  session's gap history, both scores, Kendall tau-b and top-1 victim
  agreement per snapshot (Sec. VI-F).  Gate: top-1 agreement >= 0.99.

Every step runs in libunison's kernels; this module only marshals the
workloads and turns counter arrays into rates.
"""
from __future__ import annotations

import numpy as np

from . import synth
from . import unison as U

HR_GATE_PP = 0.20
TOP1_GATE = 0.99


def hit_rate(c):
    """Hits over requests per simulation (eq. (hr-amat))."""
    req = c["requests"].astype(np.float64)
    return (c["hit_sram"].astype(np.float64) + c["hit_hbm"].astype(np.float64)) / np.maximum(req, 1)


def mean_amat(c):
    """AMAT per request in ns (eq. (hr-amat))."""
    return c["amat_sum_ns"] / np.maximum(c["requests"].astype(np.float64), 1)


def trajectory_drift(counters, meta, n_formats):
    """Per format and cell: (hit-rate drift in pp, AMAT drift in %) of
    score_q against the fp32 run of the same cell.  Arrays [n_formats,
    n_cells], cells ordered (trace, envelope)."""
    hr = hit_rate(counters)
    am = mean_amat(counters)
    cells = sorted({(int(m["trace"]), int(m["envelope"])) for m in meta})
    col = {cell: k for k, cell in enumerate(cells)}
    ref_hr = np.full(len(cells), np.nan)
    ref_am = np.full(len(cells), np.nan)
    d_hr = np.full((n_formats, len(cells)), np.nan)
    d_am = np.full((n_formats, len(cells)), np.nan)
    for i, m in enumerate(meta):
        if int(m["fmt"]) < 0:
            k = col[(int(m["trace"]), int(m["envelope"]))]
            ref_hr[k], ref_am[k] = hr[i], am[i]
    for i, m in enumerate(meta):
        f = int(m["fmt"])
        if f >= 0:
            k = col[(int(m["trace"]), int(m["envelope"]))]
            d_hr[f, k] = 100.0 * (hr[i] - ref_hr[k])
            d_am[f, k] = 100.0 * (am[i] - ref_am[k]) / ref_am[k] if ref_am[k] else 0.0
    return d_hr, d_am, cells


def run_trajectories(workload, meta, formats):
    """Runs the whole sweep batch on the GPU; returns counters and drifts."""
    sim = U.Simulator(workload)
    sim.run()
    c = sim.counters()
    d_hr, d_am, cells = trajectory_drift(c, meta, len(formats))
    return c, d_hr, d_am, cells


def tau_b(counts):
    """Kendall tau-b per snapshot from the pair counts {C, D, tie x, tie y,
    tie both}."""
    c = counts.astype(np.float64)
    cc, dd, tx, ty = c[:, 0], c[:, 1], c[:, 2], c[:, 3]
    den = np.sqrt((cc + dd + tx) * (cc + dd + ty))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(den > 0, (cc - dd) / den, np.nan)


def ranking_fidelity(rs, formats, penalty_us=5e8):
    """Per format: (mean tau-b, pooled tau-b, top-1 agreement) over the
    snapshots of RankingSet rs."""
    dev = U._dev
    gaps, nh = dev(rs.gaps_ns, np.uint64), dev(rs.n_hist)
    turn, done = dev(rs.turn), dev(rs.done)
    idx = dev(rs.idx, np.uint32)
    d, n = U.hazard_counts(dev(rs.lut_pop, np.uint32))
    g, _ = U.ema_replay(gaps, nh)
    x = U.score_fp32(turn, g, done, d, n, penalty_us)
    out = []
    for fmt in formats:
        bh, bg, tau = fmt[:3]
        w = fmt[3] if len(fmt) > 3 else 0
        _, gq = U.ema_replay(gaps, nh, bg, tau)
        y = U.score_fixed(turn, gq, done, d, n, bh, int(round(penalty_us * 1000 / tau)), w)
        counts, top1 = U.kendall(x, y, idx)
        cnt = U._host(counts, np.uint64)
        t1 = top1.cpu().numpy()
        tb = tau_b(cnt)
        pooled = tau_b(cnt.sum(axis=0, keepdims=True))[0]
        out.append((float(np.nanmean(tb)), float(pooled), float((t1 == 1).mean())))
    return out


def sweep(traces=None, rs=None, formats=None, penalty_us=5e8):
    """The full sweep.  One dict per format: its point, worst-cell and mean
    |hit-rate drift| (pp), mean AMAT drift (%), ranking statistics and the
    two gates."""
    formats = synth.format_grid() if formats is None else list(formats)
    w, meta = synth.format_sweep(traces=traces, formats=formats, penalty_us=penalty_us)
    _, d_hr, d_am, cells = run_trajectories(w, meta, formats)
    rank = ranking_fidelity(synth.fidelity_snapshots() if rs is None else rs, formats, penalty_us)
    rows = []
    for f, fmt in enumerate(formats):
        bh, bg, tau = fmt[:3]
        worst = float(np.nanmax(np.abs(d_hr[f])))
        mtau, ptau, top1 = rank[f]
        rows.append({"b_h": bh, "b_g": bg, "tau_ns": tau,
                     "divider": "exact" if len(fmt) < 4 or fmt[3] == 0 else "recip%d" % fmt[3],
                     "worst_hr_drift_pp": worst, "mean_hr_drift_pp": float(np.nanmean(np.abs(d_hr[f]))),
                     "mean_amat_drift_pct": float(np.nanmean(d_am[f])),
                     "mean_tau_b": mtau, "pooled_tau_b": ptau, "top1": top1,
                     "passes": bool(worst <= HR_GATE_PP and top1 >= TOP1_GATE)})
    return rows, len(cells)


def attainment(counters, meta):
    """eq. (attainment) per trace: A(n) = (H_on(n) - H_LRU) / (H_off - H_LRU),
    the share of the offline table's hit-rate surplus over LRU realised after
    n observed sessions, for a table rebuilt online from the first n
    completions ("online") and for a fixed table fitted on them ("prefix").
    Returns {trace: {"online" | "prefix": [(n, A(n), H(n))]}} and {trace:
    (H_LRU, H_off)}."""
    hr = hit_rate(counters)
    ref, curves = {}, {}
    for i, m in enumerate(meta):
        t = int(m["trace"])
        lru, off = ref.get(t, (None, None))
        if int(m["kind"]) == synth.ATTAIN_LRU:
            lru = hr[i]
        elif int(m["kind"]) == synth.ATTAIN_OFFLINE:
            off = hr[i]
        ref[t] = (lru, off)
    names = {synth.ATTAIN_ONLINE: "online", synth.ATTAIN_PREFIX: "prefix"}
    for i, m in enumerate(meta):
        kind = int(m["kind"])
        if kind not in names:
            continue
        t = int(m["trace"])
        lru, off = ref[t]
        a = (hr[i] - lru) / (off - lru) if off != lru else float("nan")
        curves.setdefault(t, {}).setdefault(names[kind], []).append((int(m["n"]), float(a), float(hr[i])))
    for t in curves:
        for k in curves[t]:
            curves[t][k].sort()
    return curves, ref


def run_attainment(traces=None, envelope=synth.FIDELITY_ENVELOPES[0], points=None):
    """Runs the attainment batch on the GPU (one launch)."""
    w, meta = synth.attainment_workload(traces, envelope, points)
    sim = U.Simulator(w)
    sim.run()
    c = sim.counters()
    return attainment(c, meta) + (c, w)
