"""Hand-built traces for tests (input construction only, no policy arithmetic)."""
import numpy as np

from paper_2609_09643_amd.synth import (KIND_ARRIVE, KIND_DONE, KIND_GAP_START, U64_MAX,
                                         Trace, default_params)


def trace_from_events(events, n_sessions, kvb=1, tools=None):
    """events: list of (t_ns, sid, kind, turn, length) in trace order.  The
    next_ns column of each GAP_START is filled from the session's next
    ARRIVE.  tools: optional tool class per event (read at gap onsets)."""
    ev = list(events)
    n = len(ev)
    t = np.array([e[0] for e in ev], dtype=np.uint64)
    sid = np.array([e[1] for e in ev], dtype=np.uint32)
    kind = np.array([e[2] for e in ev], dtype=np.uint32)
    turn = np.array([e[3] for e in ev], dtype=np.uint32)
    length = np.array([e[4] if e[2] == KIND_ARRIVE else 0 for e in ev], dtype=np.uint32)
    nxt = np.full(n, U64_MAX, dtype=np.uint64)
    for i in range(n):
        if kind[i] == KIND_GAP_START:
            for j in range(i + 1, n):
                if sid[j] == sid[i] and kind[j] == KIND_ARRIVE:
                    nxt[i] = t[j]
                    break
    turns = np.zeros(n_sessions, dtype=np.uint32)
    for i in range(n):
        if kind[i] == KIND_ARRIVE and sid[i] < n_sessions:
            turns[sid[i]] = max(turns[sid[i]], turn[i] + 1)
    kv = np.full(n_sessions, kvb, dtype=np.uint32) if np.isscalar(kvb) else np.asarray(kvb, np.uint32)
    tool = None if tools is None else np.asarray(tools, dtype=np.uint32)
    return Trace(t, sid, (kind << 24) | turn, length, nxt, kv, turns, tool)


def trace_from_requests(reqs, n_sessions, length=1, kvb=1, dt=10):
    """A request string: request i of session s is an ARRIVE at dt*i + dt and
    its end (GAP_START, or DONE on the session's last request) one ns later,
    so exactly one session is being served at any time."""
    last = {}
    for i, s in enumerate(reqs):
        last[s] = i
    turn = {}
    events = []
    for i, s in enumerate(reqs):
        k = turn.get(s, 0)
        turn[s] = k + 1
        ln = length(s, k) if callable(length) else length
        t0 = dt * (i + 1)
        events.append((t0, s, KIND_ARRIVE, k, ln))
        events.append((t0 + 1, s, KIND_DONE if last[s] == i else KIND_GAP_START, k, 0))
    return trace_from_events(events, n_sessions, kvb)


def single_tier_params(policy, slots, tide=0):
    """One HBM tier of unbounded bytes and `slots` session slots; no SRAM."""
    p = default_params(1)
    p["policy"] = policy
    p["tide"] = tide
    p["cap_sram_B"] = 0
    p["cap_hbm_B"] = 1 << 40
    p["n_slots"] = slots
    p["ttl_ns"] = 1 << 62
    return p
