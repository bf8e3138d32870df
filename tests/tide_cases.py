"""Hand-worked traces of the TIDE pass (eq. (budget), eq. (promote),
eq. (demote), Algorithm 1's tiering branch) with their decision lists,
worked out by hand in each docstring.  Input construction and expected
values only; shared by the oracle pins and the GPU parity test.

Common setting: Belady keys (the time of the session's next ARRIVE, larger =
evict / demote first), 1 byte per token, DMA bandwidth B = 1 byte per us, so
a gap onset's budget is its session's gap EMA in whole microseconds (the EMA
of eq. (ema) over gaps in us: 3/10 of the first gap).  The session that
opens the pass is bypassed at every arrival (its prefix exceeds both tiers),
so it holds no tier and is never a candidate itself."""
from paper_2609_09643_amd import synth
from paper_2609_09643_amd.synth import KIND_ARRIVE as A, KIND_DONE as D, KIND_GAP_START as G
from tracekit import trace_from_events

S, H, NONE = 1, 2, 0xFFFFFFFF
OP_EVICT, OP_BYPASS, OP_PROMOTE, OP_SWAP, OP_PLACE = 1, 3, 4, 5, 7


def params(cap_sram):
    p = synth.default_params(1)
    p["policy"], p["tide"] = synth.POLICY_BELADY, 1
    p["cap_sram_B"], p["cap_hbm_B"], p["n_slots"], p["dma_B_per_us"] = cap_sram, 100, 10, 1
    p["t_s_ns_per_B"], p["t_h_ns_per_B"], p["t_p_ns_per_tok"] = 1.0, 10.0, 100.0
    return p


def swap_frees_sram_and_a_demoted_session_returns():
    """SRAM 10 B.  d1 (sid 0, 4 B) and d2 (sid 1, 6 B) fill SRAM; p1 (sid 2,
    2 B) and p2 (sid 3, 3 B) land in HBM.  d1 and d2 next return at the same
    time (key 400,000), p1 at 200,000 and p2 at 300,000.  T (sid 4) arrives
    again after a 100 us gap: EMA 30 us, budget 30 B at its gap onset (e11).
    Earlier gap onsets have budget 0: their passes start and move nothing.
      it 1: p = p1 (min in HBM).  2 + 10 > 10: no promotion.  d = argmax in
            SRAM: d1 and d2 tie, the smaller id d1.  key 200,000 < 400,000,
            2 + 4 <= 30, SRAM 10 - 4 + 2 <= 10: swap (p1, d1); left 24.
      it 2: p = p2 (300,000 < d1's 400,000).  8 + 3 > 10: no promotion.
            d = d2; 300,000 < 400,000, 3 + 6 <= 24, SRAM 8 - 6 + 3 <= 10:
            swap (p2, d2); left 15, SRAM 5.
      it 3: p = d1 (d1 and d2 tie in HBM, the smaller id): 5 + 4 <= 10 and
            4 <= 15: promote d1 alone -- the session demoted at it 1 returns
            through the promote-only move into the SRAM the swaps freed.
      it 4: p = d2: 9 + 6 > 10; d = d1 (400,000); 400,000 < 400,000 fails:
            the pass ends.  Moved 6 + 9 + 4 = 19 B, DMA busy 19 us.
    p1, p2 and d1 are then SRAM hits on sessions TIDE moved there since
    their last request (three prefetch hits); d2 is an HBM hit."""
    ev = [(1000, 0, A, 0, 4), (2000, 0, G, 0, 0), (3000, 1, A, 0, 6), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 2), (6000, 2, G, 0, 0), (7000, 3, A, 0, 3), (8000, 3, G, 0, 0),
          (9000, 4, A, 0, 1000), (10000, 4, G, 0, 0), (110000, 4, A, 1, 1000),
          (111000, 4, G, 1, 0),
          (200000, 2, A, 1, 2), (201000, 2, D, 1, 0), (300000, 3, A, 1, 3), (301000, 3, D, 1, 0),
          (400000, 0, A, 1, 4), (400000, 1, A, 1, 6), (401000, 0, D, 1, 0), (401000, 1, D, 1, 0),
          (500000, 4, A, 2, 1000), (501000, 4, D, 2, 0)]
    want_log = [(0, OP_PLACE, 0, S), (2, OP_PLACE, 1, S), (4, OP_PLACE, 2, H), (6, OP_PLACE, 3, H),
                (8, OP_BYPASS, 4, NONE), (10, OP_BYPASS, 4, NONE),
                (11, OP_SWAP, 2, 0), (11, OP_SWAP, 3, 1), (11, OP_PROMOTE, 0, NONE),
                (12, OP_PLACE, 2, S), (14, OP_PLACE, 3, S), (16, OP_PLACE, 0, S),
                (17, OP_PLACE, 1, H), (20, OP_BYPASS, 4, NONE)]
    want = {"requests": 11, "miss": 7, "hit_sram": 3, "hit_hbm": 1, "bypass": 3, "evict": 0,
            "swap": 2, "promote": 1, "dma_bytes": 19, "tide_passes": 6, "prefetch_hits": 3}
    budgets = {11: (30, 19), 1: (0, 0), 5: (0, 0), 9: (0, 0)}
    return trace_from_events(ev, 5), params(10), want_log, want, budgets


def budget_runs_out_mid_pass():
    """SRAM 12 B.  X (sid 0, 10 B) and Y (sid 1, 2 B, key 800,000) fill SRAM;
    p1 (sid 2, 3 B, key 200,000) and p2 (sid 3, 4 B, key 300,000) land in
    HBM.  X returns at 20,000 ns with 11 tokens: 2 + 11 > 12, so it moves to
    HBM and frees 10 B of SRAM.  Its gap was 18 us: EMA 5.4 us, budget 5 B at
    its gap onset (e9), when X's key is its next arrival, 900,000.
      it 1: p = p1: 2 + 3 <= 12 and 3 <= 5: promote; left 2.
      it 2: p = p2: 5 + 4 <= 12 fits SRAM, but 4 > 2: no promotion.  d = Y
            (800,000 > p1's 200,000); 300,000 < 800,000 and the capacities
            after the swap hold, but 4 + 2 > 2: the budget is spent and the
            pass ends.  Moved 3 B.
    X's return at 20,000 ns is an SRAM hit; p1 returns to SRAM (one prefetch
    hit); p2 and X's last return are HBM hits; Y an SRAM hit that TIDE did not
    bring."""
    ev = [(1000, 0, A, 0, 10), (2000, 0, G, 0, 0), (3000, 1, A, 0, 2), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 3), (6000, 2, G, 0, 0), (7000, 3, A, 0, 4), (8000, 3, G, 0, 0),
          (20000, 0, A, 1, 11), (21000, 0, G, 1, 0),
          (200000, 2, A, 1, 3), (201000, 2, D, 1, 0), (300000, 3, A, 1, 4), (301000, 3, D, 1, 0),
          (800000, 1, A, 1, 2), (801000, 1, D, 1, 0), (900000, 0, A, 2, 11), (901000, 0, D, 2, 0)]
    want_log = [(0, OP_PLACE, 0, S), (2, OP_PLACE, 1, S), (4, OP_PLACE, 2, H), (6, OP_PLACE, 3, H),
                (8, OP_PLACE, 0, H), (9, OP_PROMOTE, 2, NONE),
                (10, OP_PLACE, 2, S), (12, OP_PLACE, 3, H), (14, OP_PLACE, 1, S),
                (16, OP_PLACE, 0, H)]
    want = {"requests": 9, "miss": 4, "hit_sram": 3, "hit_hbm": 2, "bypass": 0, "evict": 0,
            "swap": 0, "promote": 1, "dma_bytes": 3, "tide_passes": 5, "prefetch_hits": 1}
    budgets = {9: (5, 3), 5: (0, 0)}
    return trace_from_events(ev, 4), params(12), want_log, want, budgets


def first_illegal_move_ends_the_pass():
    """SRAM 12 B, as in the budget case, but p (sid 2) holds 13 B and q (sid
    3) 3 B, and X's gap is 70 us: EMA 21 us, budget 21 B at e9.
      it 1: p = p (key 200,000, the HBM minimum): 2 + 13 > 12, no promotion;
            d = Y: 200,000 < 800,000 and 13 + 2 <= 21, but SRAM after the
            swap would hold 2 - 2 + 13 > 12: not a legal pair, and the pass
            ends there.
    q (key 300,000) would fit free SRAM and the budget on its own, but the
    loop stops at its first illegal move and never looks past p: nothing
    moves, and q is an HBM hit on its return (X's first return and Y's are
    SRAM hits, p's and X's last return HBM hits)."""
    ev = [(1000, 0, A, 0, 10), (2000, 0, G, 0, 0), (3000, 1, A, 0, 2), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 13), (6000, 2, G, 0, 0), (7000, 3, A, 0, 3), (8000, 3, G, 0, 0),
          (72000, 0, A, 1, 11), (73000, 0, G, 1, 0),
          (200000, 2, A, 1, 13), (201000, 2, D, 1, 0), (300000, 3, A, 1, 3), (301000, 3, D, 1, 0),
          (800000, 1, A, 1, 2), (801000, 1, D, 1, 0), (900000, 0, A, 2, 11), (901000, 0, D, 2, 0)]
    want_log = [(0, OP_PLACE, 0, S), (2, OP_PLACE, 1, S), (4, OP_PLACE, 2, H), (6, OP_PLACE, 3, H),
                (8, OP_PLACE, 0, H), (10, OP_PLACE, 2, H), (12, OP_PLACE, 3, H),
                (14, OP_PLACE, 1, S), (16, OP_PLACE, 0, H)]
    want = {"requests": 9, "miss": 4, "hit_sram": 2, "hit_hbm": 3, "bypass": 0, "evict": 0,
            "swap": 0, "promote": 0, "dma_bytes": 0, "tide_passes": 5, "prefetch_hits": 0}
    budgets = {9: (21, 0)}
    return trace_from_events(ev, 4), params(12), want_log, want, budgets


def equal_keys_never_swap():
    """SRAM 10 B.  d (sid 0, 6 B) sits in SRAM and p (sid 1, 6 B) in HBM; both
    next return at 400,000 ns.  T (sid 2) opens a pass with a 30 B budget
    (a 100 us gap) at e7.
      it 1: p = p: 6 + 6 > 10, no promotion; d = d: 400,000 < 400,000 fails
            (the comparison is strict), so the pass ends although the budget
            (12 <= 30) and both capacities would allow the swap.
    Nothing moves; d is an SRAM hit, p an HBM hit."""
    ev = [(1000, 0, A, 0, 6), (2000, 0, G, 0, 0), (3000, 1, A, 0, 6), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 1000), (6000, 2, G, 0, 0), (106000, 2, A, 1, 1000), (107000, 2, G, 1, 0),
          (400000, 0, A, 1, 6), (400000, 1, A, 1, 6), (401000, 0, D, 1, 0), (401000, 1, D, 1, 0),
          (500000, 2, A, 2, 1000), (501000, 2, D, 2, 0)]
    want_log = [(0, OP_PLACE, 0, S), (2, OP_PLACE, 1, H), (4, OP_BYPASS, 2, NONE),
                (6, OP_BYPASS, 2, NONE), (8, OP_PLACE, 0, S), (9, OP_PLACE, 1, H),
                (12, OP_BYPASS, 2, NONE)]
    want = {"requests": 7, "miss": 5, "hit_sram": 1, "hit_hbm": 1, "bypass": 3, "evict": 0,
            "swap": 0, "promote": 0, "dma_bytes": 0, "tide_passes": 4, "prefetch_hits": 0}
    budgets = {7: (30, 0)}
    return trace_from_events(ev, 3), params(10), want_log, want, budgets


CASES = {
    "equal_keys_never_swap": equal_keys_never_swap,
    "swap_then_promote_back": swap_frees_sram_and_a_demoted_session_returns,
    "budget_runs_out": budget_runs_out_mid_pass,
    "first_illegal_stops": first_illegal_move_ends_the_pass,
}
