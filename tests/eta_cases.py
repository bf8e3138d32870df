"""Hand-worked traces of the tool-type arrival-table baseline (ETA): input
construction and expected values only, shared by the oracle pins and the GPU
parity test.  Single tier (no SRAM), two session slots, h = 0."""
from paper_2609_09643_amd.synth import KIND_ARRIVE as A, KIND_DONE as D, KIND_GAP_START as G
from tracekit import single_tier_params, trace_from_events

H, NONE = 2, 0xFFFFFFFF
OP_EVICT, OP_PLACE = 1, 7
ETA_TABLE = [10_000, 50_000] + [0] * 14     # class 0 expected 10 us, class 1 expected 50 us


def predicted_and_true_returns_disagree():
    """A (sid 0) opens a class-0 gap at 2,000 ns and returns at 102,000; B
    (sid 1) opens a class-1 gap at 4,000 and returns at 24,000.  C (sid 2)
    arrives at 5,000 with both slots taken by A and B.
      Belady evicts A (next arrival 102,000 > 24,000).  ETA predicts A at
      2,000 + 10,000 = 12,000 and B at 4,000 + 50,000 = 54,000: it evicts B.
      B returns at 24,000: a Belady hit; under ETA a miss, and the slots hold
      A (predicted 12,000) and the completed C (never returns): C goes.
      A returns at 102,000: under ETA an HBM hit; under Belady a miss, whose
      placement evicts one of the two completed sessions B and C, the
      smaller id B.
    Returns the trace, the row builder and, per policy, the decision list and
    (requests, misses, HBM hits)."""
    ev = [(1000, 0, A, 0, 1), (2000, 0, G, 0, 0), (3000, 1, A, 0, 1), (4000, 1, G, 0, 0),
          (5000, 2, A, 0, 1), (6000, 2, D, 0, 0), (24000, 1, A, 1, 1), (25000, 1, D, 1, 0),
          (102000, 0, A, 1, 1), (103000, 0, D, 1, 0)]
    tools = [0, 0, 0, 1, 0, 0, 0, 0, 0, 0]
    tr = trace_from_events(ev, 3, tools=tools)
    want = {
        "eta": ([(0, OP_PLACE, 0, H), (2, OP_PLACE, 1, H), (4, OP_EVICT, 1, NONE),
                 (4, OP_PLACE, 2, H), (6, OP_EVICT, 2, NONE), (6, OP_PLACE, 1, H),
                 (8, OP_PLACE, 0, H)], (5, 4, 1)),
        "belady": ([(0, OP_PLACE, 0, H), (2, OP_PLACE, 1, H), (4, OP_EVICT, 0, NONE),
                    (4, OP_PLACE, 2, H), (6, OP_PLACE, 1, H), (8, OP_EVICT, 1, NONE),
                    (8, OP_PLACE, 0, H)], (5, 4, 1)),
    }
    return tr, lambda policy: single_tier_params(policy, 2), want
