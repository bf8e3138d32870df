"""The sorted Kendall path's barrier plan against a host model of its LDS
accesses (no GPU).

The sort kernel runs 512 threads (8 wavefronts) per snapshot and skips the
workgroup barrier between two steps when neither touches an LDS entry that
another wavefront touches; a wavefront's own accesses stay ordered by its
in-order issue and a wavefront fence.  Between two workgroup barriers the
wavefronts may be at any of the steps in between, so within each such
segment no entry one wavefront writes may be read or written by another.
This test rebuilds every step's per-wavefront read and write sets from the
kernel's index maps and checks that rule for every padded size, with the
barrier plan the library itself reports (unison_debug_kendall_barrier)."""
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_09643_amd", "libunison.so")

BLOCK, WAVE, PER_T = 512, 64, 8       # threads, wavefront width, entries per thread
SIZES = (256, 512, 1024, 2048, 4096)


def mp_pad(i):
    return i + i // 8


def bitonic_steps(P):
    """(('bitonic', k, j), accesses) per pass; accesses[w] = (reads, writes) of
    wavefront w as sets of (buffer, entry): kx are the 32-bit x keys, A the
    y keys."""
    steps = []
    k = 2
    while k <= P:
        j = k // 2
        while j >= 1:
            acc = [(set(), set()) for _ in range(BLOCK // WAVE)]
            for t in range(BLOCK):
                r, wr = acc[t // WAVE]
                for q in range(PER_T // 2):
                    tt = t + q * BLOCK
                    if tt >= P // 2:
                        continue
                    i = ((tt & ~(j - 1)) << 1) | (tt & (j - 1))
                    for e in (i, i + j):
                        for buf in ("kx", "A"):
                            r.add((buf, e))
                            wr.add((buf, e))
            steps.append((("bitonic", k, j), acc))
            j //= 2
        k *= 2
    return steps


def merge_steps(P):
    """(('merge', w), accesses) per merge level.  Level L reads buffer A when L
    is even (B when odd) and writes the other.  Levels of runs below 8 place
    entry p = t + 512 e by a binary search in the other run; from 8 on, thread
    t merges outputs [8t, 8t + 8), reading anywhere in its pair of runs (in
    the padded layout after the first such level) and storing padded."""
    steps = []
    w, lvl = 1, 0
    while w < P:
        src, dst = ("A", "B") if lvl % 2 == 0 else ("B", "A")
        acc = [(set(), set()) for _ in range(BLOCK // WAVE)]
        for t in range(BLOCK):
            r, wr = acc[t // WAVE]
            if w < 8:
                for e in range(PER_T):
                    p = t + e * BLOCK
                    if p >= P:
                        continue
                    b0 = p & ~(2 * w - 1)
                    for q in range(b0, b0 + 2 * w):     # own entry and the other run
                        r.add((src, q))
                        wr.add((dst, q))                # lands inside the pair of runs
            else:
                o0 = t * PER_T
                if o0 >= P:
                    continue
                b0 = o0 & ~(2 * w - 1)
                pad = (lambda i: mp_pad(i)) if w > 8 else (lambda i: i)
                for q in range(b0, b0 + 2 * w):
                    r.add((src, pad(q)))
                for e in range(PER_T):
                    wr.add((dst, mp_pad(o0 + e)))
        steps.append((("merge", w), acc))
        w *= 2
        lvl += 1
    return steps


def races(steps, barrier_after):
    """Cross-wavefront conflicts inside the segments between workgroup
    barriers: (segment start, wave a, wave b, example entry)."""
    found = []
    seg = []
    for idx, (name, acc) in enumerate(steps):
        seg.append(acc)
        if barrier_after[idx] or idx == len(steps) - 1:
            n = len(seg[0])
            R = [set().union(*(s[w][0] for s in seg)) for w in range(n)]
            W = [set().union(*(s[w][1] for s in seg)) for w in range(n)]
            for a in range(n):
                for b in range(n):
                    if a != b:
                        hit = W[a] & (R[b] | W[b])
                        if hit:
                            found.append((idx, a, b, min(hit)))
            seg = []
    return found


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libunison.so not built; run __graft_entry__.build()")
    from paper_2609_09643_amd import unison
    return unison.lib()


def plan(lib, P, steps):
    out = []
    for name, _ in steps:
        if name[0] == "bitonic":
            b = lib.unison_debug_kendall_barrier(P, 0, name[1], name[2])
        else:
            b = lib.unison_debug_kendall_barrier(P, 1, name[1], 0)
        assert b in (0, 1), (P, name, b)
        out.append(b == 1)
    return out


@pytest.mark.parametrize("P", SIZES)
def test_bitonic_passes_share_no_entry_across_wavefronts_between_barriers(lib, P):
    steps = bitonic_steps(P)
    bar = plan(lib, P, steps)
    assert bar[-1], "the last pass is followed by the run-start scan"
    assert not races(steps, bar)
    assert not all(bar), "the plan should skip some barriers"


@pytest.mark.parametrize("P", SIZES)
def test_merge_levels_share_no_entry_across_wavefronts_between_barriers(lib, P):
    steps = merge_steps(P)
    bar = plan(lib, P, steps)
    assert bar[-1], "the last level is followed by the scan of the sorted y"
    assert not races(steps, bar), races(steps, bar)[:3]


def test_model_flags_a_barrier_taken_out():
    """The model is not vacuous: dropping the barrier after the first merge-
    path level (w = 8) of a 4,096-entry snapshot, where the next level's
    padded stores reach the entries the neighbouring wavefront reads at w = 8,
    is reported, and so is a plan without any workgroup barrier."""
    steps = merge_steps(4096)
    bar = [True] * len(steps)
    assert not races(steps, bar)
    names = [s[0] for s in steps]
    i8 = names.index(("merge", 8))
    bar[i8] = False
    found = races(steps, bar)
    assert found and all(f[0] == i8 + 1 for f in found)
    assert races(bitonic_steps(1024), [False] * len(bitonic_steps(1024)))


def test_invalid_steps_are_refused(lib):
    from paper_2609_09643_amd.unison import E_INVALID
    assert lib.unison_debug_kendall_barrier(100, 1, 8, 0) == E_INVALID      # not a power of two
    assert lib.unison_debug_kendall_barrier(8192, 1, 8, 0) == E_INVALID     # above 4,096
    assert lib.unison_debug_kendall_barrier(1024, 1, 3, 0) == E_INVALID
    assert lib.unison_debug_kendall_barrier(1024, 0, 8, 8) == E_INVALID     # stride >= stage
    assert lib.unison_debug_kendall_barrier(1024, 2, 1, 1) == E_INVALID
