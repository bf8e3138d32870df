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
barrier plan the library itself reports (unison_debug_kendall_barrier).

The bitonic passes run in groups of up to three in registers: a group loads
its entries before its first pass and stores them after its last.  The sort
keys are 8-byte entries of the first buffer (A), at padded positions.  In the
narrow form (4-byte y values) the merge sort then runs in A, its two buffers
of P padded values 16 words apart; in the wide form the 4-byte tie-breakers
live in a second buffer (B), where the merge sort of the 8-byte y values
starts.  Every merge buffer is padded.  Accesses are modelled as the 4-byte
words they touch, so the aliasing between those uses is exact.  A merge
step also reads one entry past a run whose entries are all taken, a value it
never uses; that read lands in a gap after a buffer, never on a buffer being
written (test_kendall_merge_model.py replays the step), and is not modelled."""
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_09643_amd", "libunison.so")

BLOCK, WAVE, PER_T = 512, 64, 8       # threads, wavefront width, entries per thread
SIZES = (256, 512, 1024, 2048, 4096)


def mp_pad(i):
    return i + i // 8


def group_top(L, s):
    return L - 1 - 3 * ((L - 1 - s) // 3)


def group_low(top):
    return top - 2 if top >= 2 else 0


def words(buf, i, size):
    """The 4-byte words of entry i (padded) of a buffer of size-byte entries."""
    w = size // 4
    return [(buf, mp_pad(i) * w + k) for k in range(w)]


def sort_words(i, ysize):
    """An entry's sort key (A, 8 B) and the wide form's tie-breaker (B, 4 B)."""
    return words("A", i, 8) + (words("B", i, 4) if ysize == 8 else [])


MERGE_GAP = 16


def merge_buffers(P, ysize):
    """(first source, first destination) of the merge levels, each as (LDS
    buffer, first entry): entry q of buffer b lies at merge_words(b, q, ysize)."""
    if ysize == 4:   # both in A, a gap between them
        return ("A", 0), ("A", P + P // 8 + MERGE_GAP)
    return ("B", 0), ("A", 0)


def merge_words(buf, q, ysize):
    name, shift = buf
    w = ysize // 4
    return [(name, (shift + mp_pad(q)) * w + k) for k in range(w)]


def bitonic_steps(P, ysize=8):
    """(('bitonic', k, j), accesses) per pass, then ('final',): accesses[w] =
    (reads, writes) of wavefront w as sets of (buffer, word).  Stages 2, 4 and
    8 run on each thread's 8 consecutive entries from the gather and store
    them at the end; from stage 16 on, a group with low bit b holds the
    entries that differ from the thread's base only in bits b..b+2.  The last
    group keeps its entries; after its barrier they are stored, sorted by y
    within each thread, as the merge input in B."""
    steps = []
    n_w = BLOCK // WAVE

    def empty():
        return [(set(), set()) for _ in range(n_w)]

    for k in (2, 4, 8):
        j = k // 2
        while j >= 1:
            acc = empty()
            if k == 8 and j == 1:
                for t in range(BLOCK):
                    if t * PER_T >= P:
                        continue
                    for c in range(PER_T):
                        for e in sort_words(t * PER_T + c, ysize):
                            acc[t // WAVE][1].add(e)
            steps.append((("bitonic", k, j), acc))
            j //= 2
    k, L = 16, 4
    while k <= P:
        for s in range(L - 1, -1, -1):
            top = group_top(L, s)
            lo = group_low(top)
            acc = empty()
            first, last = s == top, s == lo
            for t in range(BLOCK):
                base = ((t >> lo) << (lo + 3)) | (t & ((1 << lo) - 1))
                if base >= P:
                    continue
                r, wr = acc[t // WAVE]
                for c in range(PER_T):
                    for e in sort_words(base | (c << lo), ysize):
                        if first:
                            r.add(e)
                        if last and not (k == P and s == 0):
                            wr.add(e)
            steps.append((("bitonic", k, 1 << s), acc))
        k *= 2
        L += 1
    acc = empty()
    for t in range(BLOCK):
        for c in range(PER_T):
            i = t * PER_T + c
            if i < P:
                acc[t // WAVE][1].update(merge_words(merge_buffers(P, ysize)[0], i, ysize))
    steps.append((("final",), acc))
    return steps


def merge_steps(P, ysize=8):
    """(('merge', w), accesses) per merge level from runs of 8 (y values of
    ysize bytes).  The first level reads the per-thread sorted groups, and the
    levels alternate; thread t merges outputs [8t, 8t + 8), reading anywhere
    in its pair of runs."""
    steps = []
    w, lvl = 8, 0
    first, second = merge_buffers(P, ysize)
    while w < P:
        src, dst = (first, second) if lvl % 2 == 0 else (second, first)
        acc = [(set(), set()) for _ in range(BLOCK // WAVE)]
        for t in range(BLOCK):
            r, wr = acc[t // WAVE]
            o0 = t * PER_T
            if o0 >= P:
                continue
            b0 = o0 & ~(2 * w - 1)
            for q in range(b0, b0 + 2 * w):
                r.update(merge_words(src, q, ysize))
            for e in range(PER_T):
                wr.update(merge_words(dst, o0 + e, ysize))
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
        if name[0] == "final":
            b = 1          # the scans of the sorted runs start with workgroup barriers
        elif name[0] == "bitonic":
            b = lib.unison_debug_kendall_barrier(P, 0, name[1], name[2])
        else:
            b = lib.unison_debug_kendall_barrier(P, 1, name[1], 0)
        assert b in (0, 1), (P, name, b)
        out.append(b == 1)
    return out


@pytest.mark.parametrize("P", SIZES)
@pytest.mark.parametrize("ysize", [4, 8])
def test_bitonic_groups_share_no_entry_across_wavefronts_between_barriers(lib, P, ysize):
    steps = bitonic_steps(P, ysize)
    bar = plan(lib, P, steps)
    names = [s[0] for s in steps]
    assert bar[names.index(("bitonic", P, 1))], "the last group is read before the merge input is stored"
    assert not races(steps, bar), races(steps, bar)[:3]
    assert not all(bar), "the plan should skip some barriers"


@pytest.mark.parametrize("P", SIZES)
@pytest.mark.parametrize("ysize", [4, 8])
def test_merge_levels_share_no_entry_across_wavefronts_between_barriers(lib, P, ysize):
    steps = merge_steps(P, ysize)
    bar = plan(lib, P, steps)
    assert bar[-1], "the last level is followed by the scan of the sorted y"
    assert not races(steps, bar), races(steps, bar)[:3]


@pytest.mark.parametrize("ysize", [4, 8])
def test_whole_plan_shares_no_entry_across_wavefronts_between_barriers(lib, ysize):
    """Sort and merge as one sequence at 4,096 entries: the tie-breakers share
    B with the merge input and the later levels, the keys share A with them."""
    steps = bitonic_steps(4096, ysize) + merge_steps(4096, ysize)
    assert not races(steps, plan(lib, 4096, steps))


def test_model_flags_a_barrier_taken_out(lib):
    """The model is not vacuous: dropping any one workgroup barrier the
    library places between groups of cross-wavefront passes, or between merge
    levels, is reported, and so is a plan without any workgroup barrier."""
    for steps in (bitonic_steps(4096), merge_steps(4096)):
        bar = plan(lib, 4096, steps)
        assert not races(steps, bar)
        flagged = 0
        for i in range(len(steps) - 1):
            if bar[i]:
                cut = list(bar)
                cut[i] = False
                flagged += bool(races(steps, cut))
        assert flagged >= 3
    assert races(bitonic_steps(1024), [False] * len(bitonic_steps(1024)))
    # before the merge input is stored, every wavefront must have read its last group
    steps = bitonic_steps(4096)
    bar = plan(lib, 4096, steps)
    names = [s[0] for s in steps]
    bar[names.index(("bitonic", 4096, 1))] = False
    assert races(steps, bar)


def test_invalid_steps_are_refused(lib):
    from paper_2609_09643_amd.unison import E_INVALID
    assert lib.unison_debug_kendall_barrier(100, 1, 8, 0) == E_INVALID      # not a power of two
    assert lib.unison_debug_kendall_barrier(8192, 1, 8, 0) == E_INVALID     # above 4,096
    assert lib.unison_debug_kendall_barrier(1024, 1, 3, 0) == E_INVALID
    assert lib.unison_debug_kendall_barrier(1024, 1, 4, 0) == E_INVALID     # merged in registers
    assert lib.unison_debug_kendall_barrier(1024, 0, 8, 8) == E_INVALID     # stride >= stage
    assert lib.unison_debug_kendall_barrier(1024, 2, 1, 1) == E_INVALID
