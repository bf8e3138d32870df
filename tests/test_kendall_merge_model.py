"""Host replay of the Kendall kernel's merge levels (no GPU).

From runs of 8 the kernel merge-sorts y bottom-up by merge path: thread t
owns outputs [8t, 8t + 8) of its pair of runs, binary-searches its diagonal
for how many come from the left run, then merges them, adding the left
entries still waiting whenever it takes a right one.  A run with no entries
left keeps its head one past its end; that value is read but never taken.

This replays each thread's reads and writes in the kernel's own layouts:
every merge buffer holds entry q at q + q // 8; the packed form's two
buffers are 4-byte words, the second 16 words after the first ends, with 16
more after it; the wide form's are 8-byte entries, the tie-breaker buffer
(where the merge starts) 8 entries after the key buffer ends, with 8 more
after it.  It checks that every read lies inside the allocation, that a read
whose value is used lies in the source buffer, that no read past a run lands
on the buffer being written, and that the result is sorted with the
inversions a brute-force count finds."""
import numpy as np
import pytest

PER_T = 8


def mp_pad(q):
    return q + q // 8


def layout(P, form):
    """(first source, first destination, allocation) in the form's units."""
    sb = P + P // 8
    if form == "packed":
        gap = 16
        return 0, sb + gap, 2 * sb + 2 * gap
    gap = 8
    return sb + gap, 0, 2 * sb + 2 * gap


def merge_levels(P, runs8, form):
    """Merge the per-thread sorted groups of 8; returns (inversions, sorted)."""
    sb = P + P // 8
    src, dst, size = layout(P, form)
    mem = np.full(size, -1, dtype=np.int64)
    for q in range(P):
        mem[src + mp_pad(q)] = runs8[q]
    inv = 0
    w = PER_T
    while w < P:
        out = {}
        for t in range(P // PER_T):
            i0 = PER_T * t
            b0 = i0 & ~(2 * w - 1)
            d = i0 - b0

            def rd(q, used):
                a = src + mp_pad(q)
                assert 0 <= a < size, ("read outside the allocation", P, w, t, q)
                if used:
                    assert q < P, ("a used read past the source", P, w, t, q)
                else:
                    assert not dst <= a < dst + sb, ("a past-end read on the destination", P, w, t, q)
                return mem[a]

            lo, hi = (d - w if d > w else 0), (d if d < w else w)
            while lo < hi:
                mid = (lo + hi) >> 1
                if rd(b0 + mid, True) <= rd(b0 + w + d - 1 - mid, True):
                    lo = mid + 1
                else:
                    hi = mid
            xa, xb = b0 + lo, b0 + w + (d - lo)
            na, nb = w - lo, w - (d - lo)
            a, b = rd(xa, na > 0), rd(xb, nb > 0)
            for e in range(PER_T):
                take_a = na != 0 and (nb == 0 or a <= b)
                out[dst + mp_pad(i0) + e] = a if take_a else b
                if not take_a:
                    inv += na
                if take_a:
                    na -= 1
                    xa += 1
                else:
                    nb -= 1
                    xb += 1
                v = rd(xa if take_a else xb, (na > 0) if take_a else (nb > 0))
                if take_a:
                    a = v
                else:
                    b = v
        for k, v in out.items():
            mem[k] = v
        src, dst = dst, src
        w *= 2
    return inv, np.array([mem[src + mp_pad(q)] for q in range(P)])


@pytest.mark.parametrize("form", ["packed", "wide"])
@pytest.mark.parametrize("P", [256, 512, 1024, 2048, 4096])
@pytest.mark.parametrize("spread", [5, 1 << 31])
def test_merge_levels_stay_in_bounds_and_count_the_inversions(form, P, spread):
    rng = np.random.default_rng(P + spread % 97 + (form == "wide"))
    y = rng.integers(0, spread, P)
    groups = y.reshape(-1, PER_T)
    inside = sum(int(np.triu(g[:, None] > g[None, :], 1).sum()) for g in groups)
    inv, merged = merge_levels(P, np.sort(groups, axis=1).ravel(), form)
    assert np.array_equal(merged, np.sort(y))
    brute = sum(int((y[:i] > y[i]).sum()) for i in range(P))
    assert inside + inv == brute


def test_the_model_catches_a_missing_gap():
    """Without the gap after the first buffer, the packed form's first
    level reads past its last run onto the destination."""
    P = 256
    y = np.arange(P)[::-1].copy()
    groups = np.sort(y.reshape(-1, PER_T), axis=1).ravel()
    global layout
    saved = layout
    try:
        layout = lambda P_, form: (0, P_ + P_ // 8, 2 * (P_ + P_ // 8) + 16)
        with pytest.raises(AssertionError, match="past-end read on the destination"):
            merge_levels(P, groups, "packed")
    finally:
        layout = saved
