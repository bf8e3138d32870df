"""Pins of the oracle's scoring arithmetic against values fixed by the paper's
equations: hand-derived fixed-point worked examples, exact special cases and
error bounds of the fp32 path.  No GPU."""
import numpy as np
import pytest

import oracle

B_H, P_Z = 12, 500_000_000       # the locked format, eq. (lock)


def flat(d, n):
    return np.full(51, d, np.uint32), np.full(51, n, np.uint32)


# ------------------------------------------------------------- fixed point
# Worked by hand from eq. (uq), eq. (hq), eq. (survq), eq. (t1), eq. (t2),
# eq. (scoreq):  Lambda = 4095, floor(0.01*4095 + 1/2) = 41.

def test_fixed_h0_score_is_gap():
    d, n = flat(0, 1)                     # h = 0 -> sigma_q = Lambda, T2 = 0
    g = np.array([0, 1, 12345, 2_000_000, 2 ** 32 - 1], np.uint64)
    out = oracle.score_fixed(np.zeros(5), g, np.zeros(5), d, n, B_H, P_Z)
    assert out.tolist() == g.tolist()


def test_fixed_h1_penalty_term():
    d, n = flat(7, 7)                     # h = 1 -> h_q = 4095, sigma_q = 41
    out = oracle.score_fixed([3], [0], [0], d, n, B_H, P_Z)
    # T2 = floor((4095 - 41) * 5e8 / 4095) = floor(494,993,894.99)
    assert int(out[0]) == 494_993_894
    out = oracle.score_fixed([3], [41], [0], d, n, B_H, P_Z)
    # T1 = floor(41 * 4095 / 41) = 4095
    assert int(out[0]) == 494_993_894 + 4095


def test_fixed_worked_example_h_1_24():
    d, n = flat(1, 24)
    # h_q = floor(4095/24 + 1/2) = floor(171.125) = 171; sigma_q = 3924
    assert oracle.lut_q(d, n, B_H)[0] == 171
    out = oracle.score_fixed([5], [2_000_000], [0], d, n, B_H, P_Z)
    # T1 = floor(2e6*4095/3924) = 2,087,155 ; T2 = floor(171*5e8/4095) = 20,879,120
    assert int(out[0]) == 2_087_155 + 20_879_120 == 22_966_275


def test_fixed_b16_floor_and_penalty():
    d, n = flat(3, 3)
    # Lambda = 65535: floor(655.35 + 0.5) = 655 ; T2 = floor(64880*5e8/65535)
    out = oracle.score_fixed([0], [0], [0], d, n, 16, P_Z)
    assert int(out[0]) == 495_002_670


def test_fixed_done_is_saturated():
    d, n = flat(1, 24)
    out = oracle.score_fixed([0, 50, 60], [5, 0, 2 ** 32 - 1], [1, 1, 1], d, n, B_H, P_Z)
    assert all(int(v) == 2 ** 64 - 1 for v in out)


def test_fixed_saturates_at_64_bits():
    d, n = flat(1, 1)
    out = oracle.score_fixed([0], [2 ** 64 - 1], [0], d, n, B_H, 2 ** 63)
    assert int(out[0]) == 2 ** 64 - 1


def test_quantizer_special_points():
    # Q(0) = 0, Q(1) = Lambda, Q(1/2) = floor(2047.5 + 0.5) = 2048, rounding at .5 goes up
    assert oracle.lut_q(*flat(0, 5), 12)[0] == 0
    assert oracle.lut_q(*flat(5, 5), 12)[0] == 4095
    assert oracle.lut_q(*flat(1, 2), 12)[0] == 2048
    assert oracle.lut_q(*flat(1, 2), 1)[0] == 1          # 1/2 * 1 + 1/2 = 1
    assert oracle.lut_q(*flat(1, 3), 1)[0] == 0          # 1/3 + 1/2 < 1
    assert oracle.lut_q(*flat(0, 0), 12)[0] == 0          # n = 0 -> h = 0


def test_fixed_turn_clamps_at_50():
    d = np.zeros(51, np.uint32)
    n = np.ones(51, np.uint32)
    d[50] = 1                                      # h(50) = 1, others 0
    out = oracle.score_fixed([49, 50, 51, 200], [1000] * 4, [0] * 4, d, n, B_H, P_Z)
    assert int(out[0]) == 1000
    assert out[1] == out[2] == out[3] != out[0]


def test_fixed_monotone_in_gap_and_hazard():
    rng = np.random.default_rng(3)
    g = np.sort(rng.integers(0, 2 ** 32, 200).astype(np.uint64))
    for dd in (0, 1, 5, 23, 24):
        out = oracle.score_fixed(np.zeros(200), g, np.zeros(200), *flat(dd, 24), B_H, P_Z)
        assert np.all(np.diff(out.astype(object)) >= 0)
    prev = None
    for dd in range(25):                            # larger hazard -> larger score
        v = int(oracle.score_fixed([0], [123456], [0], *flat(dd, 24), B_H, P_Z)[0])
        assert prev is None or v >= prev
        prev = v


# -------------------------------------------------------------- EMA pins

def test_integer_ema_sequence():
    # eq. (ema-int) at tau = 1 us on gaps of 2, 4, 1 s from g_q = 0:
    # 600,000 -> 1,620,000 -> 1,434,000
    gaps = np.array([[2_000_000_000, 4_000_000_000, 1_000_000_000]], np.uint64)
    want = [0, 600_000, 1_620_000, 1_434_000]
    for k in range(4):
        g, gq = oracle.ema_replay(gaps, [k])
        assert int(gq[0]) == want[k]
        # every intermediate value is an integer below 2^24: the fp32 EMA is exact
        assert float(g[0]) == want[k]


def test_integer_ema_gap_clip():
    gaps = np.array([[2 ** 60, 0]], np.uint64)
    _, gq = oracle.ema_replay(gaps, [1], b_g=32, tau_ns=1000)
    assert int(gq[0]) == (3 * (2 ** 32 - 1)) // 10        # eq. (gapq) clip
    _, gq = oracle.ema_replay(gaps, [1], b_g=64, tau_ns=1)
    assert int(gq[0]) == (3 * 2 ** 60) // 10


def test_float_ema_within_rounding_bound():
    """eq. (ema) on whole-microsecond samples: the fp32 register stays within
    its rounding bound of the exact rational EMA."""
    from fractions import Fraction
    rng = np.random.default_rng(11)
    gaps = rng.integers(1_000_000, 300_000_000_000, (300, 8)).astype(np.uint64)
    gaps[0, 0] = 999           # below one microsecond: the sample is 0
    nh = rng.integers(0, 9, 300).astype(np.uint8)
    nh[0] = 1
    g, _ = oracle.ema_replay(gaps, nh)
    assert float(g[0]) == 0.0
    for i in range(300):
        ref = Fraction(0)
        for k in range(nh[i]):
            ref = (3 * Fraction(int(gaps[i, k]) // 1000) + 7 * ref) / 10
        assert abs(float(g[i]) - float(ref)) <= 2e-6 * max(float(ref), 1.0)


def test_ema_sample_clips_at_32_bits():
    gaps = np.array([[(2 ** 32 + 5) * 1000, 0]], np.uint64)
    g, gq = oracle.ema_replay(gaps, [1], b_g=32)
    assert int(gq[0]) == (3 * (2 ** 32 - 1)) // 10
    assert float(g[0]) == np.float32(np.float32(3.0) * np.float32(2 ** 32 - 1)) / np.float32(10)


# ------------------------------------------------------------ fp32 score

def test_f32_h0_score_is_gap_exactly():
    rng = np.random.default_rng(5)
    g = (rng.random(1000) * 3e8).astype(np.float32)
    out = oracle.score_f32(rng.integers(0, 60, 1000), g, np.zeros(1000), *flat(0, 9), 5e8)
    assert np.array_equal(out.view(np.uint32), g.view(np.uint32))


def test_f32_done_is_inf():
    out = oracle.score_f32([0, 7], [1.0, 0.0], [1, 1], *flat(1, 9), 5e8)
    assert np.all(np.isinf(out)) and np.all(out > 0)


def test_f32_sigma_floor():
    # h >= 0.99 -> sigma = 0.01f: score = g/0.01 + 0.99 P (within fp32 rounding)
    g = np.array([0.0, 1.0, 5e6, 2e8], np.float32)
    for d, n in ((99, 100), (1, 1), (250, 251)):
        out = oracle.score_f32(np.zeros(4), g, np.zeros(4), *flat(d, n), 5e8)
        sigma = 0.01
        ref = g.astype(np.float64) / sigma + (1 - sigma) * 5e8
        assert np.allclose(out, ref, rtol=4e-7, atol=0)


def test_f32_matches_real_formula_within_bound():
    rng = np.random.default_rng(9)
    n = 5000
    turn = rng.integers(0, 70, n)
    g = (rng.lognormal(np.log(4e6), 1.5, n)).astype(np.float32)
    d = rng.integers(0, 30, 51).astype(np.uint32)
    nn = (d + rng.integers(0, 200, 51)).astype(np.uint32)
    for P in (5e8, 5e7, 0.0):
        out = oracle.score_f32(turn, g, np.zeros(n), d, nn, P)
        t = np.minimum(turn, 50)
        h = np.where(nn[t] > 0, d[t] / np.maximum(nn[t], 1), 0.0)
        sig = np.maximum(0.01, 1 - h)
        ref = g.astype(np.float64) / sig + (1 - sig) * P
        # u = 2^-24.  sigma = fl(1 - fl(h)) carries an absolute error <= u(1 + h),
        # i.e. a relative error <= u(1 + h/sigma) after the cancellation; so
        # a = g/sigma is off by <= a*u*(3 + 2h/sigma), b = 1 - sigma (exact by
        # Sterbenz) by <= 2u absolutely, c = b*P by <= 3uP, the sum by u*ref.
        u = 2.0 ** -24
        a = g.astype(np.float64) / sig
        bound = a * u * (3 + 2 * h / sig) + 3 * u * P + 2 * u * ref
        assert np.all(np.abs(out - ref) <= bound)


def test_f32_lut_is_ratio_of_counts():
    d = np.arange(51, dtype=np.uint32)
    n = (np.arange(51) * 3 + 1).astype(np.uint32)
    hf = oracle.lut_f32(d, n)
    assert np.all(np.abs(hf - d / n) <= 2.0 ** -24 * (d / n))
    assert oracle.lut_f32(*flat(0, 0))[0] == 0.0


# ---------------------------------------------- reciprocal-table divider
# The sweep's other divider type: eq. (t1) multiplies by r[sigma_q] =
# floor(2^W / sigma_q + 1/2), read from a table of depth Lambda, and shifts
# right by W.  Worked by hand for the (g_q = 2e6, h = 1/24) example above,
# where sigma_q = 3924 and the exact T1 is 2,087,155:
#   W = 16: 65,536 / 3924 = 16.70  -> r = 17;
#           T1 = floor(2e6 * 4095 * 17 / 65,536) = floor(2,124,481.2) = 2,124,481
#   W = 24: 16,777,216 / 3924 = 4275.54 -> r = 4276;
#           T1 = floor(8.19e9 * 4276 / 16,777,216) = floor(2,087,380.9) = 2,087,380

def test_reciprocal_divider_worked_example():
    d, n = flat(1, 24)
    for w, t1 in ((16, 2_124_481), (24, 2_087_380)):
        out = oracle.score_fixed([5], [2_000_000], [0], d, n, B_H, P_Z, recip_bits=w)
        assert int(out[0]) == t1 + 20_879_120, w


def test_reciprocal_divider_is_exact_on_powers_of_two():
    """sigma_q = 2048 (h_q = 2047, from d/n = 2047/4095) divides 2^W: the
    stored reciprocal is exact and so is T1."""
    d, n = flat(2047, 4095)
    assert oracle.lut_q(d, n, B_H)[0] == 2047
    g = np.array([0, 1, 999, 2_000_000, 2 ** 40 + 3], np.uint64)
    exact = oracle.score_fixed(np.zeros(5), g, np.zeros(5), d, n, B_H, P_Z)
    for w in (12, 16, 24):
        lut = oracle.score_fixed(np.zeros(5), g, np.zeros(5), d, n, B_H, P_Z, recip_bits=w)
        assert lut.tolist() == exact.tolist(), w


@pytest.mark.parametrize("w", [8, 12, 16, 20, 24, 32])
def test_reciprocal_divider_error_bound(w):
    """|r - 2^W / sigma| <= 1/2, so |T1_lut - T1_exact| <= g_q Lambda / 2^(W+1) + 1
    (the two floors add at most 1): checked on random gaps and every sigma_q
    the hazard counts reach, at b_h = 8, 12 and 16; T2 is the same in both."""
    rng = np.random.default_rng(w)
    for b_h in (8, 12, 16):
        lam = 2 ** b_h - 1
        for _ in range(20):
            nn = int(rng.integers(1, 500))
            dd = int(rng.integers(0, nn + 1))
            d, n = flat(dd, nn)
            g = rng.integers(0, 2 ** 36, 64, dtype=np.uint64)
            exact = oracle.score_fixed(np.zeros(64), g, np.zeros(64), d, n, b_h, 0)
            lut = oracle.score_fixed(np.zeros(64), g, np.zeros(64), d, n, b_h, 0, recip_bits=w)
            bound = g.astype(object) * lam / 2 ** (w + 1) + 1
            diff = np.abs(lut.astype(object) - exact.astype(object))
            assert all(x <= b for x, b in zip(diff, bound)), (b_h, dd, nn)


def test_reciprocal_divider_off_is_the_exact_score():
    d, n = flat(1, 24)
    g = np.array([0, 7, 2_000_000], np.uint64)
    a = oracle.score_fixed([0, 3, 9], g, [0, 0, 0], d, n, B_H, P_Z)
    b = oracle.score_fixed([0, 3, 9], g, [0, 0, 0], d, n, B_H, P_Z, recip_bits=0)
    assert a.tolist() == b.tolist()
