"""Pins for the oracle's screening statistics (CPU only).

Hand-built cases with answers worked out from the definition (the tolerance
test |c - r| <= atol + rtol*|r| in binary32 with two roundings, NaN never
matching unless the equal-NaN flag is set, equal infinities matching, maxima
ignoring NaN, squared-error sums over finite pairs), closed forms for the
relative L2 error, invariants under Hypothesis, and a brute-force sweep of
special values against exact rational arithmetic.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from tests.exact import round_to_f32

INF = float("inf")
NAN = float("nan")


def f32a(*vals):
    return np.array(vals, dtype=np.float32)


def scr(r, c, atol, rtol, flags=0, dtype="f32"):
    return oracle.screen(r, c, dtype, atol, rtol, flags)


def assert_stats(s, **want):
    for k, v in want.items():
        got = s[k]
        if isinstance(v, float) and math.isnan(v):
            assert math.isnan(got), (k, got)
        else:
            assert got == v, (k, got, v)


# ---------------------------------------------------------- hand cases ---

def test_h1_identical_candidate():
    r = oracle.gen("f32", 1000, oracle.DIST_NORMAL, seed=0, stream_id=1)
    s = scr(r, r.copy(), 1e-5, 1e-5)
    assert_stats(s, numel=1000, mismatches=0, bitwise_equal=1, max_abs_err=0.0,
                 max_rel_err=0.0, rel_l2=0.0, sum_sq_diff=0.0, passed=1)
    assert s["sum_sq_ref"] > 0


def test_h2_signed_zero():
    s = scr(f32a(0.0), f32a(-0.0), 0.0, 0.0)
    assert_stats(s, mismatches=0, bitwise_equal=0, max_abs_err=0.0, max_rel_err=0.0,
                 rel_l2=0.0, sum_sq_ref=0.0)


def test_h3_nan_candidate():
    s = scr(f32a(1.0), f32a(NAN), 1e-5, 1e-5)
    assert_stats(s, mismatches=1, nan_count=1, max_abs_err=0.0, max_rel_err=0.0,
                 sum_sq_diff=0.0, sum_sq_ref=1.0, rel_l2=0.0, passed=0)


def test_h4_equal_infinities_match():
    s = scr(f32a(INF), f32a(INF), 1e-5, 1e-5)
    assert_stats(s, mismatches=0, pos_inf_count=1, max_abs_err=0.0, sum_sq_ref=0.0,
                 rel_l2=0.0, bitwise_equal=1)


def test_h5_opposite_infinities():
    s = scr(f32a(INF), f32a(-INF), 1e-5, 1e-5)
    assert_stats(s, mismatches=1, neg_inf_count=1, pos_inf_count=0, max_abs_err=INF,
                 max_rel_err=0.0)


def test_h6_finite_against_infinite_reference():
    s = scr(f32a(INF), f32a(5.0), 1e-5, 1e-5)
    assert_stats(s, mismatches=1, max_abs_err=INF, max_rel_err=0.0, sum_sq_diff=0.0)


def test_h7_zero_reference():
    s = scr(f32a(0.0), f32a(1.0), 0.0, 0.5)
    assert_stats(s, mismatches=1, max_abs_err=1.0, max_rel_err=INF, sum_sq_diff=1.0,
                 sum_sq_ref=0.0, rel_l2=INF)


def test_h8_boundary_is_inclusive():
    rtol = 2.0**-10
    s = scr(f32a(1.0), f32a(1.0 + 2.0**-10), 0.0, rtol)
    assert_stats(s, mismatches=0, max_abs_err=2.0**-10, max_rel_err=2.0**-10)
    s = scr(f32a(1.0), f32a(1.0 + 2.0**-10 + 2.0**-23), 0.0, rtol)
    assert_stats(s, mismatches=1)


def test_h9_subnormal_tolerance_rounds_to_zero():
    tiny = 2.0**-149
    # rtol*|r| = 2^-150 is a tie between 0 and 2^-149 and rounds to even (0)
    s = scr(f32a(tiny), f32a(0.0), 0.0, 0.5)
    assert_stats(s, mismatches=1, max_abs_err=tiny, max_rel_err=1.0)


def test_h10_subnormal_difference():
    s = scr(f32a(2.0**-149), f32a(2.0**-148), 1e-8, 0.0)
    assert_stats(s, mismatches=0, max_abs_err=2.0**-149, max_rel_err=1.0)


def test_h11_f16_overflow_to_infinity():
    r = np.array([0x7BFF], dtype=np.uint16)  # 65504
    c = np.array([0x7C00], dtype=np.uint16)  # +inf
    s = scr(r, c, 1e-3, 1e-3, dtype="f16")
    assert_stats(s, mismatches=1, pos_inf_count=1, max_abs_err=INF, max_rel_err=INF,
                 sum_sq_diff=0.0, sum_sq_ref=65504.0**2, rel_l2=0.0)


def test_h12_bf16_one_ulp():
    r = np.array([0x3F80], dtype=np.uint16)  # 1.0
    c = np.array([0x3F81], dtype=np.uint16)  # 1 + 2^-7
    s = scr(r, c, 1e-2, 1e-2, dtype="bf16")
    assert_stats(s, mismatches=0, bitwise_equal=0, max_abs_err=2.0**-7, max_rel_err=2.0**-7)


def test_h13_mixed_vector():
    r = f32a(1, 2, 3, 4, 5, 6, 7, 8)
    c = f32a(1, NAN, INF, -INF, 5.1, 6, 7, 8)
    s = scr(r, c, 1e-5, 1e-5)
    d = float(np.float32(5.1)) - 5.0  # exact: same binade
    assert_stats(s, mismatches=4, nan_count=1, pos_inf_count=1, neg_inf_count=1,
                 max_abs_err=INF, max_rel_err=INF, sum_sq_diff=d * d, sum_sq_ref=204.0)
    assert s["rel_l2"] == pytest.approx(math.sqrt(d * d / 204.0), rel=1e-15)


def test_h14_equal_nan_flag():
    s = scr(f32a(NAN), f32a(NAN), 1e-5, 1e-5)
    assert_stats(s, mismatches=1, nan_count=1, max_abs_err=0.0, sum_sq_ref=0.0, rel_l2=0.0)
    s = scr(f32a(NAN), f32a(NAN), 1e-5, 1e-5, flags=oracle.EQUAL_NAN)
    assert_stats(s, mismatches=0, nan_count=1)
    # the flag does not make NaN match a number
    s = scr(f32a(1.0), f32a(NAN), 1e-5, 1e-5, flags=oracle.EQUAL_NAN)
    assert_stats(s, mismatches=1)


def _exact_f32_round(x: Fraction) -> float:
    return round_to_f32(x)


def test_h15_tolerance_uses_two_roundings():
    # Find (r, atol, rtol) where fl(atol + fl(rtol*|r|)) differs from the
    # fused fl(atol + rtol*|r|); place c at |c - r| equal to the two-rounding
    # tolerance.  The two-rounding rule matches; a fused tolerance would not.
    rng = np.random.default_rng(15)
    found = 0
    for _ in range(200000):
        r = np.float32(rng.uniform(0.5, 2.0))
        atol = np.float32(rng.uniform(1e-4, 1e-2))
        rtol = np.float32(rng.uniform(1e-4, 1e-2))
        t2 = np.float32(atol + np.float32(rtol * r))
        tf = _exact_f32_round(Fraction(float(atol)) + Fraction(float(rtol)) * Fraction(float(r)))
        if float(t2) <= tf:
            continue
        c = np.float32(r + t2)
        if np.float32(c - r) != t2:
            continue
        s = scr(f32a(r), f32a(c), float(atol), float(rtol))
        assert s["mismatches"] == 0, (r, atol, rtol, c)
        found += 1
        if found == 20:
            break
    assert found == 20


def test_h16_relative_error_uses_the_reference():
    # max rel comes from the second element, max abs from the first
    r = f32a(1000.0, 1e-3)
    c = f32a(1001.0, 2e-3)
    s = scr(r, c, 0.0, 0.0)
    assert s["max_abs_err"] == 1.0
    assert s["max_rel_err"] == float(np.float32(np.float32(2e-3) - np.float32(1e-3))
                                     / np.float32(1e-3))
    # a binary32 quotient: 1/3 rounded once
    s = scr(f32a(3.0), f32a(4.0), 0.0, 0.0)
    assert s["max_rel_err"] == float(np.float32(1.0) / np.float32(3.0))


def test_overflowing_difference_is_an_infinite_squared_error():
    # both values finite, c - r overflows binary32: the term is +inf, and so
    # is the sum and the relative L2 error (not NaN)
    fmax = 3.4028234663852886e38
    s = scr(f32a(fmax, 1.0), f32a(-fmax, 1.0), 1e-5, 1e-5)
    assert_stats(s, mismatches=1, max_abs_err=INF, max_rel_err=INF, sum_sq_diff=INF,
                 sum_sq_ref=fmax * fmax + 1.0, rel_l2=INF)
    parts = oracle.screen(f32a(fmax, 1.0, 2.0), f32a(-fmax, 1.0, 2.5), "f32", 1e-5, 1e-5, chunk=1)
    assert parts["sum_sq_diff"] == INF and parts["rel_l2"] == INF


def test_rel_l2_closed_form():
    s = scr(f32a(3.0, 4.0), f32a(3.5, 4.0), 0.0, 0.0)
    assert s["sum_sq_diff"] == 0.25 and s["sum_sq_ref"] == 25.0
    assert s["rel_l2"] == pytest.approx(0.1, rel=1e-15)


def test_empty_input():
    s = scr(f32a(), f32a(), 1e-5, 1e-5)
    assert_stats(s, numel=0, mismatches=0, bitwise_equal=1, max_abs_err=0.0, rel_l2=0.0,
                 passed=1)


# ---------------------------------------------------- brute force grid ---

SPECIALS = [0.0, -0.0, 2.0**-149, -(2.0**-149), 2.0**-126, 1e-8, 1e-6, 0.5, 1.0, -1.0,
            1.0 + 2.0**-23, 3.0, 65504.0, 3.4028234663852886e38, -3.4028234663852886e38,
            INF, -INF, NAN]


def _exact_stats_pair(c, r, atol, rtol):
    """Match bit, d and q of one pair from exact rationals rounded explicitly."""
    fin = lambda x: math.isfinite(x)
    if math.isnan(c) or math.isnan(r):
        match = False
        d = NAN
    else:
        if fin(c) and fin(r):
            d = _exact_f32_round(abs(Fraction(c) - Fraction(r)))
        elif c == r:
            d = NAN
        else:
            d = INF
        if c == r:
            match = True
        elif fin(r):
            tol = _exact_f32_round(Fraction(atol) + Fraction(_exact_f32_round(Fraction(rtol) * abs(Fraction(r)))))
            match = (not math.isnan(d)) and d <= tol
        else:
            match = False
    return match, d


def test_brute_force_special_pairs():
    atol, rtol = float(np.float32(1e-5)), float(np.float32(1e-5))
    for c in SPECIALS:
        for r in SPECIALS:
            s = scr(f32a(r), f32a(c), atol, rtol)
            match, d = _exact_stats_pair(c, r, atol, rtol)
            assert s["mismatches"] == (0 if match else 1), (c, r)
            want_abs = d if (not math.isnan(d) and d > 0) else 0.0
            assert s["max_abs_err"] == want_abs, (c, r, s["max_abs_err"], want_abs)


# ------------------------------------------------------------ invariants ---

finite32 = st.floats(width=32, allow_nan=False, allow_infinity=False)
any32 = st.floats(width=32, allow_nan=True, allow_infinity=True)


@st.composite
def pairs(draw, elements=any32, min_size=0, max_size=64):
    n = draw(st.integers(min_size, max_size))
    r = draw(st.lists(elements, min_size=n, max_size=n))
    c = draw(st.lists(elements, min_size=n, max_size=n))
    return f32a(*r) if n else f32a(), f32a(*c) if n else f32a()


TMAX = float(np.float32(1e-2))
tols = st.tuples(st.floats(0, TMAX, width=32), st.floats(0, TMAX, width=32))


@settings(max_examples=200, deadline=None)
@given(st.lists(st.floats(width=32, allow_nan=False), max_size=64), tols)
def test_i1_identical_without_nan(vals, tol):
    r = f32a(*vals) if vals else f32a()
    s = scr(r, r.copy(), *tol)
    assert s["mismatches"] == 0 and s["bitwise_equal"] == 1
    assert s["max_abs_err"] == 0.0 and s["max_rel_err"] == 0.0 and s["rel_l2"] == 0.0


@settings(max_examples=200, deadline=None)
@given(pairs(), tols, st.randoms(use_true_random=False))
def test_i2_permutation_invariance(rc, tol, rnd):
    r, c = rc
    perm = list(range(r.size))
    rnd.shuffle(perm)
    a = scr(r, c, *tol)
    b = scr(r[perm], c[perm], *tol)
    for k in ("numel", "mismatches", "nan_count", "pos_inf_count", "neg_inf_count",
              "max_abs_err", "max_rel_err", "bitwise_equal"):
        assert a[k] == b[k], k
    for k in ("sum_sq_diff", "sum_sq_ref"):
        assert a[k] == pytest.approx(b[k], rel=1e-12, abs=0)


@settings(max_examples=200, deadline=None)
@given(pairs(max_size=128), tols, st.integers(1, 40))
def test_i3_chunk_and_merge(rc, tol, chunk):
    r, c = rc
    whole = scr(r, c, *tol)
    parts = oracle.screen(r, c, "f32", tol[0], tol[1], chunk=chunk)
    for k in whole:
        if k in ("sum_sq_diff", "sum_sq_ref", "rel_l2"):
            assert parts[k] == pytest.approx(whole[k], rel=1e-12, abs=0) or (
                math.isinf(whole[k]) and parts[k] == whole[k])
        else:
            assert parts[k] == whole[k], k


@settings(max_examples=200, deadline=None)
@given(pairs(), tols, tols)
def test_i5_i6_i9_monotone_tolerance(rc, t1, t2):
    r, c = rc
    lo = (min(t1[0], t2[0]), min(t1[1], t2[1]))
    hi = (max(t1[0], t2[0]), max(t1[1], t2[1]))
    a = scr(r, c, *lo)
    b = scr(r, c, *hi)
    assert b["mismatches"] <= a["mismatches"] <= r.size
    assert a["nan_count"] <= a["mismatches"]


@settings(max_examples=200, deadline=None)
@given(pairs(elements=st.floats(2.0**-40, 2.0**40, width=32) | st.floats(-(2.0**40), -(2.0**-40), width=32)),
       tols, st.integers(-30, 30))
def test_i7_power_of_two_scaling(rc, tol, e):
    r, c = rc
    scale = np.float32(2.0**e)
    a = scr(r, c, *tol)
    b = scr(r * scale, c * scale, float(np.float32(tol[0]) * scale), tol[1])
    assert a["mismatches"] == b["mismatches"]
    assert a["max_rel_err"] == b["max_rel_err"]
    assert b["max_abs_err"] == float(np.float32(a["max_abs_err"]) * scale)


@settings(max_examples=100, deadline=None)
@given(st.integers(1, 500), st.integers(0, 50), st.integers(0, 2**32 - 1))
def test_i8_nan_positions_counted_exactly(n, m, seed):
    rng = np.random.default_rng(seed)
    r = rng.standard_normal(n).astype(np.float32)
    c = r.copy()
    m = min(m, n)
    idx = rng.choice(n, size=m, replace=False)
    c[idx] = np.float32(NAN)
    s = scr(r, c, 1e-5, 1e-5)
    assert s["nan_count"] == m and s["mismatches"] == m


def test_16bit_widening_matches_f32_screen():
    # a 16-bit screen is the binary32 screen of the exactly widened values
    rng = np.random.default_rng(3)
    for dt, widen in (("f16", oracle.f16_to_f32_n), ("bf16", oracle.bf16_to_f32_n)):
        r = rng.integers(0, 1 << 16, size=4096, dtype=np.uint32).astype(np.uint16)
        c = r.copy()
        flip = rng.random(4096) < 0.3
        c[flip] ^= rng.integers(1, 64, size=int(flip.sum()), dtype=np.uint32).astype(np.uint16)
        s16 = scr(r, c, 1e-3, 1e-3, dtype=dt)
        s32 = scr(widen(r), widen(c), 1e-3, 1e-3)
        for k in s16:
            if k == "bitwise_equal":
                continue
            if isinstance(s16[k], float) and math.isnan(s16[k]):
                assert math.isnan(s32[k])
            else:
                assert s16[k] == s32[k], k
