"""Pins for the oracle's position search (CPU): inputs built by hand with the
answer planted at known indices, ties, NaN, infinite ratios and the 16-bit
storage types.  Each expected index comes from the construction, not from
re-evaluating the oracle's formula."""
import numpy as np
import pytest

import oracle

ATOL = RTOL = 1e-3


def stats_and_locate(r, c, dt="f32", flags=0):
    s = oracle.screen(r, c, dt, ATOL, RTOL, flags)
    return oracle.locate(r, c, dt, ATOL, RTOL, s["max_abs_err"], s["max_rel_err"], flags)


def base(n=1000, seed=0):
    rng = np.random.default_rng(seed)
    return (rng.uniform(1.0, 2.0, n)).astype(np.float32)  # |r| in [1, 2): no zeros


def test_identical_candidate_has_no_positions():
    r = base()
    assert stats_and_locate(r, r.copy()) == (-1, -1, -1)


def test_first_mismatch_is_the_lowest_planted_index():
    r = base()
    c = r.copy()
    for p in (700, 123, 450):
        c[p] = r[p] + 0.5
    fm, _, _ = stats_and_locate(r, c)
    assert fm == 123


def test_unique_largest_difference_and_ratio():
    r = base()
    c = r.copy()
    c[10] = r[10] + 0.25          # d = 0.25
    c[900] = r[900] + 0.75        # the unique largest d
    r2 = r.copy()
    # the largest ratio: a planted small reference value with a modest difference
    r2[333] = np.float32(0.01)
    c2 = c.copy()
    c2[333] = np.float32(0.02)    # ratio 1, others <= 0.75 / 1
    fm, ai, ri = stats_and_locate(r2, c2)
    assert (fm, ai, ri) == (10, 900, 333)


def test_ties_resolve_to_the_lowest_index():
    r = np.full(600, 2.0, dtype=np.float32)
    c = r.copy()
    for p in (599, 17, 250):
        c[p] = np.float32(2.5)    # the same difference and ratio at three places
    assert stats_and_locate(r, c) == (17, 17, 17)


def test_nan_is_a_mismatch_but_never_a_maximum():
    r = base()
    c = r.copy()
    c[40] = np.nan
    c[500] = r[500] + 0.125
    fm, ai, ri = stats_and_locate(r, c)
    assert fm == 40 and ai == 500 and ri == 500


def test_equal_nan_flag_removes_the_mismatch():
    r = base()
    r[7] = np.nan
    c = r.copy()
    assert stats_and_locate(r, c)[0] == 7                 # NaN never matches by default
    assert stats_and_locate(r, c, flags=oracle.EQUAL_NAN)[0] == -1


def test_infinite_ratio_at_a_zero_reference():
    # d > 0 over |r| = 0 is +inf; the first such element carries max_rel, the
    # small one (1e-9 <= atol) still matches, the large one is the first
    # mismatch and the largest difference

    r = base()
    c = r.copy()
    r[250], c[250] = 0.0, np.float32(1e-9)
    r[800], c[800] = 0.0, np.float32(3.0)
    fm, ai, ri = stats_and_locate(r, c)
    assert (fm, ai, ri) == (800, 800, 250)


@pytest.mark.parametrize("dt,conv", [("f16", oracle.f32_to_f16_n), ("bf16", oracle.f32_to_bf16_n)])
def test_sixteen_bit_storage(dt, conv):
    r32 = np.full(2048, 1.5, dtype=np.float32)
    c32 = r32.copy()
    c32[1500] = 1.75   # exactly representable in both 16-bit formats
    c32[64] = 1.625
    r = conv(r32)
    c = conv(c32)
    fm, ai, ri = stats_and_locate(r, c, dt)
    assert (fm, ai, ri) == (64, 1500, 1500)


def test_positions_agree_with_the_statistics():
    # consistency between the two oracle functions on random data: the
    # element at each position attains the recorded maximum
    rng = np.random.default_rng(5)
    r = rng.standard_normal(5000).astype(np.float32)
    c = (r + rng.standard_normal(5000).astype(np.float32) * 1e-3).astype(np.float32)
    s = oracle.screen(r, c, "f32", ATOL, RTOL)
    fm, ai, ri = oracle.locate(r, c, "f32", ATOL, RTOL, s["max_abs_err"], s["max_rel_err"])
    assert np.float32(abs(np.float32(c[ai] - r[ai]))) == np.float32(s["max_abs_err"])
    assert fm >= 0 and not oracle.match(float(c[fm]), float(r[fm]), ATOL, RTOL)
    assert all(oracle.match(float(c[i]), float(r[i]), ATOL, RTOL) for i in range(fm))
