"""Pins of the oracle's rung statistics (CPU).

Each check ties the oracle to something other than its own formulas:
numpy's linear percentile (the library definition the quantile reading
follows), closed forms on the samples 1..N and on constant rows, and the
properties the paper states for the runtime score (Eq. 2 and Section 3.1).
A plausible slip -- h = N p instead of (N - 1) p, a reversed sort, a mean
over N - 1, the ratio upside down, the clamp on the wrong side of 1 us, a
dropped rung term -- fails at least one of them.
"""
import math

import numpy as np
import pytest

import oracle

QS = (0.5, 0.9, 0.95, 0.99)
KEYS = ("p50", "p90", "p95", "p99")


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 10, 16, 17, 60, 63, 64, 65, 100, 101, 1000, 4096])
def test_quantiles_match_numpy_linear(n):
    rng = np.random.default_rng(n)
    for trial in range(5):
        t = rng.lognormal(3.0, 0.3, n)
        st = oracle.row_stats(t)
        for q, k in zip(QS, KEYS):
            want = float(np.percentile(t, 100 * q, method="linear"))
            # numpy evaluates the same interpolation in a different but
            # equivalent form: a few units in the last place apart at most
            assert math.isclose(st[k], want, rel_tol=4e-16, abs_tol=0.0), (n, q, st[k], want)


@pytest.mark.parametrize("n", [1, 2, 11, 21, 101, 1001])
def test_closed_forms_on_one_to_n(n):
    """Samples 1..N in any order: mean (N + 1) / 2; q(p) = 1 + (N - 1) p
    exactly where (N - 1) p is an integer."""
    t = np.arange(1, n + 1, dtype=np.float64)
    np.random.default_rng(n).shuffle(t)
    st = oracle.row_stats(t)
    assert st["mean"] == (n + 1) / 2
    assert st["p50"] == (n + 1) / 2
    if n == 101:
        assert (st["p90"], st["p95"], st["p99"]) == (91.0, 96.0, 100.0)
        assert st["tail90"] == 91.0 / 51.0
    if n == 1001:
        assert (st["p90"], st["p95"], st["p99"]) == (901.0, 951.0, 991.0)
    if n == 1:
        assert all(st[k] == 1.0 for k in KEYS)


def test_two_samples_interpolate():
    st = oracle.row_stats(np.array([30.0, 10.0]))
    assert st["p50"] == 20.0
    assert st["p90"] == 10.0 + 0.9 * 20.0
    assert st["p99"] == 10.0 + 0.99 * 20.0
    assert st["mean"] == 20.0


def test_constant_rows_and_order():
    st = oracle.row_stats(np.full(60, 123.25))
    assert st["mean"] == 123.25 and all(st[k] == 123.25 for k in KEYS)
    assert st["tail90"] == st["tail95"] == st["tail99"] == 1.0
    rng = np.random.default_rng(5)
    for n in (4, 16, 60):
        t = rng.gamma(2.0, 10.0, n) + 50.0
        st = oracle.row_stats(t)
        assert t.min() <= st["p50"] <= st["p90"] <= st["p95"] <= st["p99"] <= t.max()
        assert 1.0 <= st["tail90"] <= st["tail95"] <= st["tail99"]


def test_invalid_rows():
    for bad in ([1.0, float("nan")], [1.0, float("inf")], [1.0, 0.0], [2.0, -1.0]):
        st = oracle.row_stats(np.array(bad))
        assert st["valid"] == 0 and math.isnan(st["mean"]) and math.isnan(st["p50"])
    rows, sc = oracle.rung_stats(np.array([[[1.0, 2.0]], [[1.0, float("nan")]]]), base=0)
    assert sc[0]["valid"] == 1 and sc[1]["valid"] == 0
    assert sc[1]["score"] == -math.inf and math.isnan(sc[1]["latency"])
    assert math.isnan(rows[1][0]["speedup"])


def test_speedup_is_a_ratio_of_means():
    """Appendix A.5: speedup per shape = mean base time / mean optimized time."""
    base = np.array([[2.0, 2.0, 2.0, 2.0], [8.0, 8.0, 8.0, 8.0]])
    fast = np.array([[1.0, 1.0, 0.5, 1.5], [4.0, 3.0, 5.0, 4.0]])  # means 1 and 4
    rows, sc = oracle.rung_stats(np.stack([base, fast]), base=0)
    assert rows[1][0]["speedup"] == 2.0 and rows[1][1]["speedup"] == 2.0
    assert rows[0][0]["speedup"] == 1.0
    assert sc[0]["latency"] == 5.0 and sc[1]["latency"] == 2.5 and sc[1]["speedup"] == 2.0
    rows, sc = oracle.rung_stats(np.stack([base, fast]), base=-1)
    assert math.isnan(rows[1][0]["speedup"]) and math.isnan(sc[1]["speedup"])


def test_score_properties():
    """Eq. 2 and Section 3.1: the leading term is executions per second with
    the latency in us, clamped at 1 us; gamma(r) = alpha r + beta b_r is small
    and favours later rungs, which have larger budgets (repeats 4, 16, 60 in
    Appendix A.2)."""
    a, b = oracle.ALPHA, oracle.BETA
    assert (a, b) == (0.02, 0.01)
    budgets = {0: 4, 1: 16, 2: 60}
    # executions per second: 250 us -> 4000 per second, plus gamma
    assert oracle.rung_score_of(250.0, 0, 0.0) == 4000.0
    # every latency at or below 1 us scores the same
    s1 = {oracle.rung_score_of(x, 1, 16.0) for x in (1e-3, 0.5, 1.0)}
    assert len(s1) == 1 and s1.pop() == 1e6 + a * 1 + b * 16
    # equal latency: later rung (larger budget) scores higher, by gamma only
    for lat in (3.0, 250.0, 2606.0):
        s = [oracle.rung_score_of(lat, r, budgets[r]) for r in (0, 1, 2)]
        assert s[0] < s[1] < s[2]
        assert math.isclose(s[2] - s[0], a * 2 + b * (60 - 4), rel_tol=1e-9)
    # faster is always better, whatever the rungs, once the gap exceeds gamma
    assert oracle.rung_score_of(1000.0, 0, 4) > oracle.rung_score_of(1001.0, 2, 60)
    # gamma breaks near-ties: latencies whose leading terms differ by less
    # than gamma(2) - gamma(0) rank by rung
    assert oracle.rung_score_of(2606.0, 2, 60) > oracle.rung_score_of(2605.9, 0, 4)


# ------------------------------------------------------------- promotion ---

def test_survival_reproduces_table_a1_matvec():
    """Fig. 4 prints the MatVec run's counts: 21 enter rung 0, 5 fail, 7 are
    promoted; 7 enter rung 1, 2 fail, 3 are promoted; 3 enter rung 2, none
    fail.  Table A.1's MatVec row (Fail% of those entering, Promotion% of
    the original 21) must follow: 23.8, 33.3, 28.6, 14.3."""
    fail, promo = oracle.rung_survival([21, 7, 3], [5, 2, 0], [7, 3, 3], 21)
    assert [round(x, 1) for x in fail[:2]] == [23.8, 28.6]
    assert [round(x, 1) for x in promo[:2]] == [33.3, 14.3]
    assert fail[2] == 0.0


def test_promotion_rule_reproduces_fig4_counts():
    """With the fraction 2/5 of the successful non-baseline candidates (and
    the baseline carried), the rule promotes Fig. 4's numbers: 16 successes
    at rung 0 (15 and the baseline) -> six promoted plus the baseline; 5 at
    rung 1 (4 and the baseline) -> two plus the baseline -- whatever the
    scores."""
    rng = np.random.default_rng(44)
    for trial in range(50):
        s0 = rng.uniform(100, 1000, 21)
        v0 = np.ones(21, np.int32)
        v0[rng.choice(np.arange(1, 21), 5, replace=False)] = 0  # 5 failures, baseline 0 passes
        s0[v0 == 0] = -np.inf
        _, _, p0 = oracle.rung_promote(s0, v0, base=0, num=2, den=5)
        assert p0.sum() == 7 and p0[0] == 1
        survivors = np.flatnonzero(p0)
        v1 = np.ones(7, np.int32)
        v1[rng.choice(np.arange(1, 7), 2, replace=False)] = 0  # 2 fail at rung 1
        s1 = np.where(v1 == 1, rng.uniform(100, 1000, 7), -np.inf)
        _, _, p1 = oracle.rung_promote(s1, v1, base=0, num=2, den=5)
        assert p1.sum() == 3 and p1[0] == 1
        assert survivors.size == 7


def test_ranking_matches_a_library_sort():
    """Ranks against Python's sort on the key (-score, index): higher scores
    first, equal scores by the lower index; invalid (-inf) last."""
    rng = np.random.default_rng(7)
    for n in (1, 2, 5, 21, 100, 1000):
        s = np.round(rng.uniform(0, 10, n), 0)  # many ties
        v = (rng.uniform(size=n) > 0.2).astype(np.int32)
        s[v == 0] = -np.inf
        rank, order, _ = oracle.rung_promote(s, v, base=-1, num=1, den=2)
        want = sorted(range(n), key=lambda i: (-s[i], i))
        assert list(order) == want
        assert all(rank[order[r]] == r for r in range(n))


def test_promotion_hand_cases():
    inf = np.inf
    # ties broken by index; baseline carried although it ranks last
    rank, order, p = oracle.rung_promote([1.0, 5.0, 5.0, 2.0, 9.0], [1] * 5, base=0, num=1, den=2)
    assert list(order) == [4, 1, 2, 3, 0] and list(p) == [1, 1, 0, 0, 1]
    # fraction 0: only the baseline; fraction 1: every valid candidate
    _, _, p = oracle.rung_promote([3.0, 2.0, 1.0], [1, 1, 1], base=1, num=0, den=5)
    assert list(p) == [0, 1, 0]
    _, _, p = oracle.rung_promote([3.0, -inf, 1.0], [1, 0, 1], base=0, num=5, den=5)
    assert list(p) == [1, 0, 1]
    # an invalid baseline is not carried; no baseline at all
    _, _, p = oracle.rung_promote([-inf, 4.0, 8.0, 6.0], [0, 1, 1, 1], base=0, num=1, den=3)
    assert list(p) == [0, 0, 1, 0]
    _, _, p = oracle.rung_promote([4.0, 8.0, 6.0], [1, 1, 1], base=-1, num=2, den=3)
    assert list(p) == [0, 1, 1]
    # ceil, in integers: 7 eligible at 2/5 -> 3 (14/5 = 2.8)
    _, _, p = oracle.rung_promote(np.arange(8.0), [1] * 8, base=0, num=2, den=5)
    assert p.sum() == 4 and list(np.flatnonzero(p)) == [0, 5, 6, 7]


def test_invalid_and_nan_rank_last():
    """Pruned candidates (invalid, or a NaN score) rank after every valid
    one, in index order, whatever their score field holds."""
    s = np.array([np.nan, 5.0, 7.0, 1e9, 2.0])
    v = np.array([1, 1, 1, 0, 1], np.int32)
    rank, order, p = oracle.rung_promote(s, v, base=-1, num=1, den=1)
    assert list(order) == [2, 1, 4, 0, 3]
    assert list(p) == [1, 1, 1, 0, 1]
