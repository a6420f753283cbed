"""Parity of the rung statistics (kb_rung_stats) with the oracle (GPU).

The same binary64 timing samples go to the library (on the device) and to
the oracle.  Every field must be the same bits: the sort is exact, the
quantile interpolation, the tail ratios, the speedups and the score are each
evaluated with one rounding per operation in the order the definitions
give, and every sum runs left to right on both sides.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
import synth
from tests.helpers import ensure_built

pytestmark = pytest.mark.gpu

ROW_MAP = {"mean_us": "mean", "p50_us": "p50", "p90_us": "p90", "p95_us": "p95", "p99_us": "p99",
           "p90_over_p50": "tail90", "p95_over_p50": "tail95", "p99_over_p50": "tail99",
           "speedup_vs_base": "speedup", "n_samples": "n", "valid": "valid"}
SCORE_MAP = {"latency_us": "latency", "score": "score", "speedup_vs_base": "speedup",
             "valid": "valid"}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def same(a, b):
    if isinstance(a, float) and math.isnan(a):
        return isinstance(b, float) and math.isnan(b)
    return a == b


def check(samples, dev, base=0, rung=0, budget=0.0, alpha=0.02, beta=0.01, label=""):
    C, S, N = samples.shape
    grows, gscores = kb.rung_stats(torch.from_numpy(samples).to(dev), base, rung, budget, alpha, beta)
    orows, oscores = oracle.rung_stats(samples, base, rung, budget, alpha, beta)
    bad = []
    for c in range(C):
        for s in range(S):
            for gk, ok in ROW_MAP.items():
                if not same(grows[c][s][gk], orows[c][s][ok]):
                    bad.append(("row", c, s, gk, grows[c][s][gk], orows[c][s][ok]))
        for gk, ok in SCORE_MAP.items():
            if not same(gscores[c][gk], oscores[c][ok]):
                bad.append(("score", c, gk, gscores[c][gk], oscores[c][ok]))
    assert not bad, "%s: %d fields differ, first %s" % (label, len(bad), bad[:6])
    return grows, gscores


@pytest.mark.parametrize("n_iter", [1, 2, 3, 4, 5, 16, 31, 60, 63, 64, 65, 100, 128, 1000, 4095, 4096])
def test_iteration_counts(dev, n_iter):
    say("rung stats n_iter", n_iter)
    t = synth.timing_samples(9, 3, n_iter, seed=n_iter).numpy()
    check(t, dev, base=0, rung=1, budget=16.0, label="n_iter=%d" % n_iter)


@pytest.mark.parametrize("rung,budget", [(0, 4.0), (1, 16.0), (2, 60.0)])
@pytest.mark.parametrize("C,S", [(1, 1), (21, 3), (300, 1), (1024, 3)])
def test_rungs_and_sizes(dev, rung, budget, C, S):
    """The paper's rung schedule (4, 16, 60 repeats) over candidate lists
    from one to the bench size."""
    say("rung stats", rung, C, S)
    n = synth.RUNG_REPEATS[rung]
    t = synth.timing_samples(C, S, n, seed=100 * rung + C).numpy()
    check(t, dev, base=0, rung=rung, budget=budget, label="r%d C=%d S=%d" % (rung, C, S))


def test_ties_and_exact_values(dev):
    """Repeated values, constant rows and the closed forms of 1..N."""
    C, S, N = 4, 2, 101
    t = np.empty((C, S, N))
    t[0] = np.arange(1, N + 1)
    t[1] = 7.5
    t[2] = np.repeat(np.array([3.0, 4.0, 5.0]), [40, 40, 21])[None, :]
    t[3] = np.round(np.random.default_rng(3).uniform(10, 20, (S, N)), 1)
    for c in range(C):
        for s in range(S):
            np.random.default_rng(c * 7 + s).shuffle(t[c, s])
    rows, scores = check(t, dev, base=1, rung=2, budget=60.0, label="ties")
    assert rows[0][0]["p90_us"] == 91.0 and rows[0][0]["mean_us"] == 51.0
    assert rows[1][0]["p99_over_p50"] == 1.0


def test_invalid_samples_and_baselines(dev):
    t = synth.timing_samples(6, 2, 16, seed=9).numpy()
    t[1, 0, 3] = np.nan
    t[2, 1, 15] = np.inf
    t[3, 0, 0] = 0.0
    t[4, 1, 7] = -5.0
    for base in (0, -1, 1, 5):
        check(t, dev, base=base, rung=1, budget=16.0, label="invalid base=%d" % base)
    t2 = synth.timing_samples(6, 2, 100, seed=10).numpy()
    t2[1, 1, 99] = np.nan
    check(t2, dev, base=1, rung=1, budget=16.0, label="invalid long rows")


def test_sub_microsecond_latencies(dev):
    """Latencies at or below 1 us take the clamp of Eq. 2's leading term."""
    t = synth.timing_samples(5, 2, 16, seed=4, shape_us=[0.2, 0.9]).numpy()
    _, scores = check(t, dev, base=0, rung=0, budget=4.0, label="sub-us")
    assert any(s["score"] == 1e6 + 0.04 for s in scores)


def test_alpha_beta_variants(dev):
    t = synth.timing_samples(33, 3, 60, seed=12).numpy()
    for alpha, beta, budget in ((0.0, 0.0, 0.0), (1.0, 0.5, 123.25), (-0.3, 2.0, 7.0)):
        check(t, dev, base=2, rung=3, budget=budget, alpha=alpha, beta=beta,
              label="alpha=%g beta=%g" % (alpha, beta))
