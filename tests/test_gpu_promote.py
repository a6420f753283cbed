"""The promotion decision (kb_rung_promote) against the oracle, and the
three-rung funnel of Fig. 4 run end to end on the device (GPU).

Ranks, orders and promotion flags are integers: they must be equal.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
import synth
from tests.helpers import ensure_built, oracle_records

pytestmark = pytest.mark.gpu

SCORE_DTYPE = np.dtype([("latency_us", "<f8"), ("score", "<f8"), ("speedup_vs_base", "<f8"),
                        ("valid", "<i4"), ("reserved", "<i4")])
assert SCORE_DTYPE.itemsize == 32


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def score_buffer(scores, valid, dev):
    a = np.zeros(len(scores), SCORE_DTYPE)
    a["score"] = scores
    a["valid"] = valid
    a["latency_us"] = 1.0
    return torch.from_numpy(a.view(np.uint8).copy()).to(dev)


def check(scores, valid, dev, base, num, den, label=""):
    n = len(scores)
    buf = score_buffer(scores, valid, dev)
    rank, order, prom = kb.kb_rung_promote(buf, n, base, num, den)
    o_rank, o_order, o_prom = oracle.rung_promote(scores, valid, base, num, den)
    g = rank.cpu().numpy(), order.cpu().numpy(), prom.cpu().numpy()
    assert np.array_equal(g[0], o_rank), (label, "rank")
    assert np.array_equal(g[1], o_order), (label, "order")
    assert np.array_equal(g[2], o_prom), (label, "promoted")
    return g


@pytest.mark.parametrize("n", [1, 2, 3, 21, 255, 256, 257, 1000, 4096, 65536])
def test_random_scores(dev, n):
    say("promote n", n)
    rng = np.random.default_rng(n)
    for trial, (num, den) in enumerate(((2, 5), (1, 3), (0, 1), (1, 1), (1, 2))):
        s = np.round(rng.uniform(0, 50, n), 0) * 1.5 + 100.0  # many ties
        v = (rng.uniform(size=n) > 0.15).astype(np.int32)
        junk = rng.choice([np.nan, np.inf, 1e300, -np.inf, 7.0], size=n)
        s = np.where(v == 1, s, junk)
        base = [-1, 0, n // 2, n - 1, 0][trial]
        check(s, v, dev, base, num, den, "n=%d %d/%d base=%d" % (n, num, den, base))


def test_nan_scores_invalid_baseline_and_all_equal(dev):
    check(np.array([np.nan, 5.0, 7.0, 1e9, 2.0]), np.array([1, 1, 1, 0, 1], np.int32), dev, -1, 1, 1,
          "nan")
    check(np.array([-np.inf, 4.0, 8.0, 6.0]), np.array([0, 1, 1, 1], np.int32), dev, 0, 1, 3,
          "invalid base")
    check(np.full(300, 42.0), np.ones(300, np.int32), dev, 17, 2, 5, "all equal")
    check(np.zeros(9), np.zeros(9, np.int32), dev, 3, 2, 5, "all invalid")


def outputs_for(ref, fails, k):
    """Candidate k's output: the reference with in-tolerance noise, or with a
    block of wrong values when it fails."""
    g = torch.Generator(device=ref.device).manual_seed(1000 + k)
    out = ref + 1e-7 * torch.randn(ref.shape, generator=g, device=ref.device, dtype=ref.dtype)
    if k in fails:
        out[100 * k: 100 * k + 50] += 1.0
    return out


def test_fig4_funnel_on_device(dev):
    """The MatVec run of Fig. 4, replayed with synthetic outputs and timings:
    21 candidates (index 0 the baseline) enter rung 0, whose screen rejects 5;
    the scores of the 16 survivors (4 timed iterations each) are ranked and
    2/5 of the 15 non-baseline ones are promoted with the baseline (7);
    rung 1 (16 iterations) rejects 2 of them and promotes 2 of the remaining
    4 with the baseline (3); rung 2 (60 iterations) passes all 3.  Every
    rung's verdicts, scores and promotion decisions come from the library
    and are checked against the oracle; the survival table is Table A.1's
    MatVec row."""
    K = 21
    ref = torch.randn(65536, generator=torch.Generator(device=dev).manual_seed(5), device=dev)
    atol = rtol = 1e-5
    alive = list(range(K))
    entering, failed_n, promoted_n = [], [], []
    for rung, n_iter in enumerate(synth.RUNG_REPEATS):
        if rung == 0:
            fails = {3, 7, 11, 15, 19}
        elif rung == 1:
            fails = set([c for c in alive if c != 0][:2])
        else:
            fails = set()
        cands = [outputs_for(ref, fails, k) for k in alive]
        recs, summ = kb.screen(ref, cands, atol, rtol)
        orc = oracle_records(ref, cands, atol, rtol)
        verdict = [r["mismatches"] == 0 and r["status"] == 0 for r in recs]
        assert verdict == [o["mismatches"] == 0 for o in orc]
        assert [not v for v in verdict] == [k in fails for k in alive]
        # failed candidates are not timed: their rows are invalid
        t = synth.timing_samples(K, 3, n_iter, seed=rung).numpy()[alive]
        t[[not v for v in verdict]] = np.nan
        base = alive.index(0)
        rows, scores = kb.kb_rung_stats(torch.from_numpy(t).to(dev), base, rung,
                                        float(n_iter))
        g_rows, g_scores = kb.rung_records(rows, scores, len(alive), 3)
        o_rows, o_scores = oracle.rung_stats(t, base, rung, float(n_iter))
        assert [s["score"] for s in g_scores] == [s["score"] for s in o_scores]
        entering.append(len(alive))
        failed_n.append(sum(not v for v in verdict))
        if rung == len(synth.RUNG_REPEATS) - 1:
            promoted_n.append(sum(verdict))  # the finalists
            best = max(range(len(alive)), key=lambda i: (g_scores[i]["score"], -i))
            say("best", alive[best], g_scores[best])
            break
        rank, order, prom = kb.kb_rung_promote(scores, len(alive), base, 2, 5)
        o_rank, o_order, o_prom = oracle.rung_promote([s["score"] for s in o_scores],
                                                       [s["valid"] for s in o_scores], base, 2, 5)
        prom = prom.cpu().numpy()
        assert np.array_equal(prom, o_prom) and np.array_equal(rank.cpu().numpy(), o_rank)
        promoted_n.append(int(prom.sum()))
        alive = [alive[i] for i in range(len(alive)) if prom[i]]
    assert (entering, failed_n, promoted_n) == ([21, 7, 3], [5, 2, 0], [7, 3, 3])
    fail_pct, promo_pct = kb.kb_rung_survival(entering, failed_n, promoted_n, K)
    assert [round(x, 1) for x in fail_pct[:2]] == [23.8, 28.6]
    assert [round(x, 1) for x in promo_pct[:2]] == [33.3, 14.3]
