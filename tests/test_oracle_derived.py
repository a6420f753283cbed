"""Pins of the oracle's derived seeded inputs (no GPU): Student-t values,
softmax rows, distinct index draws, planted changes and scatters
(oracle/kbo_derived.c).

Each function is held to something other than itself: closed forms, the
t(3) distribution in closed form, scipy's softmax, brute force on tiny
inputs, the raw word stream (pinned against rocRAND in test_oracle_philox),
the uniform and normal maps (pinned in test_oracle_maps), exact rational
arithmetic, and mask frequencies."""
import math
from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.exact import round_to_f32

SQRT3 = math.sqrt(3.0)
T3_5PCT = 3.182446305284263  # two-sided 5% point of Student's t with 3 degrees of freedom


def rho(xa):
    """Box-Muller radius of word xa: the cosine branch at angle 0 (pinned)."""
    return oracle.box_muller64(xa, 0)[0]


# ------------------------------------------------------------- Student-t ---

def test_student_t_equal_pairs_is_sqrt3():
    """Words (A, 0, A, 0): z0 = z2 = rho(A), z1 = z3 = 0, so t = rho / sqrt(rho^2 / 3) = sqrt(3)."""
    for A in (0, 1, 12345, 0x7FFFFFFF, 0xFFFFFFFE):
        t64 = oracle.student_t3((A, 0, A, 0), exact=True)
        assert abs(t64 - SQRT3) <= 4e-16 * SQRT3, (A, t64)
        assert oracle.student_t3((A, 0, A, 0)) == np.float32(SQRT3)


def test_student_t_ratio_of_radii():
    """Words (A, 0, B, 0): t = sqrt(3) rho(A) / rho(B): the numerator is the
    cosine branch of the first pair, the denominator the second pair's."""
    rng = np.random.default_rng(1)
    for A, B in rng.integers(0, 0xFFFFFFFF, size=(50, 2)):
        want = SQRT3 * rho(int(A)) / rho(int(B))
        got = oracle.student_t3((int(A), 0, int(B), 0), exact=True)
        assert abs(got - want) <= 1e-15 * abs(want), (A, B, got, want)


def test_student_t_quarter_and_half_turns():
    """Angle pi/2 in the first pair (xb = 2^30): z0 = rho cos(fl(pi/2)),
    z1 = rho (the sine branch enters the chi-square); with the second pair's
    radius 0 (xa = 2^32 - 1), t = sqrt(3) cos(fl(pi/2)) exactly up to
    rounding -- positive and tiny.  Angle pi (xb = 2^31): z0 = -rho, z1 ~ 0,
    so with equal radii t = -sqrt(3)."""
    c = math.cos(math.pi / 2)  # fl(pi/2) is below pi/2, so this is +6.12e-17
    for A in (0, 99, 0xABCDEF01):
        t = oracle.student_t3((A, 1 << 30, 0xFFFFFFFF, 77), exact=True)
        assert abs(t - SQRT3 * c) <= 1e-12 * SQRT3 * c, (A, t)
        t = oracle.student_t3((A, 1 << 31, A, 0), exact=True)
        assert abs(t + SQRT3) <= 1e-15, (A, t)
    # numerator radius 0: t = 0
    assert oracle.student_t3((0xFFFFFFFF, 5, 17, 3), exact=True) == 0.0


def test_student_t_second_pair_angle():
    """The second pair at angle pi/4 (xb = 2^29): z2 = z3 = rho(B) / sqrt(2),
    so z2^2 + z3^2 = rho(B)^2 and t = sqrt(3) rho(A) / rho(B) again."""
    for A, B in ((3, 5), (1000, 2 ** 31), (2 ** 32 - 7, 11)):
        want = SQRT3 * rho(A) / rho(B)
        got = oracle.student_t3((A, 0, B, 1 << 29), exact=True)
        assert abs(got - want) <= 1e-14 * abs(want), (A, B, got, want)


def t3_cdf(t):
    """Closed-form CDF of Student's t with 3 degrees of freedom."""
    x = t / SQRT3
    return 0.5 + (np.arctan(x) + x / (1.0 + x * x)) / np.pi


def _t3_samples(n, stream_id, threads=8):
    chunk = n // threads
    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(lambda i: oracle.gen("f32", chunk, oracle.DIST_STUDENT_T3, 0.0, 1.0, seed=0,
                                                 stream_id=stream_id, sub=0, offset=i * chunk),
                            range(threads)))
    return np.concatenate(parts)


def test_student_t_distribution():
    """2^24 draws of the seeded stream: the two-sided tail beyond 3.182446
    holds 5% (+-10 binomial standard deviations), the median is 0, and the
    empirical CDF stays within 3.3/sqrt(n) of the closed form everywhere on
    a grid (a Kolmogorov-Smirnov bound)."""
    n = 1 << 24
    t = _t3_samples(n, (5 << 8) | 0)
    assert np.isfinite(t).all()
    tail = np.mean(np.abs(t.astype(np.float64)) > T3_5PCT)
    assert abs(tail - 0.05) < 10 * math.sqrt(0.05 * 0.95 / n), tail
    assert abs(np.median(t)) < 2e-3
    ts = np.sort(t.astype(np.float64))
    grid = np.concatenate([np.linspace(-20, 20, 801), [-100.0, -50.0, 50.0, 100.0]])
    emp = np.searchsorted(ts, grid, side="right") / n
    ks = np.max(np.abs(emp - t3_cdf(grid)))
    assert ks < 3.3 / math.sqrt(n), ks


def test_student_t_location_scale_and_rounding():
    """kbo_gen's STUDENT_T3 element g is fmaf(t(block g), scale, location),
    then rounded to the storage type; block g is the whole block g."""
    g = np.arange(40, dtype=np.uint64)
    t = oracle.gen("f32", 40, oracle.DIST_STUDENT_T3, 0.0, 1.0, seed=9, stream_id=77, sub=3)
    for i in range(40):
        w = oracle.stream_block(9, 77, 3, int(g[i]))
        assert t[i] == oracle.student_t3(w)
    u = oracle.gen("f32", 40, oracle.DIST_STUDENT_T3, 1.5, 0.25, seed=9, stream_id=77, sub=3)
    exact = [round_to_f32(Fraction(float(x)) * Fraction(0.25) + Fraction(1.5)) for x in t]
    assert list(u) == [np.float32(e) for e in exact]
    h = oracle.gen("f16", 40, oracle.DIST_STUDENT_T3, 0.0, 1.0, seed=9, stream_id=77, sub=3, offset=0)
    assert np.array_equal(h, t.astype(np.float16).view(np.uint16))


# --------------------------------------------------------------- softmax ---

def test_softmax_against_scipy():
    """Rows of many lengths and scales against scipy's softmax in binary64,
    rounded to binary32: at most one unit in the last place apart (the two
    sum in different orders), and almost always identical."""
    from scipy.special import softmax
    rng = np.random.default_rng(2)
    same = total = 0
    for n in (1, 2, 3, 7, 64, 1000, 1024, 4097):
        for scale in (0.1, 2.0, 30.0, 400.0):
            x = (rng.standard_normal(n) * scale).astype(np.float32)
            got = oracle.softmax_row(x)
            want = softmax(x.astype(np.float64)).astype(np.float32)
            diff = np.abs(got.view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
            assert diff.max() <= 1, (n, scale)
            same += int((diff == 0).sum())
            total += n
    assert same >= 0.999 * total, (same, total)


def test_softmax_closed_forms():
    for n in (1, 2, 4, 1024):
        assert np.all(oracle.softmax_row(np.full(n, 3.25, np.float32)) == np.float32(1.0 / n))
    assert np.all(oracle.softmax_row(np.zeros(3, np.float32)) == np.float32(1.0 / 3.0))
    # a row dominated by one logit: the others underflow to 0 in binary32
    p = oracle.softmax_row(np.array([0.0, 200.0, 0.0], np.float32))
    assert list(p) == [0.0, 1.0, 0.0]
    # ln 3 against 0: 3/4 and 1/4 (exp(ln 3) is 3 within an ulp of binary64)
    p = oracle.softmax_row(np.array([0.0, math.log(3.0)], np.float32))
    assert abs(float(p[1]) - 0.75) <= 2 ** -24 and abs(float(p[0]) - 0.25) <= 2 ** -26


def test_softmax_shift_invariance():
    """Integer logits shifted by an integer (both exact in binary32): the
    same row, bit for bit."""
    rng = np.random.default_rng(3)
    for n in (5, 300):
        x = rng.integers(-20, 20, n).astype(np.float32)
        assert np.array_equal(oracle.softmax_row(x), oracle.softmax_row(x + np.float32(7)))


def test_softmax_rows_invariants():
    """The 256 x 1024 rows of logits 2z: every probability positive, and
    every row sums to 1 within 1024 units of 2^-24."""
    p = oracle.gen_softmax_rows(256, 1024, 2.0, seed=0, stream_id=(3 << 8) | 0, sub=0)
    assert p.shape == (256, 1024) and np.all(p > 0)
    assert np.max(np.abs(p.astype(np.float64).sum(axis=1) - 1.0)) <= 1024 * 2.0 ** -24
    # rows start at the right logits: row 7 from logits at offset 7 * 1024
    z = oracle.gen("f32", 1024, oracle.DIST_NORMAL, 0.0, 2.0, seed=0, stream_id=(3 << 8), sub=0, offset=7 * 1024)
    assert np.array_equal(p[7], oracle.softmax_row(z))
    q = oracle.gen_softmax_rows(2, 1024, 2.0, seed=0, stream_id=(3 << 8), sub=0, row0=6)
    assert np.array_equal(q, p[6:8])


# ---------------------------------------------------------- index draws ---

def test_indices_brute_force_tiny():
    """n = 5 and n = 3: the draws are ((w1 << 32) | w0) mod n of blocks
    0, 1, 2, ... with repeats skipped, written out by brute force."""
    for n, stream in ((5, 17), (3, 4), (7, 1 << 20)):
        want, j = [], 0
        while len(want) < n:
            w = oracle.stream_block(0, stream, 2, j)
            x = ((w[1] << 32) | w[0]) % n
            if x not in want:
                want.append(x)
            j += 1
        assert list(oracle.gen_indices(n, n, seed=0, stream_id=stream, sub=2)) == want
        assert list(oracle.gen_indices(2, n, seed=0, stream_id=stream, sub=2)) == want[:2]


def test_indices_word_stream_at_2_pow_32():
    """With n = 2^32 a draw is word 0 of block j, i.e. element 4j of the
    u32 stream (which rocRAND pins)."""
    m = 200
    words = oracle.gen("u32", 4 * m, oracle.DIST_U32, seed=3, stream_id=(4 << 8) | 3, sub=9)[::4]
    assert len(set(words.tolist())) == m
    assert np.array_equal(oracle.gen_indices(m, 1 << 32, seed=3, stream_id=(4 << 8) | 3, sub=9),
                          words.astype(np.uint64))


def test_indices_properties():
    for m, n in ((5, 65536), (64, 8 * 2048 * 4096), (1000, 1000), (1, 1)):
        idx = oracle.gen_indices(m, n, seed=0, stream_id=(1 << 8) | 3, sub=2)
        assert len(idx) == m and len(set(idx.tolist())) == m and int(idx.max()) < n
    with pytest.raises(ValueError):
        oracle.gen_indices(6, 5)
    with pytest.raises(ValueError):
        oracle.gen_indices(0, 0)


# ------------------------------------------------------- planted changes ---

def _f16_bits(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def _bf16_bits(x):
    import torch
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


WIDEN = {"f32": lambda s: s, "f16": lambda s: s.view(np.float16).astype(np.float32),
         "bf16": lambda s: (s.astype(np.uint32) << 16).view(np.float32)}
NARROW = {"f32": lambda x: np.asarray(x, np.float32), "f16": _f16_bits, "bf16": _bf16_bits}


def _src(dt, n, rng):
    x = (rng.standard_normal(n) * 4).astype(np.float32)
    return NARROW[dt](x)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_add_uniform(dt):
    """On zeros the change is the uniform stream itself; otherwise one
    binary32 addition (numpy), then the storage rounding."""
    n, a, b = 4099, -1e-3, 2e-3
    u = oracle.gen("f32", n, oracle.DIST_UNIFORM, a, b, seed=1, stream_id=11, sub=5, offset=13)
    zero = NARROW[dt](np.zeros(n, np.float32))
    got0 = oracle.perturb(zero, dt, oracle.PERTURB_ADD_UNIFORM, a, b, 0.0, seed=1, stream_id=11, sub=5, offset=13)
    assert np.array_equal(got0, NARROW[dt](u))
    src = _src(dt, n, np.random.default_rng(4))
    got = oracle.perturb(src, dt, oracle.PERTURB_ADD_UNIFORM, a, b, 0.0, seed=1, stream_id=11, sub=5, offset=13)
    assert np.array_equal(got, NARROW[dt](WIDEN[dt](src) + u))


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_rel_uniform_exact(dt):
    """fmaf(x, e, x): one rounding of the exact x e + x (exact rationals),
    then the storage rounding; on ones it is the binary32 sum 1 + e."""
    n, a, b = 1500, -2.0 ** -6, 2.0 ** -6
    e = oracle.gen("f32", n, oracle.DIST_UNIFORM, a, b, seed=2, stream_id=12, sub=0)
    ones = NARROW[dt](np.ones(n, np.float32))
    got1 = oracle.perturb(ones, dt, oracle.PERTURB_REL_UNIFORM, a, b, 0.0, seed=2, stream_id=12, sub=0)
    assert np.array_equal(got1, NARROW[dt](np.float32(1.0) + e))
    src = _src(dt, n, np.random.default_rng(5))
    x = WIDEN[dt](src)
    want = np.array([round_to_f32(Fraction(float(xi)) * Fraction(float(ei)) + Fraction(float(xi)))
                     for xi, ei in zip(x, e)], np.float32)
    got = oracle.perturb(src, dt, oracle.PERTURB_REL_UNIFORM, a, b, 0.0, seed=2, stream_id=12, sub=0)
    assert np.array_equal(got, NARROW[dt](want))


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_add_normal(dt):
    """On zeros the change is the NORMAL stream with mean 0 and standard
    deviation a; otherwise one binary32 addition of it."""
    n, s = 3001, 1e-4
    z = oracle.gen("f32", n, oracle.DIST_NORMAL, 0.0, s, seed=0, stream_id=(3 << 8) | 1, sub=7, offset=2)
    zero = NARROW[dt](np.zeros(n, np.float32))
    got0 = oracle.perturb(zero, dt, oracle.PERTURB_ADD_NORMAL, s, 0, 0, seed=0, stream_id=(3 << 8) | 1, sub=7, offset=2)
    assert np.array_equal(got0, NARROW[dt](z))
    src = _src(dt, n, np.random.default_rng(6))
    got = oracle.perturb(src, dt, oracle.PERTURB_ADD_NORMAL, s, 0, 0, seed=0, stream_id=(3 << 8) | 1, sub=7, offset=2)
    assert np.array_equal(got, NARROW[dt](WIDEN[dt](src) + z))


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_masked_changes(dt):
    """SCALE_WHERE and FLIP_LSB_WHERE: the mask is u < p with u the [0, 1)
    uniform stream; p = 0 copies, p = 1 changes everything, and p = 0.01
    changes a 1% share."""
    n = 1 << 16
    src = _src(dt, n, np.random.default_rng(7))
    u = oracle.gen("f32", n, oracle.DIST_UNIFORM, 0.0, 1.0, seed=0, stream_id=(1 << 8) | 2, sub=3)
    kw = dict(seed=0, stream_id=(1 << 8) | 2, sub=3)
    scaled = NARROW[dt](WIDEN[dt](src) * np.float32(1.01))
    ui = np.uint32 if dt == "f32" else np.uint16
    bits = lambda a: np.asarray(a).view(ui)
    flipped = (bits(src) ^ ui(1)).view(src.dtype)
    for op, changed in ((oracle.PERTURB_SCALE_WHERE, scaled), (oracle.PERTURB_FLIP_LSB_WHERE, flipped)):
        assert np.array_equal(bits(oracle.perturb(src, dt, op, 1.01, 0, 0.0, **kw)), bits(src))
        assert np.array_equal(bits(oracle.perturb(src, dt, op, 1.01, 0, 1.0, **kw)), bits(changed))
        got = oracle.perturb(src, dt, op, 1.01, 0, 0.01, **kw)
        mask = u < np.float32(0.01)
        assert np.array_equal(bits(got), np.where(mask, bits(changed), bits(src)))
        assert abs(mask.mean() - 0.01) < 10 * math.sqrt(0.01 * 0.99 / n)


def _classes(bits):
    mag = bits & 0x7FFFFFFF
    return {"zero": mag == 0, "sub": (mag > 0) & (mag < 0x00800000), "inf": mag == 0x7F800000}


def test_specials_degenerate_thresholds():
    """Thresholds (a, b, p) = (1, 1, 1): every element a subnormal with an
    odd mantissa; (0, 1, 1): signed zeros; (0, 0, 1): infinities; (0, 0, 0):
    a copy.  Signs are balanced."""
    n = 1 << 16
    src = np.random.default_rng(8).standard_normal(n).astype(np.float32)
    kw = dict(seed=0, stream_id=(5 << 8) | 2, sub=0)
    run = lambda a, b, p: oracle.perturb(src, "f32", oracle.PERTURB_SPECIALS, a, b, p, **kw).view(np.uint32)
    sub = run(1.0, 1.0, 1.0)
    assert _classes(sub)["sub"].all() and np.all(sub & 1 == 1)
    zero = run(0.0, 1.0, 1.0)
    assert _classes(zero)["zero"].all()
    inf = run(0.0, 0.0, 1.0)
    assert _classes(inf)["inf"].all()
    assert np.array_equal(run(0.0, 0.0, 0.0), src.view(np.uint32))
    for arr in (sub, zero, inf):
        neg = np.mean(arr >> 31)
        assert abs(neg - 0.5) < 10 * math.sqrt(0.25 / n), neg


def test_specials_frequencies_and_words():
    """The five-gigabyte reference's recipe on 2^22 elements: subnormals and
    zeros with probability 2^-10 each, infinities 2^-20, the rest kept; and
    every element as the stream's words say (u from word 0, the sign from
    the top bit of word 1, the mantissa from word 2), read through the
    pinned u32 and uniform streams."""
    n = 1 << 22
    a, b, p = 2.0 ** -10, 2.0 ** -9, 2.0 ** -9 + 2.0 ** -20
    src = np.random.default_rng(9).standard_normal(n).astype(np.float32)
    kw = dict(seed=0, stream_id=(5 << 8) | 2, sub=0)
    got = oracle.perturb(src, "f32", oracle.PERTURB_SPECIALS, a, b, p, **kw).view(np.uint32)
    c = _classes(got)
    for name, prob in (("sub", 2.0 ** -10), ("zero", 2.0 ** -10)):
        assert abs(c[name].mean() - prob) < 8 * math.sqrt(prob / n), name
    assert 0 < c["inf"].sum() < 20
    kept = ~(c["sub"] | c["zero"] | c["inf"])
    assert np.array_equal(got[kept], src.view(np.uint32)[kept])
    m = 1 << 16
    u = oracle.gen("f32", 4 * m, oracle.DIST_UNIFORM, 0.0, 1.0, **kw)[0::4]
    w = oracle.gen("u32", 4 * m, oracle.DIST_U32, **kw)
    sign = w[1::4] & np.uint32(0x80000000)
    want = np.where(u < np.float32(a), sign | (w[2::4] & np.uint32(0x7FFFFF)) | np.uint32(1),
                    np.where(u < np.float32(b), sign,
                             np.where(u < np.float32(p), sign | np.uint32(0x7F800000), src[:m].view(np.uint32))))
    assert np.array_equal(got[:m], want)


def test_zero_subnormal_rel():
    """p = 1 with a zero range: zeros change sign, subnormals become the zero
    of their sign, normal values, infinities and NaN stay; p = 0 copies; with
    p = 1/2 and a 1e-7 range, normal values become fmaf(x, d, x) with d the
    [a, b) value of word 1 (exact rationals), half of them or so."""
    vals = np.array([0.0, -0.0, 2.0 ** -149, -(2.0 ** -130), 1.5, -3e30, np.inf, -np.inf, np.nan], np.float32)
    src = np.resize(vals, 9 * 50)
    kw = dict(seed=0, stream_id=(5 << 8) | 1, sub=4)
    got = oracle.perturb(src, "f32", oracle.PERTURB_ZERO_SUBNORMAL_REL, 0.0, 0.0, 1.0, **kw).view(np.uint32)
    sb = src.view(np.uint32)
    mag = sb & 0x7FFFFFFF
    zero, sub = mag == 0, (mag > 0) & (mag < 0x00800000)
    assert np.array_equal(got[zero], sb[zero] ^ np.uint32(0x80000000))
    assert np.array_equal(got[sub], sb[sub] & np.uint32(0x80000000))
    assert np.array_equal(got[~(zero | sub)], sb[~(zero | sub)])
    assert np.array_equal(oracle.perturb(src, "f32", oracle.PERTURB_ZERO_SUBNORMAL_REL, -1e-7, 1e-7, 0.0,
                                         **kw).view(np.uint32), sb)
    n = 4000
    x = np.random.default_rng(10).standard_normal(n).astype(np.float32)
    got = oracle.perturb(x, "f32", oracle.PERTURB_ZERO_SUBNORMAL_REL, -1e-7, 1e-7, 0.5, **kw)
    u = oracle.gen("f32", 4 * n, oracle.DIST_UNIFORM, 0.0, 1.0, **kw)[0::4]
    d = oracle.gen("f32", 4 * n, oracle.DIST_UNIFORM, -1e-7, 1e-7, **kw)[1::4]
    hit = u < np.float32(0.5)
    want = np.array([round_to_f32(Fraction(float(xi)) * Fraction(float(di)) + Fraction(float(xi)))
                     for xi, di in zip(x, d)], np.float32)
    assert np.array_equal(got[hit], want[hit]) and np.array_equal(got[~hit], x[~hit])
    assert abs(hit.mean() - 0.5) < 0.05


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_nan_results_are_canonical(dt):
    """A NaN that the arithmetic creates (inf * e + inf with e < 0) or passes
    on (a NaN input) is stored as the dtype's positive quiet NaN; a masked-out
    NaN is copied bit for bit."""
    qnan = {"f32": 0x7FC00000, "f16": 0x7E00, "bf16": 0x7FC0}[dt]
    ui = np.uint32 if dt == "f32" else np.uint16
    neg_nan = {"f32": 0xFFC00001, "f16": 0xFE01, "bf16": 0xFFC1}[dt]
    src = NARROW[dt](np.full(64, np.inf, np.float32))
    got = oracle.perturb(src, dt, oracle.PERTURB_REL_UNIFORM, -0.5, -0.25, 0.0, seed=0, stream_id=1)
    assert np.all(got.view(ui) == qnan)
    src = np.full(64, neg_nan, ui)
    if dt == "f32":
        src = src.view(np.float32)
    got = oracle.perturb(src, dt, oracle.PERTURB_ADD_UNIFORM, 0.0, 1.0, 0.0, seed=0, stream_id=1)
    assert np.all(got.view(ui) == qnan)
    got = oracle.perturb(src, dt, oracle.PERTURB_SCALE_WHERE, 2.0, 0.0, 0.0, seed=0, stream_id=1)
    assert np.all(got.view(ui) == neg_nan)


def test_perturb_refuses_undefined_pairs():
    with pytest.raises(ValueError):
        oracle.perturb(np.zeros(4, np.uint16), "f16", oracle.PERTURB_SPECIALS)
    with pytest.raises(ValueError):
        oracle.perturb(np.zeros(4, np.float32), "f32", 9)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_scatter(dt):
    ref = NARROW[dt](np.array([1.0, -2.0, 0.0, -0.0, 5.0], np.float32))
    dst = ref.copy()
    oracle.scatter(dst, ref, dt, [1, 3, 99], oracle.SCATTER_INF_SIGN_OF_REF)
    w = WIDEN[dt](dst)
    assert w[1] == -np.inf and w[3] == -np.inf and np.array_equal(dst[[0, 2, 4]], ref[[0, 2, 4]])
    oracle.scatter(dst, ref, dt, [0, 4], oracle.SCATTER_NAN)
    qnan = {"f32": 0x7FC00000, "f16": 0x7E00, "bf16": 0x7FC0}[dt]
    assert int(dst[0].view(np.uint32 if dt == "f32" else np.uint16)) == qnan and np.isnan(WIDEN[dt](dst)[4])
