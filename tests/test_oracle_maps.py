"""Pins for the oracle's word -> float maps and storage conversions (CPU only).

uniform: u = (x >> 8) * 2^-24 over all 2^24 values; U(a, b) = fmaf(u, b - a, a)
  against exact rational arithmetic rounded once, plus range and monotonicity
  over every u.
normal: closed-form points of the Box-Muller transform (angle 0, pi/2, pi;
  radius at u1 = 1/2, 1 and 2^-32), the radius and angle identities on random
  word pairs, and distribution tests on 2^22 draws.
conversions: binary32 -> binary16 / bfloat16 over all 2^32 inputs against
  numpy's and torch's conversions; the widenings over all 2^16 inputs.
"""
import math
from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.exact import round_to_f32


def f32(x):
    return float(np.float32(x))


# ---------------------------------------------------------------- uniform ---

def test_u01_is_exact_top_24_bits():
    k = np.arange(1 << 24, dtype=np.uint32)
    low = np.random.default_rng(1).integers(0, 256, size=k.size, dtype=np.uint32)
    x = (k << np.uint32(8)) | low
    got = oracle.uniform_n(x, 0.0, 1.0)  # fmaf(u, 1, 0) == u
    assert np.array_equal(got, (k.astype(np.float64) * 2.0**-24).astype(np.float32))
    assert oracle.u01(0xFFFFFFFF) == 1.0 - 2.0**-24
    assert oracle.u01(0x000000FF) == 0.0


@pytest.mark.parametrize("a,b", [(-1e-6, 1e-6), (-1.0, 1.0), (0.0, 1.0), (2.5, 7.25),
                                 (-3.0e-38, 1.0e-38)])
def test_uniform_single_rounding_and_range(a, b):
    a32, b32 = f32(a), f32(b)
    width = f32(np.float32(b32) - np.float32(a32))
    k = np.arange(1 << 24, dtype=np.uint32)
    vals = oracle.uniform_n(k << np.uint32(8), a32, b32)
    # every value lies in [a, b] and is non-decreasing in u
    assert vals.min() >= np.float32(a32) and vals.max() <= np.float32(b32)
    assert np.all(np.diff(vals.astype(np.float64)) >= 0)
    # exact rational check of fmaf(u, fl(b - a), a) on a sample of u
    rng = np.random.default_rng(7)
    for kk in list(rng.integers(0, 1 << 24, size=300)) + [0, 1, (1 << 24) - 1, 1 << 23]:
        u = Fraction(int(kk), 1 << 24)
        want = round_to_f32(u * Fraction(width) + Fraction(a32))
        assert float(vals[int(kk)]) == want, (kk, float(vals[int(kk)]), want)


# ----------------------------------------------------------------- normal ---

def test_normal_closed_form_points():
    half = (1 << 31) - 1  # u1 = (x_a + 1) / 2^32 = 1/2
    rho_half = math.sqrt(2.0 * math.log(2.0))
    # angle 0: cosine branch is the radius, sine branch is exactly zero
    assert oracle.normal01(half, 0, 0) == f32(rho_half)
    assert oracle.normal01(half, 0, 1) == 0.0
    # angle pi/2 (x_b = 2^30): sine branch is the radius, cosine branch ~ 0
    assert oracle.normal01(half, 1 << 30, 1) == f32(rho_half)
    assert abs(oracle.normal01(half, 1 << 30, 0)) < 1e-15
    # angle pi (x_b = 2^31): cosine branch is minus the radius
    assert oracle.normal01(half, 1 << 31, 0) == f32(-rho_half)
    assert abs(oracle.normal01(half, 1 << 31, 1)) < 1e-15
    # x_a = 2^32 - 1: u1 = 1, radius 0
    for xb in (0, 12345, 1 << 31):
        assert oracle.normal01(0xFFFFFFFF, xb, 0) == 0.0
        assert oracle.normal01(0xFFFFFFFF, xb, 1) == 0.0
    # x_a = 0: u1 = 2^-32 (the +1 keeps the logarithm finite)
    assert oracle.normal01(0, 0, 0) == f32(math.sqrt(64.0 * math.log(2.0)))


def test_normal_radius_and_angle_identities():
    rng = np.random.default_rng(11)
    for _ in range(2000):
        xa, xb = (int(v) for v in rng.integers(0, 2**32, size=2))
        z0 = oracle.normal01(xa, xb, 0)
        z1 = oracle.normal01(xa, xb, 1)
        u1 = (xa + 1) / 2.0**32
        r2 = -2.0 * math.log(u1)
        # z0^2 + z1^2 is the squared radius, from x_a only
        assert abs(z0 * z0 + z1 * z1 - r2) <= 4e-7 * r2 + 1e-30
        # atan2(z1, z0) is the angle 2*pi*x_b/2^32, from x_b only
        if r2 > 1e-6:
            ang = math.atan2(z1, z0) % (2 * math.pi)
            want = 2 * math.pi * xb / 2.0**32
            diff = abs(ang - want)
            assert min(diff, 2 * math.pi - diff) < 1e-6 / math.sqrt(r2) + 1e-7


def test_gen_normal_pairs_words_per_half_block():
    seed, sid, sub = 5, 0x301, 2
    n = 16
    got = oracle.gen("f32", n, oracle.DIST_NORMAL, 0.0, 1.0, seed, sid, sub, 0)
    for g in range(n):
        w = oracle.stream_block(seed, sid, sub, g // 4)
        p = (g % 4) // 2
        assert got[g] == np.float32(oracle.normal01(w[2 * p], w[2 * p + 1], g % 2))


def test_gen_normal_distribution():
    from scipy import stats
    z = oracle.gen("f32", 1 << 22, oracle.DIST_NORMAL, 0.0, 1.0, seed=0, stream_id=9)
    z64 = z.astype(np.float64)
    assert abs(z64.mean()) < 2e-3
    assert abs(z64.var() - 1.0) < 3e-3
    ks = stats.kstest(z64[:1 << 20], "norm")
    assert ks.pvalue > 1e-4
    # mean / std arguments: fmaf(z, std, mean), one rounding
    y = oracle.gen("f32", 512, oracle.DIST_NORMAL, 3.0, 0.75, seed=0, stream_id=9)
    for zi, yi in zip(z[:512], y):
        assert float(yi) == round_to_f32(Fraction(float(zi)) * Fraction(0.75) + 3)


def test_gen_uniform_distribution():
    u = oracle.gen("f32", 1 << 20, oracle.DIST_UNIFORM, -1.0, 1.0, seed=0, stream_id=3)
    assert u.min() >= -1.0 and u.max() <= 1.0
    assert abs(float(u.astype(np.float64).mean())) < 3e-3
    assert abs(float(u.astype(np.float64).var()) - 1.0 / 3.0) < 3e-3


# ------------------------------------------------------------ conversions ---

def _chunks(total, size):
    return [(lo, min(total, lo + size)) for lo in range(0, total, size)]


def test_f32_to_f16_all_inputs():
    def check(bounds):
        lo, hi = bounds
        x = np.arange(lo, hi, dtype=np.uint64).astype(np.uint32).view(np.float32)
        got = oracle.f32_to_f16_n(x)
        with np.errstate(over="ignore", invalid="ignore"):
            want = x.astype(np.float16).view(np.uint16)
        nan = np.isnan(x)
        ok_finite = np.array_equal(got[~nan], want[~nan])
        # NaN: quiet NaN with the sign kept
        ok_nan = np.all((got[nan] & 0x7FFF) == 0x7E00) and np.array_equal(
            got[nan] >> 15, (x.view(np.uint32)[nan] >> 31).astype(np.uint16))
        return ok_finite and ok_nan
    with ThreadPoolExecutor(8) as ex:
        assert all(ex.map(check, _chunks(1 << 32, 1 << 24)))


def test_f32_to_bf16_all_inputs():
    import torch

    def check(bounds):
        lo, hi = bounds
        x = np.arange(lo, hi, dtype=np.uint64).astype(np.uint32).view(np.float32)
        got = oracle.f32_to_bf16_n(x)
        want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        nan = np.isnan(x)
        return (np.array_equal(got[~nan], want[~nan])
                and np.all((got[nan] & 0x7FFF) == 0x7FC0))
    with ThreadPoolExecutor(8) as ex:
        assert all(ex.map(check, _chunks(1 << 32, 1 << 24)))


def _conversion_sample():
    """About 3 M binary32 bit patterns: a prime stride over all of them, every
    pattern whose value rounds into or near the binary16 subnormals or near
    the binary16 overflow threshold (sampled with a small stride), the exact
    halfway cases of both narrowings under random upper bits, and NaNs whose
    payload sits only in the low bits."""
    rng = np.random.default_rng(2024)
    parts = [np.arange(0, 1 << 32, 2039, dtype=np.uint64)]
    for e_lo, e_hi in ((96, 114), (140, 144)):  # exponent fields: f16 subnormal targets, near 65520
        parts.append(np.arange(e_lo << 23, e_hi << 23, 61, dtype=np.uint64))
    hi = rng.integers(0, 1 << 19, 1 << 16, dtype=np.uint64)
    parts.append((hi << 13) | 0x1000)            # f16 halfway (13 dropped bits)
    parts.append(((hi << 16) & 0xFFFF0000) | 0x8000)  # bf16 halfway (16 dropped bits)
    parts.append(np.array([0x7F800001, 0xFF800001, 0x7F80FFFF, 0x7FC00000, 0x477FEFFF, 0x477FF000,
                           0x477FE000, 0x33000000, 0x33000001, 0x337FFFFF, 0x387FC000, 0x387FE000],
                          dtype=np.uint64))
    x = np.concatenate(parts) & 0xFFFFFFFF
    x = np.concatenate([x, x ^ (1 << 31)])  # both signs
    return x.astype(np.uint32).view(np.float32)


def test_conversions_sampled():
    """The two narrowings on a sample that reaches every branch of the
    definition (numpy's binary16 and torch's bfloat16 as references); the
    exhaustive tests below cover every input."""
    import torch
    x = _conversion_sample()
    nan = np.isnan(x)
    got = oracle.f32_to_f16_n(x)
    with np.errstate(over="ignore", invalid="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.all((got[nan] & 0x7FFF) == 0x7E00)
    got = oracle.f32_to_bf16_n(x)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.all((got[nan] & 0x7FFF) == 0x7FC0)


def test_widenings_all_inputs():
    import torch
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    f = oracle.f16_to_f32_n(h)
    want = h.view(np.float16).astype(np.float32)
    nan = np.isnan(want)
    assert np.array_equal(f[~nan].view(np.uint32), want[~nan].view(np.uint32))
    assert np.all(np.isnan(f[nan]))
    # NaN payloads move to the top of the binary32 significand unchanged
    assert np.array_equal(f[nan].view(np.uint32) & 0x7FFFFFFF,
                          0x7F800000 | ((h[nan].astype(np.uint32) & 0x3FF) << 13))
    b = oracle.bf16_to_f32_n(h)
    wantb = torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    nanb = np.isnan(wantb)
    assert np.array_equal(b[~nanb].view(np.uint32), wantb[~nanb].view(np.uint32))
    assert np.array_equal(b.view(np.uint32), h.astype(np.uint32) << 16)


def test_gen_16bit_rounds_the_binary32_value():
    for dt, conv in (("f16", oracle.f32_to_f16_n), ("bf16", oracle.f32_to_bf16_n)):
        v32 = oracle.gen("f32", 4096, oracle.DIST_NORMAL, 0.0, 64.0, seed=0, stream_id=4, sub=1)
        v16 = oracle.gen(dt, 4096, oracle.DIST_NORMAL, 0.0, 64.0, seed=0, stream_id=4, sub=1)
        assert np.array_equal(v16, conv(v32))
