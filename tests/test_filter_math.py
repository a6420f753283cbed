"""The binary32 facts the position search's cheap filters rest on (CPU only).

The kernels only skip a chunk when a filter says no element of it can
qualify, so each filter must let through every element whose definition
holds.  These tests check the arithmetic behind that on random binary32 bit
patterns (every exponent, subnormals, zeros, infinities, NaNs), with numpy's
IEEE binary32 operations standing for the device's:

* mismatch: not (d <= tol) implies fl(d - tol) > 0 or NaN, and for finite d
  and tol the two are the same test; the NaN-propagating maximum over a
  lane's elements keeps that;
* max rel: an element whose quotient fl(d / a) is max_rel gives
  d - T a >= 0 for the threshold T the kernel takes for max_rel (a scaled
  max_rel when it is finite and at least 2^-100, 2^100 for +inf);
* a consistent record never has a max rel below 2^-100: a nonzero
  fl(|c - r|) / |r| of binary32 values is at least 2^-25.
"""
import numpy as np

N = 1 << 21


def random_f32(rng, n):
    """Binary32 values from uniformly drawn bit patterns, mixed with values
    near the ends of the range and exact specials."""
    x = rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32).view(np.float32)
    spec = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, np.finfo(np.float32).max,
                     np.finfo(np.float32).tiny, np.float32(2.0 ** -149)], np.float32)
    pick = rng.random(n) < 0.02
    x = x.copy()
    x[pick] = rng.choice(spec, size=int(pick.sum()))
    return x


def rel_threshold(max_rel):
    """The kernel's T for positive max_rel values (binary32 arithmetic)."""
    m = np.asarray(max_rel, np.float32)
    scaled = (m * np.float32(1.0 - 2.0 ** -20)).astype(np.float32)
    return np.where(np.isinf(m), np.float32(2.0 ** 100),
                    np.where(m < np.float32(2.0 ** -100), np.float32(0.0), scaled)).astype(np.float32)


def test_difference_sign_is_the_mismatch_order():
    rng = np.random.default_rng(11)
    with np.errstate(all="ignore"):
        d = np.abs(random_f32(rng, N))
        tol = random_f32(rng, N)
        # also pairs one ulp apart, both ways, and equal pairs
        k = N // 4
        tol[:k] = np.nextafter(d[:k], np.float32(np.inf))
        tol[k:2 * k] = np.nextafter(d[k:2 * k], np.float32(-np.inf))
        tol[2 * k:2 * k + k // 4] = d[2 * k:2 * k + k // 4]
        t = d - tol
    assert t.dtype == np.float32
    mismatch = ~(d <= tol)
    passes = (t > 0) | np.isnan(t)
    assert not np.any(mismatch & ~passes), "a mismatch the filter would skip"
    fin = np.isfinite(d) & np.isfinite(tol)
    assert np.array_equal((t > 0)[fin], (d > tol)[fin])


def test_lane_maximum_keeps_the_filter():
    """Eight elements per lane: the NaN-propagating maximum of fl(d - tol)
    is positive or NaN exactly when some element's is."""
    rng = np.random.default_rng(12)
    with np.errstate(all="ignore"):
        d = np.abs(random_f32(rng, N)).reshape(-1, 8)
        tol = random_f32(rng, N).reshape(-1, 8)
        t = d - tol
    m = np.maximum.reduce(t, axis=1)
    lane = ~(m <= 0)
    each = np.any((t > 0) | np.isnan(t), axis=1)
    assert np.array_equal(lane, each)


def exact_sign_d_minus_ta(d, T, a):
    """sign(d - T a) for binary32 d, T, a with a finite: T a is exact in
    binary64 (two 24-bit significands), and the binary64 difference keeps
    the sign of the exact one (it is zero only when that is zero)."""
    return np.sign(d.astype(np.float64) - T.astype(np.float64) * a.astype(np.float64))


def test_max_rel_threshold_passes_every_element_at_max_rel():
    rng = np.random.default_rng(13)
    with np.errstate(all="ignore"):
        d = np.abs(random_f32(rng, N))
        a = np.abs(random_f32(rng, N))
        ok = np.isfinite(a) & ~np.isnan(d)
        d, a = d[ok], a[ok]
        q = d / a
    pos = q > 0  # (q NaN: 0/0 and inf/inf, never a positive max_rel)
    d, a, q = d[pos], a[pos], q[pos]
    with np.errstate(over="ignore"):
        T = rel_threshold(q)
    s = exact_sign_d_minus_ta(d, T, a)
    assert np.all(s >= 0), (d[s < 0][:4], a[s < 0][:4], q[s < 0][:4])
    # every kind of max_rel was met: ordinary, +inf (a zero reference, an
    # overflow, an infinite difference) and the smallest quotients
    assert np.any(np.isinf(q) & (a == 0)) and np.any(np.isinf(q) & (a > 0)) and np.any(q < 2.0 ** -100)


def test_nonzero_relative_error_of_distinct_values_is_at_least_2_to_minus_25():
    rng = np.random.default_rng(14)
    with np.errstate(all="ignore"):
        r = random_f32(rng, N)
        c = r.copy()
        # neighbours and random partners of every exponent
        half = N // 2
        c[:half] = np.nextafter(r[:half], np.where(rng.random(half) < 0.5, np.float32(np.inf), np.float32(-np.inf)))
        c[half:] = random_f32(rng, N - half)
        d = np.abs(c - r)
        q = d / np.abs(r)
    ok = np.isfinite(q) & (q > 0)
    assert ok.sum() > N // 4
    assert q[ok].min() >= np.float32(2.0 ** -25)
