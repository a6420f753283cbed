"""The fail-fast screening mode (KB_FAIL_FAST) against the oracle (GPU).

What the mode fixes, and what is checked here:
  * a candidate without mismatch is read in full: its counts, flags and
    maxima are the same as without the flag and its sums agree within 1e-6
    (the fail-fast launch splits the work differently, so the binary64 sums
    may round differently), and the record equals the oracle's;
  * a candidate with a mismatch keeps its verdict (mismatches >= 1) and its
    record describes the elements that were compared, numel being their
    count: every count and maximum is at most the oracle's over the whole
    tensor, and the sums are at most the whole sums;
  * when every element mismatches, the compared elements are whole chunks,
    and on a reference that repeats every chunk the record must equal the
    oracle's over as many elements;
  * a single planted mismatch is always counted, exactly once;
  * the failed words the mode keeps in the workspace never leak into a later
    call on the same workspace.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
from tests.helpers import (assert_records_match, check_partial, ensure_built, oracle_records, oracle_workload,
                           same_record, storage)

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
CONV = {"f32": lambda x: x.astype(np.float32), "f16": oracle.f32_to_f16_n, "bf16": oracle.f32_to_bf16_n}
FF = kb.KB_FAIL_FAST
ATOL = RTOL = 1e-2


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(arr, dt, dev):
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(dev)
    bits = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).to(dev)
    return bits.view(TORCH_DT[dt])


def same_bits(a, b):
    """Two records with every field the same (NaN equal to NaN)."""
    for f in a:
        x, y = a[f], b[f]
        if x != y and not (isinstance(x, float) and x != x and y != y):
            return False
    return True


def make_case(dt, n, seed):
    """A reference and six candidates: three that pass (copy, in-tolerance
    noise, a copy with a -0 for +0 swap), three that fail (first element,
    last element, every element)."""
    rng = np.random.default_rng(seed)
    r32 = rng.uniform(0.5, 2.0, n).astype(np.float32)
    r32[:: 97] = 0.0
    noise = (r32 * rng.uniform(-2e-3, 2e-3, n)).astype(np.float32)
    cands = [r32.copy(), r32 + noise, r32.copy(), r32.copy(), r32.copy(), r32 + np.float32(1.0)]
    cands[2][r32 == 0.0] = -0.0
    cands[3][0] = r32[0] + 3.0
    cands[4][n - 1] = r32[n - 1] - 3.0
    return r32, cands


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n", [1, 511, 4097, 70001, (1 << 20) + 37])
def test_mixed_candidates(dev, dt, n):
    say("fail-fast mixed", dt, n)
    r32, cands = make_case(dt, n, n + 5)
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    full, fsum = kb.screen(ref, cd, ATOL, RTOL, 0)
    fast, ssum = kb.screen(ref, cd, ATOL, RTOL, FF)
    orc = oracle_records(ref, cd, ATOL, RTOL, 0)
    assert_records_match(full, orc, "full %s n=%d" % (dt, n))
    assert ssum == fsum, (ssum, fsum)
    for k, (g, f, o) in enumerate(zip(fast, full, orc)):
        label = "%s n=%d cand %d" % (dt, n, k)
        if o["mismatches"] == 0:
            assert same_record(g, f), (label, g, f)
        else:
            check_partial(g, o, label)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("n", [4 * 512, 70001, (1 << 22) + 300])
@pytest.mark.parametrize("k", [1, 5])
def test_all_mismatch_whole_chunks(dev, dt, n, k):
    """Every element mismatches: a wave stops after its first chunk, and a
    work-group that starts once the failure is known reads nothing, so the
    compared elements are whole chunks (which ones depends on timing).  With
    a reference that repeats every 512 elements every chunk has the same
    statistics, so the record must equal the oracle's over any numel
    elements made of whole chunks: the first ones, say."""
    say("fail-fast whole chunks", dt, n, k)
    rng = np.random.default_rng(k * 1000 + n % 997)
    period = rng.standard_normal(512).astype(np.float32)
    r32 = np.resize(period, n)
    bad = (r32 + np.float32(4.0)).astype(np.float32)
    cands = [r32.copy() for _ in range(k)]
    cands[k // 2] = bad
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    fast, _ = kb.screen(ref, cd, ATOL, RTOL, FF)
    g = fast[k // 2]
    m = g["numel"]
    assert m % 512 == 0 and 0 < m <= (n // 512) * 512, g
    assert g["mismatches"] == m, g
    if n >= (1 << 22):
        assert m < n // 2, ("no early stop", g)
    o = oracle.screen(storage(ref)[:m], storage(cd[k // 2])[:m], dt, ATOL, RTOL, 0)
    assert_records_match([g], [o], "whole chunks %s n=%d k=%d" % (dt, n, k))
    for j, c in enumerate(fast):
        if j != k // 2:
            assert c["numel"] == n and c["mismatches"] == 0 and c["bitwise_equal"] == 1, (j, c)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n", [600, 70001, (1 << 21) + 17])
def test_single_mismatch_counted_once(dev, dt, n):
    """Only a mismatch sets a failed word, so the wave that holds the one
    mismatching element reaches it and counts it."""
    say("fail-fast single", dt, n)
    rng = np.random.default_rng(n)
    r32 = rng.uniform(1.0, 2.0, n).astype(np.float32)
    cands = []
    for p in (0, n // 3, n - 1):
        c = r32.copy()
        c[p] = 100.0
        cands.append(c)
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    fast, summ = kb.screen(ref, cd, ATOL, RTOL, FF)
    orc = oracle_records(ref, cd, ATOL, RTOL, 0)
    assert summ["n_failed"] == 3 and summ["n_passed"] == 0, summ
    for k, (g, o) in enumerate(zip(fast, orc)):
        assert g["mismatches"] == 1 == o["mismatches"], (k, g)
        check_partial(g, o, "%s n=%d single %d" % (dt, n, k))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_sparse_random_failures(dev, dt):
    """Failures scattered at random, with NaN and infinities among them, in
    long candidate lists (several groups, two-level finish)."""
    n = (1 << 20) + 333
    rng = np.random.default_rng(4242)
    r32 = rng.standard_normal(n).astype(np.float32)
    cands = []
    for k in range(19):
        c = (r32 + r32 * rng.uniform(-1e-3, 1e-3, n)).astype(np.float32)
        if k % 3:
            idx = rng.choice(n, size=1 + k * 7, replace=False)
            c[idx] += rng.uniform(0.5, 5.0, idx.size).astype(np.float32)
            if k % 5 == 1:
                c[idx[: 3]] = [np.nan, np.inf, -np.inf][: min(3, idx.size)]
        cands.append(c)
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    for flags in (0, kb.KB_EQUAL_NAN):
        say("fail-fast sparse", dt, flags)
        full, fsum = kb.screen(ref, cd, ATOL, RTOL, flags)
        fast, ssum = kb.screen(ref, cd, ATOL, RTOL, flags | FF)
        orc = oracle_records(ref, cd, ATOL, RTOL, flags)
        assert_records_match(full, orc, "full sparse %s" % dt)
        assert ssum == fsum
        for k, (g, f, o) in enumerate(zip(fast, full, orc)):
            if o["mismatches"] == 0:
                assert same_record(g, f), (k, g, f)
            else:
                check_partial(g, o, "sparse %s cand %d" % (dt, k))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_one_group_many_super_groups(dev, dt):
    """Four candidates over millions of elements: one group, screened in one
    round that spans every resident work-group, so the finish's second level
    combines more than 48 super-groups, with the per-candidate read counts
    and reference sums of the mode.  Three candidates pass (their records are
    whole), one fails in its last element."""
    n = 12 * (1 << 20) + 333
    rng = np.random.default_rng(77)
    r32 = rng.standard_normal(n).astype(np.float32)
    cands = [(r32 + r32 * rng.uniform(-2e-3, 2e-3, n)).astype(np.float32) for _ in range(3)]
    bad = r32.copy()
    bad[n - 1] += np.float32(9.0)
    cands.insert(2, bad)
    plan = kb.kb_screen_launch(4, n, {"f32": kb.KB_F32, "bf16": kb.KB_BF16}[dt])
    say("fail-fast one group", dt, plan)
    assert plan["n_groups"] == 1 and (plan["blocks_per_group"] + 15) // 16 > 48, plan
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    full, fsum = kb.screen(ref, cd, ATOL, RTOL, 0)
    fast, ssum = kb.screen(ref, cd, ATOL, RTOL, FF)
    orc = oracle_records(ref, cd, ATOL, RTOL, 0)
    assert_records_match(full, orc, "full one group %s" % dt)
    assert ssum == fsum and fsum["n_failed"] == 1, (ssum, fsum)
    for k, (g, f, o) in enumerate(zip(fast, full, orc)):
        if o["mismatches"] == 0:
            assert same_record(g, f), (k, g, f)
        else:
            check_partial(g, o, "one group %s cand %d" % (dt, k))


def test_workload_c2_full_size(dev):
    """The fail-fast screen bench.py times: the 16-candidate 4096 x 4096
    bf16 workload at its full size."""
    w, _ = oracle_workload("c2", dev, seed=0)
    torch.cuda.synchronize()
    say("fail-fast c2 full size")
    full, fsum = kb.screen(w.ref, w.cands, w.atol, w.rtol, 0)
    fast, ssum = kb.screen(w.ref, w.cands, w.atol, w.rtol, FF)
    orc = oracle_records(w.ref, w.cands, w.atol, w.rtol, 0)
    assert_records_match(full, orc, "c2 full")
    assert ssum == fsum and fsum["n_failed"] > 0 and fsum["n_passed"] > 0, (ssum, fsum)
    for k, (g, f, o) in enumerate(zip(fast, full, orc)):
        if o["mismatches"] == 0:
            assert same_record(g, f), (k, g, f)
        else:
            check_partial(g, o, "c2 full cand %d" % k)
    del w
    torch.cuda.empty_cache()


def test_wide_range_sums_of_passing_candidates(dev):
    """Passing candidates on heavy-tailed fp32 data whose binary64 sums are
    not exact (so their bits depend on the summation order), over 2^22+
    elements and three candidate groups: the fail-fast launch uses another
    stripe count than the plain one, and the records must still agree --
    counts, flags and maxima exactly, sums within 1e-6 -- and both must
    equal the oracle's."""
    n = (1 << 22) + 1029
    rng = np.random.default_rng(515)
    # Student-t-like magnitudes over many binades, with in-tolerance noise
    r32 = (rng.standard_normal(n) / np.sqrt(rng.chisquare(3, n) / 3)).astype(np.float32)
    r32 *= np.float32(2.0) ** rng.integers(-20, 20, n).astype(np.float32)
    K = 11
    cands = [(r32 + r32 * rng.uniform(-5e-7, 5e-7, n)).astype(np.float32) for _ in range(K - 1)]
    bad = r32.copy()
    bad[n // 2] = np.float32(7.0) * r32[n // 2] + np.float32(1.0)
    cands.insert(4, bad)
    ref = to_dev(r32, "f32", dev)
    cd = [to_dev(c, "f32", dev) for c in cands]
    plain = kb.kb_screen_launch(K, n, kb.KB_F32)
    say("fail-fast wide-range sums", plain)
    assert plain["n_groups"] >= 3, plain
    full, fsum = kb.screen(ref, cd, 1e-8, 1e-6, 0)
    fast, ssum = kb.screen(ref, cd, 1e-8, 1e-6, FF)
    orc = oracle_records(ref, cd, 1e-8, 1e-6, 0)
    assert_records_match(full, orc, "wide-range full")
    assert ssum == fsum and fsum["n_failed"] == 1, (ssum, fsum)
    inexact = 0
    for k, (g, f, o) in enumerate(zip(fast, full, orc)):
        if o["mismatches"] == 0:
            assert same_record(g, f), (k, g, f)
            assert_records_match([g], [o], "wide-range fail-fast cand %d" % k)
            inexact += g["sum_sq_ref"] != f["sum_sq_ref"] or g["sum_sq_diff"] != f["sum_sq_diff"]
        else:
            check_partial(g, o, "wide-range cand %d" % k)
    say("passing candidates whose sums differ in the last bits:", inexact)


def test_workspace_left_clean(dev):
    """Fail, then pass, on one workspace and one record buffer: the second
    call must read the (now passing) candidates in full."""
    dt, n = "f32", (1 << 20) + 5
    rng = np.random.default_rng(9)
    r32 = rng.standard_normal(n).astype(np.float32)
    ref = to_dev(r32, dt, dev)
    good = [to_dev(r32, dt, dev) for _ in range(6)]
    bad = [to_dev(r32 + np.float32(1.0), dt, dev) for _ in range(6)]
    d_stats, ws = kb.kb_screen(ref, bad, ATOL, RTOL, FF)
    first, s1 = kb.kb_screen_stats(d_stats, 6)
    assert s1["n_failed"] == 6
    for flags in (FF, 0, FF):
        kb.kb_screen(ref, good, ATOL, RTOL, flags, workspace=ws, d_stats=d_stats)
        recs, summ = kb.kb_screen_stats(d_stats, 6)
        assert summ["n_passed"] == 6, (flags, summ)
        for g in recs:
            assert g["numel"] == n and g["mismatches"] == 0 and g["bitwise_equal"] == 1, g
    # after fail-fast calls that stopped candidates, the next plain call is exact
    kb.kb_screen(ref, bad, ATOL, RTOL, FF, workspace=ws, d_stats=d_stats)
    kb.kb_screen(ref, bad, ATOL, RTOL, 0, workspace=ws, d_stats=d_stats)
    recs, _ = kb.kb_screen_stats(d_stats, 6)
    for g in recs:
        assert g["numel"] == n and g["mismatches"] == n, g


def test_rejected_and_empty(dev):
    """The policy gate and empty tensors behave as without the flag."""
    ref = torch.zeros(1000, dtype=torch.float32, device=dev)
    cands = [ref.clone(), None, torch.zeros(999, dtype=torch.float32, device=dev),
             torch.ones(1000, dtype=torch.float32, device=dev)]
    a, sa = kb.screen(ref, cands, ATOL, RTOL, 0)
    b, sb = kb.screen(ref, cands, ATOL, RTOL, FF)
    for k in (0, 1, 2):
        assert same_bits(a[k], b[k]), (k, a[k], b[k])
    assert b[3]["mismatches"] >= 1 and sa == sb
    e = torch.zeros(0, dtype=torch.float32, device=dev)
    a, _ = kb.screen(e, [e.clone()], ATOL, RTOL, 0)
    b, _ = kb.screen(e, [e.clone()], ATOL, RTOL, FF)
    assert same_bits(a[0], b[0])
