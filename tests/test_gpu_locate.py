"""Parity of the position search with the oracle (GPU), in both forms: the
separate pass (kb_screen, then kb_screen_locate) and the positions found in
the screening pass itself (kb_screen_ex with opts.d_loc).

The oracle's kbo_locate runs on host copies of the same bytes with the
oracle's own maxima (equal to the library's by the screening parity).  Every
position must be equal, and the records of the screening pass with
positions must match the oracle's like those of the plain pass."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
import synth
from tests.helpers import (assert_records_match, dtype_name, ensure_built, oracle_records, oracle_workload,
                           storage)

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
CONV = {"f32": lambda x: x.astype(np.float32), "f16": oracle.f32_to_f16_n, "bf16": oracle.f32_to_bf16_n}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def to_dev(arr, dt, dev):
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(dev)
    bits = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).to(dev)
    return bits.view(TORCH_DT[dt])


def oracle_positions(ref, cands, atol, rtol, flags=0, records=None):
    """The oracle's positions of every candidate (and its records, appended
    to `records` when given)."""
    dt = dtype_name(ref)
    r = storage(ref)
    out = []
    for c in cands:
        cs = storage(c)
        s = oracle.screen(r, cs, dt, atol, rtol, flags)
        if records is not None:
            records.append(s)
        fm, ai, ri = oracle.locate(r, cs, dt, atol, rtol, s["max_abs_err"], s["max_rel_err"], flags)
        out.append({"first_mismatch": fm, "max_abs_index": ai, "max_rel_index": ri})
    return out


def say(*a):
    print(*a, flush=True)


def check(ref, cands, atol, rtol, flags=0, label="", want=None):
    """Both forms against the oracle's positions (computed here unless given)."""
    say("positions", label, len(cands), tuple(ref.shape), ref.dtype)
    recs, locs = kb.locate(ref, cands, atol, rtol, flags)
    frecs, flocs = kb.screen_positions(ref, cands, atol, rtol, flags)
    orecs = []
    if want is None:
        want = oracle_positions(ref, cands, atol, rtol, flags, orecs)
    for k, (g, f, w) in enumerate(zip(locs, flocs, want)):
        assert g == w, (label, "separate pass", k, g, w)
        assert f == w, (label, "screening pass", k, f, w)
    # the records of the pass with positions: the oracle's, to the same bar as
    # the plain pass, and every exact field equal to the plain pass's
    if orecs:
        assert_records_match(frecs, orecs, label + " (records with positions)")
    for a, b in zip(frecs, recs):
        assert {f: a[f] for f in a if f not in ("sum_sq_diff", "sum_sq_ref", "rel_l2")} == \
            {f: b[f] for f in b if f not in ("sum_sq_diff", "sum_sq_ref", "rel_l2")}, (label, a, b)
    return flocs


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n", [1, 511, 512, 4097, 70001, 1 << 20])
def test_planted_positions(dev, dt, n):
    rng = np.random.default_rng(n)
    r32 = rng.uniform(1.0, 2.0, n).astype(np.float32)
    cands = [r32.copy() for _ in range(5)]
    # 1: one mismatch late (in the ragged tail when there is one)
    cands[1][n - 1] = 7.0
    # 2: mismatches at several places, the lowest one chosen
    for p in sorted({n // 2, n // 3, (2 * n) // 3}):
        cands[2][p] = 5.0
    # 3: tie of the largest difference and ratio
    for p in sorted({n - 1, n // 5, n // 7}):
        cands[3][p] = r32[p] + 0.5
    # 4: NaN first, then the maximum
    cands[4][n // 9] = np.nan
    cands[4][n - 1 - n // 11] = r32[n - 1 - n // 11] + 0.25
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    check(ref, cd, 1e-3, 1e-3, 0, "%s n=%d" % (dt, n))


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_random_ragged(dev, dt):
    rng = np.random.default_rng(17)
    n = 3 * 512 * 37 + 211
    r32 = rng.standard_normal(n).astype(np.float32)
    r32[rng.integers(0, n, 40)] = 0.0
    cands = []
    for k in range(9):
        c = (r32 + rng.standard_normal(n).astype(np.float32) * (10.0 ** (-5 + k / 2))).astype(np.float32)
        if k % 3 == 0:
            c[rng.integers(0, n, 3)] = np.inf
        cands.append(c)
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    check(ref, cd, 1e-3, 1e-3, 0, dt)
    check(ref, cd, 1e-3, 1e-3, kb.KB_EQUAL_NAN, dt + " equal_nan")


@pytest.mark.parametrize("name,scale,K", [("c1", 1.0, 4), ("c2", 1 / 64, 16), ("c3", 1 / 8, 64),
                                          ("c4", 1 / 256, 16), ("c4", 1 / 256, 40), ("c5", 1 / 512, 8)])
def test_workloads(dev, name, scale, K):
    w, _ = oracle_workload(name, dev, seed=0, scale=scale, K=K)
    check(w.ref, w.cands, w.atol, w.rtol, 0, name)


def test_max_rel_filter_near_misses(dev):
    """The max-rel search filters with d - T a >= 0, T just below max_rel,
    and confirms by division.  Here every chunk but the last full one holds
    a near miss (ratio 0.5 - 2^-23, which passes the filter but is not the
    maximum 0.5), so every wave meets one in its first chunk and must go on
    to the one element whose ratio is 0.5, in the last full chunk.  binary32
    only: the ratios of two 16-bit values cannot come that close to 0.5
    without equalling it."""
    n_chunks = 200
    n = 512 * n_chunks + 77
    rng = np.random.default_rng(31)
    r32 = np.ones(n, np.float32)
    c32 = r32.copy()
    near = np.arange(n_chunks - 1) * 512 + rng.integers(0, 512, n_chunks - 1)
    c32[near] = np.float32(1.5) - np.float32(2.0 ** -23)
    hit = (n_chunks - 1) * 512 + 300
    c32[hit] = 1.5
    ref = to_dev(r32, "f32", dev)
    cand = to_dev(c32, "f32", dev)
    locs = check(ref, [cand], 1.0, 0.0, 0, "near misses")
    assert locs[0] == {"first_mismatch": -1, "max_abs_index": hit, "max_rel_index": hit}, locs


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_maxima_tied_in_every_chunk(dev, dt):
    """One element per chunk (at a drawn slot) with the same abs and rel
    error, so every wave meets the maximum in its first chunk and the waves
    of a work-group share it at once: the wave holding the smallest index
    must still record it (in the screening pass the shared value filters the
    other elements)."""
    n_chunks = 300
    n = 512 * n_chunks + 33
    rng = np.random.default_rng(23)
    r32 = np.ones(n, np.float32)
    c32 = r32.copy()
    hits = np.arange(n_chunks) * 512 + rng.integers(0, 512, n_chunks)
    c32[hits] = 1.5
    # a larger abs error, but a smaller rel one, late in the array
    r32[n - 700] = 4.0
    c32[n - 700] = 5.0
    ref = to_dev(CONV[dt](r32), dt, dev)
    cand = to_dev(CONV[dt](c32), dt, dev)
    locs = check(ref, [cand, ref.clone()], 1e-3, 1e-3, 0, "%s ties" % dt)
    assert locs[0] == {"first_mismatch": int(hits[0]), "max_abs_index": n - 700,
                       "max_rel_index": int(hits[0])}, locs


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_non_finite_references(dev, dt):
    """References with +-inf and NaN scattered through many chunks.  The
    cheap pass sends every such element to the exact pass, which applies the
    definition (a non-finite reference matches only an equal candidate, or a
    NaN one under KB_EQUAL_NAN)."""
    n = 512 * 40 + 5
    rng = np.random.default_rng(41)
    r32 = rng.uniform(-2.0, 2.0, n).astype(np.float32)
    special = rng.choice(n, size=n // 30, replace=False)
    r32[special] = rng.choice(np.array([np.inf, -np.inf, np.nan], np.float32), size=special.size)
    cands = [r32.copy() for _ in range(5)]
    # 1: an infinity of the reference replaced by a finite value, late
    late_inf = [i for i in special if np.isinf(r32[i]) and i > n // 2]
    cands[1][late_inf[0]] = 1.0
    # 2: in-tolerance noise on the finite elements only
    fin = np.isfinite(r32)
    cands[2][fin] = r32[fin] * (1 + rng.uniform(-1e-4, 1e-4, int(fin.sum()))).astype(np.float32)
    # 3: an infinity of the opposite sign
    cands[3][late_inf[-1]] = -r32[late_inf[-1]]
    # 4: every NaN of the reference replaced by 0
    cands[4][np.isnan(r32)] = 0.0
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    for flags in (0, kb.KB_EQUAL_NAN):
        check(ref, cd, 1e-2, 1e-2, flags, "%s non-finite flags=%d" % (dt, flags))


def test_workload_c2_full_size(dev):
    """The 16-candidate 4096 x 4096 bf16 workload at its full size, the
    position search bench.py times."""
    w, _ = oracle_workload("c2", dev, seed=0)
    torch.cuda.synchronize()
    locs = check(w.ref, w.cands, w.atol, w.rtol, 0, "c2 full")
    assert sum(l["first_mismatch"] >= 0 for l in locs) > 0 and all(l["max_abs_index"] >= 0 for l in locs)
    del w
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
def test_indices_beyond_32_bits(dev, dt):
    """2^32 + 777 elements (8.6 GB per 16-bit tensor, 17.2 GB per fp32 one,
    byte offsets past 2^34): element indices and counts past 32 bits in the
    screen and the position search.  The candidate is the reference except
    at three planted elements, so the expected record and positions follow
    from the construction (the oracle would take minutes over 4 G elements):
    a difference of 4 below 2^32, and a tie of the largest difference 8
    (relative error 8) at 2^32 + 5, in the last whole chunk, and in the
    ragged tail."""
    n = (1 << 32) + 777
    ref = torch.empty(n, dtype=TORCH_DT[dt], device=dev)
    kb.kb_gen_inputs(ref, kb.KB_DIST_NORMAL, 0.0, 1.0, seed=5, stream_id=0x3232)
    cand = ref.clone()
    low, high, tail = 3 << 30, (1 << 32) + 5, n - 3
    assert high < (n // 512) * 512 <= tail
    for i, c in ((low, 5.0), (high, 9.0), (tail, 9.0)):
        ref[i] = 1.0
        cand[i] = c
    torch.cuda.synchronize()
    say("indices beyond 32 bits", dt)
    recs, locs = kb.locate(ref, [cand], 1e-2, 1e-2)
    r = recs[0]
    assert r["numel"] == n and r["mismatches"] == 3 and r["nan_count"] == 0, r
    assert r["max_abs_err"] == 8.0 and r["max_rel_err"] == 8.0 and r["bitwise_equal"] == 0, r
    assert r["sum_sq_diff"] == 16.0 + 64.0 + 64.0, r
    assert 0.99 * n < r["sum_sq_ref"] < 1.01 * n, r
    assert locs[0] == {"first_mismatch": low, "max_abs_index": high, "max_rel_index": high}, locs
    say("indices beyond 32 bits, positions in the screening pass")
    frecs, flocs = kb.screen_positions(ref, [cand], 1e-2, 1e-2)
    assert flocs == locs, (flocs, locs)
    assert {f: v for f, v in frecs[0].items() if f != "sum_sq_ref"} == \
        {f: v for f, v in r.items() if f != "sum_sq_ref"}, (frecs[0], r)
    # fail-fast: a passing copy is read in full (its element count, summed
    # over work-groups, is past 2^32) and its record is the plain one
    same = ref.clone()
    full, _ = kb.screen(ref, [cand, same], 1e-2, 1e-2, 0)
    fast, summ = kb.screen(ref, [cand, same], 1e-2, 1e-2, kb.KB_FAIL_FAST)
    assert summ["n_failed"] == 1 and summ["n_passed"] == 1, summ
    assert fast[1] == full[1] and full[1]["numel"] == n and full[1]["bitwise_equal"] == 1, (fast[1], full[1])
    assert 1 <= fast[0]["mismatches"] <= 3 and fast[0]["numel"] <= n, fast[0]
    del ref, cand, same
    torch.cuda.empty_cache()


def test_rejected_and_identical(dev):
    r = torch.randn(5000, device=dev)
    cands = [r.clone(), None, r.to(torch.float16), r.clone()]
    cands[3][4321] = float("nan")
    for fn in (kb.locate, kb.screen_positions):
        recs, locs = fn(r, cands, 1e-5, 1e-5)
        assert locs[0] == {"first_mismatch": -1, "max_abs_index": -1, "max_rel_index": -1}
        assert locs[1] == locs[0] and locs[2] == locs[0]
        assert locs[3] == {"first_mismatch": 4321, "max_abs_index": -1, "max_rel_index": -1}


def test_positions_without_elements(dev):
    """No element to read (an empty reference, or every candidate rejected):
    the records come from the table alone and every position is -1."""
    none = {"first_mismatch": -1, "max_abs_index": -1, "max_rel_index": -1}
    e = torch.empty(0, device=dev)
    recs, locs = kb.screen_positions(e, [e.clone(), None], 1e-5, 1e-5)
    assert locs == [none, none] and recs[0]["passed"] == 1 and recs[1]["passed"] == 0
    r = torch.randn(1000, device=dev)
    recs, locs = kb.screen_positions(r, [None, r.to(torch.float16)], 1e-5, 1e-5)
    assert locs == [none, none] and not any(x["passed"] for x in recs)


def test_positions_many_candidates_host_table(dev):
    """More candidates than travel in the kernel arguments (the launch table
    in pinned host memory), rejected ones among them, with ties planted."""
    rng = np.random.default_rng(77)
    n = 512 * 9 + 100
    r32 = rng.uniform(-1.0, 1.0, n).astype(np.float32)
    ref = to_dev(r32, "f32", dev)
    cands, host = [], []
    for k in range(kb.KB_INLINE_CANDS + 72):
        if k % 41 == 5:
            cands.append(None)
            continue
        c = r32.copy()
        for p in rng.integers(0, n, 1 + k % 4):
            c[p] = r32[p] + 0.5
        c += rng.standard_normal(n).astype(np.float32) * np.float32(1e-6 * (k % 3))
        cands.append(to_dev(c, "f32", dev))
    live = [c for c in cands if c is not None]
    want = oracle_positions(ref, live, 1e-4, 1e-4)
    recs, locs = kb.screen_positions(ref, cands, 1e-4, 1e-4)
    it = iter(want)
    for k, (c, l) in enumerate(zip(cands, locs)):
        w = {"first_mismatch": -1, "max_abs_index": -1, "max_rel_index": -1} if c is None else next(it)
        assert l == w, (k, l, w)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_positions_many_super_groups(dev, dt):
    """One candidate group over 2^24 elements: many stripes, combined in two
    levels, with the maxima tied in stripes far apart (the smallest index
    must survive both levels) and the first mismatch late."""
    n = 1 << 24
    rng = np.random.default_rng(5)
    r32 = rng.uniform(1.0, 2.0, n).astype(np.float32)
    cands = [r32.copy() for _ in range(3)]
    for p in (n - 1000, n // 3 + 17, n // 2):
        cands[0][p] = r32[p] + 0.75
    cands[1][n - 600] = 0.0
    ref = to_dev(CONV[dt](r32), dt, dev)
    cd = [to_dev(CONV[dt](c), dt, dev) for c in cands]
    check(ref, cd, 1e-2, 1e-2, 0, "%s many super-groups" % dt)


def test_screener_positions_repeated(dev):
    """Repeated launches of one Screener with positions: the workspace is
    left clean by each call, and every launch gives the same records and
    positions."""
    w, _ = oracle_workload("c2", dev, seed=1, scale=1 / 64, K=16)
    want = oracle_positions(w.ref, w.cands, w.atol, w.rtol)
    s = kb.Screener(w.ref, w.cands, w.atol, w.rtol, positions=True)
    first = None
    for _ in range(3):
        s.launch()
        s.read()
        recs = s.records()
        assert s.positions() == want
        first = first or recs
        assert recs == first


WIDEN = {"f32": lambda s: s.view(np.float32), "f16": oracle.f16_to_f32_n, "bf16": oracle.bf16_to_f32_n}


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_separate_pass_given_maxima(dev, dt):
    """kb_screen_locate takes the maxima from the records it is given.  With
    maxima other than the candidate's own -- a value many elements exceed,
    one no element has, +inf, a tiny subnormal, a max rel below 2^-100 --
    the cheap pass must still let through every element that equals them:
    the positions equal the oracle's kbo_locate for the same maxima."""
    n = 512 * 64 + 129
    rng = np.random.default_rng(57)
    r32 = rng.standard_normal(n).astype(np.float32)
    zeros = rng.choice(n, 40, replace=False)
    r32[zeros] = 0.0  # d / 0 = +inf where the candidate differs
    c32 = (r32 * (1 + rng.uniform(-2e-2, 2e-2, n))).astype(np.float32)
    c32[zeros[:20]] = 0.5
    c32[rng.choice(n, 5, replace=False)] = np.inf  # d = +inf
    ref = to_dev(CONV[dt](r32), dt, dev)
    cand = to_dev(CONV[dt](c32), dt, dev)
    rs, cs = storage(ref), storage(cand)
    r, c = WIDEN[dt](rs), WIDEN[dt](cs)
    with np.errstate(all="ignore"):
        d = np.abs(c - r)
        q = d / np.abs(r)
    fin_d = np.flatnonzero(np.isfinite(d) & (d > 0))
    fin_q = np.flatnonzero(np.isfinite(q) & (q > 0))
    k1, k2 = int(fin_d[len(fin_d) // 3]), int(fin_q[len(fin_q) // 2])
    absent = np.nextafter(d[k1], np.float32(np.inf))
    while np.any(d == absent):
        absent = np.nextafter(absent, np.float32(np.inf))
    atol, rtol = 1e-3, 1e-3
    d_stats, _ = kb.kb_screen(ref, [cand], atol, rtol, 0)
    torch.cuda.synchronize()
    base = (kb.KbStats * 1).from_buffer_copy(d_stats.cpu().numpy().tobytes())
    assert base[0].mismatches > 0
    cases = [(d[k1], q[k2]), (absent, q[k2]), (np.inf, np.inf), (np.float32(2.0 ** -140), np.float32(2.0 ** -110)),
             (np.nanmax(d[np.isfinite(d)]), np.float32(2.0 ** -101)), (d[k1], np.inf)]
    for max_abs, max_rel in cases:
        rec = (kb.KbStats * 1).from_buffer_copy(bytes(base))
        rec[0].max_abs_err, rec[0].max_rel_err = float(max_abs), float(max_rel)
        given = torch.frombuffer(bytearray(bytes(rec)), dtype=torch.uint8).to(dev)
        say("given maxima", dt, float(max_abs), float(max_rel))
        got = kb.kb_screen_locate(ref, [cand], atol, rtol, given)
        fm, ai, ri = oracle.locate(rs, cs, dt, atol, rtol, float(max_abs), float(max_rel))
        assert got[0] == {"first_mismatch": fm, "max_abs_index": ai, "max_rel_index": ri}, \
            (dt, float(max_abs), float(max_rel), got[0], (fm, ai, ri))
