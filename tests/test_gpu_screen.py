"""Parity of the HIP screening path with the CPU oracle (GPU).

Every case hands the same bytes to the library (on the GPU, through the C
interface) and to the oracle (host copy), then compares every record field:
counts, flags and maxima exactly, the binary64 sums and the relative L2 error
within 1e-6 relative.
"""
import math
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
import synth
from tests.helpers import (THREADS, assert_records_match, check_partial, dtype_name, ensure_built,
                           oracle_positions_host, oracle_records, oracle_workload, same_record, storage)

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(arr, dt, dev):
    """numpy storage (float32 or uint16 bits) -> device tensor of dtype dt."""
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(dev)
    bits = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).to(dev)
    return bits.view(TORCH_DT[dt])


def run_case(ref, cands, atol, rtol, flags=0, label=""):
    recs, _ = kb.screen(ref, cands, atol, rtol, flags)
    orc = oracle_records(ref, cands, atol, rtol, flags)
    assert_records_match(recs, orc, label)
    return recs


# ------------------------------------------------------------ hand cases ---

INF, NAN = float("inf"), float("nan")
HAND = [
    # (dtype, ref values, cand values, atol, rtol, flags)
    ("f32", [0.0], [-0.0], 0.0, 0.0, 0),
    ("f32", [1.0], [NAN], 1e-5, 1e-5, 0),
    ("f32", [INF], [INF], 1e-5, 1e-5, 0),
    ("f32", [INF], [-INF], 1e-5, 1e-5, 0),
    ("f32", [INF], [5.0], 1e-5, 1e-5, 0),
    ("f32", [0.0], [1.0], 0.0, 0.5, 0),
    ("f32", [1.0, 1.0], [1.0 + 2**-10, 1.0 + 2**-10 + 2**-23], 0.0, 2**-10, 0),
    ("f32", [2.0**-149], [0.0], 0.0, 0.5, 0),
    ("f32", [2.0**-149], [2.0**-148], 1e-8, 0.0, 0),
    ("f32", [1, 2, 3, 4, 5, 6, 7, 8], [1, NAN, INF, -INF, 5.1, 6, 7, 8], 1e-5, 1e-5, 0),
    ("f32", [NAN], [NAN], 1e-5, 1e-5, 0),
    ("f32", [NAN], [NAN], 1e-5, 1e-5, kb.KB_EQUAL_NAN),
    ("f32", [1.0], [NAN], 1e-5, 1e-5, kb.KB_EQUAL_NAN),
    ("f32", [1000.0, 1e-3], [1001.0, 2e-3], 0.0, 0.0, 0),
    ("f32", [3.0, 4.0], [3.5, 4.0], 0.0, 0.0, 0),
    ("f32", [3.4028234663852886e38, -3.4028234663852886e38], [-3.4028234663852886e38, INF], 1e-5, 1e-5, 0),
]


@pytest.mark.parametrize("case", range(len(HAND)))
def test_hand_cases(dev, case):
    dt, r, c, atol, rtol, flags = HAND[case]
    say("hand case", case, HAND[case])
    ref = to_dev(np.array(r, dtype=np.float32), dt, dev)
    cand = to_dev(np.array(c, dtype=np.float32), dt, dev)
    run_case(ref, [cand], atol, rtol, flags, "hand %d" % case)


def test_hand_16bit(dev):
    say("hand 16-bit cases")
    ref = to_dev(np.array([0x7BFF], dtype=np.uint16), "f16", dev)
    cand = to_dev(np.array([0x7C00], dtype=np.uint16), "f16", dev)
    run_case(ref, [cand], 1e-3, 1e-3, 0, "f16 overflow")
    ref = to_dev(np.array([0x3F80], dtype=np.uint16), "bf16", dev)
    cand = to_dev(np.array([0x3F81], dtype=np.uint16), "bf16", dev)
    run_case(ref, [cand], 1e-2, 1e-2, 0, "bf16 ulp")


# ------------------------------------------------------ random, ragged ---

SPECIAL_F32 = np.array([0.0, -0.0, 2.0**-149, -(2.0**-149), 2.0**-126, 1e-30, np.inf, -np.inf,
                        np.nan, 3.4028234663852886e38, 65504.0, 1e-8], dtype=np.float32)


def random_pair(rng, dt, n, K):
    """Reference and K candidates with perturbations at many scales and
    injected special values."""
    if dt == "f32":
        r = (rng.standard_normal(n) * np.exp(rng.uniform(-8, 8, n))).astype(np.float32)
    else:
        r32 = rng.standard_normal(n).astype(np.float32) * np.float32(4.0)
        r = oracle.f32_to_f16_n(r32) if dt == "f16" else oracle.f32_to_bf16_n(r32)
    spec_idx = rng.random(n) < 0.01
    if dt == "f32":
        r[spec_idx] = rng.choice(SPECIAL_F32, size=int(spec_idx.sum()))
    else:
        r[spec_idx] = rng.integers(0, 1 << 16, size=int(spec_idx.sum())).astype(np.uint16)
    cands = []
    for k in range(K):
        c = r.copy()
        mode = k % 5
        if dt == "f32":
            if mode == 1:
                # (a reference near the binary32 maximum may round to an
                # infinity here: one more special value)
                with np.errstate(over="ignore"):
                    c = (r * (1 + rng.uniform(-1e-5, 1e-5, n))).astype(np.float32)
            elif mode == 2:
                c = (r + rng.standard_normal(n).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
            elif mode == 3:
                m = rng.random(n) < 0.02
                c[m] = rng.choice(SPECIAL_F32, size=int(m.sum()))
            elif mode == 4:
                c = c.view(np.uint32) ^ (rng.random(n) < 0.05).astype(np.uint32)
                c = c.view(np.float32)
        else:
            if mode in (1, 2):
                flip = rng.random(n) < (0.05 if mode == 1 else 0.5)
                c = c ^ (flip * rng.integers(1, 1 << (3 + mode * 3), size=n)).astype(np.uint16)
            elif mode == 3:
                m = rng.random(n) < 0.02
                c[m] = rng.integers(0, 1 << 16, size=int(m.sum())).astype(np.uint16)
            elif mode == 4:
                c = c ^ (rng.random(n) < 0.001).astype(np.uint16)
        cands.append(c)
    return r, cands


SIZES = [1, 3, 7, 8, 9, 63, 255, 256, 257, 1023, 4095, 4096, 4099, 65536 + 5, (1 << 20) + 13]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_random_ragged(dev, dt):
    rng = np.random.default_rng({"f32": 1, "f16": 2, "bf16": 3}[dt])
    for n in SIZES:
        for K in (1, 3, 9, 17):
            if n > 100000 and K > 9:
                continue
            say("random", dt, "n", n, "K", K)
            r, cs = random_pair(rng, dt, n, K)
            atol, rtol = (1e-5, 1e-5) if dt == "f32" else (1e-3, 1e-3)
            ref = to_dev(r, dt, dev)
            cands = [to_dev(c, dt, dev) for c in cs]
            run_case(ref, cands, atol, rtol, int(rng.integers(0, 2)), "%s n=%d K=%d" % (dt, n, K))


# ------------------------------------- rare paths of the chunk loop ---
# Each case reaches a rule of the definition that the kernel's fast path
# only meets through a rare branch, at sizes that run the chunk loop (not
# only the ragged tail, which applies the definition element by element).


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_signed_zero_is_the_only_difference(dev, dt):
    """A candidate that differs from the reference only in the sign of one
    zero: it matches everywhere, but it is not bitwise identical."""
    say("signed zero only", dt)
    rng = np.random.default_rng(31)
    n = 512 * 64 + 7
    r32 = rng.standard_normal(n).astype(np.float32)
    r32[rng.integers(0, n, n // 10)] = 0.0
    zeros = np.flatnonzero(r32 == 0.0)
    inner = zeros[(zeros > 512 * 8) & (zeros < n - 512)]
    conv = {"f32": lambda x: x, "f16": lambda x: x.astype(np.float16).view(np.uint16),
            "bf16": lambda x: (x.view(np.uint32) >> 16).astype(np.uint16)}[dt]
    r = conv(r32)
    sign = np.float32(-0.0) if dt == "f32" else np.uint16(0x8000)
    cands = []
    for pos in (inner[0], inner[len(inner) // 2], zeros[-1]):
        c = r.copy()
        c[pos] = sign
        cands.append(c)
    recs = run_case(to_dev(r, dt, dev), [to_dev(c, dt, dev) for c in cands], 0.0, 0.0, 0, "signed zero " + dt)
    assert all(x["bitwise_equal"] == 0 and x["mismatches"] == 0 for x in recs)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_all_differences_tiny(dev, dt):
    """Differences all far below 2^-60: their binary32 squares would
    underflow, so the sum of squared differences needs binary64 squares."""
    say("tiny differences", dt)
    rng = np.random.default_rng(32)
    n = 512 * 48 + 100
    r32 = (rng.standard_normal(n) * 2.0**-70).astype(np.float32)
    c32 = (r32 * (1.0 + rng.uniform(-1, 1, n) * 2.0**-9)).astype(np.float32)
    if dt == "bf16":
        r = (r32.view(np.uint32) >> 16).astype(np.uint16)
        c = (c32.view(np.uint32) >> 16).astype(np.uint16)
    else:
        r, c = r32, c32
    recs = run_case(to_dev(r, dt, dev), [to_dev(c, dt, dev)], 0.0, 1e-3, 0, "tiny " + dt)
    assert 0.0 < recs[0]["sum_sq_diff"] < 2.0**-140


def test_max_rel_underflow_blind_spot(dev):
    """The max-rel filter's blind spot: with subnormal references, the
    residual d - O|r| of an element whose quotient exceeds the running
    maximum O can round to zero.  Every wave first meets elements of
    quotient fl(5/7) (r = 7 s, c = 12 s, s = 2^-149), then, in its last
    chunk, elements of quotient fl(8/11) (r = 11 s, c = 19 s), whose
    residual 8 s - fl(5/7) 11 s is below s / 2.  The record must hold
    fl(8/11)."""
    say("max-rel blind spot")
    n = 1 << 21
    plan = kb.kb_screen_launch(1, n, kb.KB_F32)
    wstride = 4 * plan["blocks_per_group"]  # chunks per round of the group's waves
    n_chunks = n // 512
    assert n_chunks >= 2 * wstride, plan
    s = np.float32(2.0**-149)
    r = np.full(n, 7, dtype=np.float32) * s
    c = np.full(n, 12, dtype=np.float32) * s
    last = (n_chunks - wstride) * 512  # every wave's last chunk
    r[last:] = np.float32(11) * s
    c[last:] = np.float32(19) * s
    recs = run_case(to_dev(r, "f32", dev), [to_dev(c, "f32", dev)], 0.0, 0.0, 0, "blind spot")
    assert recs[0]["max_rel_err"] == float(np.float32(8.0) / np.float32(11.0))


# ----------------------------------------------- the five workloads ---

SCALED = [("c1", 1.0, None), ("c2", 1 / 64, None), ("c3", 1.0, None), ("c4", 1 / 64, None),
          ("c5", 1 / 256, None)]


# ------------------------------------------------------- launch shapes ---

@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_one_group_many_super_groups(dev, dt):
    """At most four candidates over millions of elements form one group that
    gets a stripe per resident work-group: the finish's second level then
    combines more than 48 super-groups of 16 stripes (more than 64 takes its
    lanes two passes), which no other case reaches."""
    n = 12 * (1 << 20) + 333
    rng = np.random.default_rng(23)
    r, cs = random_pair(rng, dt, n, 5)
    code = {"f32": kb.KB_F32, "bf16": kb.KB_BF16}[dt]
    atol, rtol = (1e-5, 1e-5) if dt == "f32" else (1e-3, 1e-3)
    ref = to_dev(r, dt, dev)
    for picks in ([2], [1, 2, 3, 4]):
        K = len(picks)
        plan = kb.kb_screen_launch(K, n, code)
        S = (plan["blocks_per_group"] + 15) // 16
        say("one group", dt, "K", K, plan, "super-groups", S)
        assert plan["n_groups"] == 1 and S > 48, plan
        cands = [to_dev(cs[i], dt, dev) for i in picks]
        for flags in (0, kb.KB_EQUAL_NAN):
            run_case(ref, cands, atol, rtol, flags, "%s one group K=%d flags=%d" % (dt, K, flags))
        del cands


@pytest.mark.parametrize("name,scale,K", SCALED)
def test_workloads_scaled(dev, name, scale, K):
    say("workload", name, "scale", scale)
    w, _ = oracle_workload(name, dev, seed=0, scale=scale, K=K)
    run_case(w.ref, w.cands, w.atol, w.rtol, 0, name)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workloads_full_size(dev, name):
    """The exact sizes and launch configuration the benchmark times, on the
    workload the oracle built (the oracle screens its own host arrays); and,
    at those sizes, the positions of every candidate in both forms and the
    fail-fast screen."""
    spec = synth.SPECS[name]
    code = {"f32": kb.KB_F32, "f16": kb.KB_F16, "bf16": kb.KB_BF16}[spec["dtype"]]
    say("full-size workload", name, kb.kb_screen_launch(spec["K"], math.prod(spec["shape"]), code))
    w, ow = oracle_workload(name, dev, seed=0)
    torch.cuda.synchronize()
    recs, _ = kb.screen(w.ref, w.cands, w.atol, w.rtol)
    orc = oracle_records(ow.ref, ow.cands, ow.atol, ow.rtol, dt=ow.dtype)
    assert_records_match(recs, orc, name + " full")
    # the positions at the same sizes, in both forms (the separate pass, and
    # the screening pass with positions), against kbo_locate with the
    # oracle's own maxima
    say("full-size positions", name)
    want = oracle_positions_host(ow.ref, ow.cands, ow.dtype, ow.atol, ow.rtol, orc)
    _, sep = kb.locate(w.ref, w.cands, w.atol, w.rtol)
    frecs, fused = kb.screen_positions(w.ref, w.cands, w.atol, w.rtol)
    assert_records_match(frecs, orc, name + " full, with positions")
    bad = [(k, s_, f, o) for k, (s_, f, o) in enumerate(zip(sep, fused, want)) if s_ != o or f != o]
    assert not bad, (name, len(bad), bad[:4])
    # the fail-fast screen at the same sizes: a passing candidate's record
    # is its plain record (sums within 1e-6), a failing one's is bounded by
    # the oracle's over the whole tensor
    say("full-size fail-fast", name)
    fast, ssum = kb.screen(w.ref, w.cands, w.atol, w.rtol, kb.KB_FAIL_FAST)
    for k, (g, f, o) in enumerate(zip(fast, recs, orc)):
        if o["mismatches"] == 0:
            assert same_record(g, f), (name, k, g, f)
        else:
            check_partial(g, o, "%s full cand %d" % (name, k))
    del w, ow
    torch.cuda.empty_cache()


# ---------------------------------------------------------- policy gate ---

def test_policy_gate_rejects_and_others_unaffected(dev):
    say("policy gate")
    g = torch.Generator(device=dev).manual_seed(5)
    ref = torch.randn(1000, generator=g, device=dev)
    good = ref + 1e-7
    wide = torch.randn(2000, generator=g, device=dev)
    cands = [good, ref.half(), ref[:999].clone(), ref.view(10, 100).clone(), wide[::2], None,
             ref.clone()]
    recs, summ = kb.screen(ref, cands, 1e-5, 1e-5)
    assert [r["status"] for r in recs] == [0, kb.KB_REJECT_DTYPE, kb.KB_REJECT_SHAPE,
                                          kb.KB_REJECT_SHAPE, kb.KB_REJECT_LAYOUT,
                                          kb.KB_REJECT_NULL, 0]
    for k in (1, 2, 3, 4, 5):
        r = recs[k]
        assert r["numel"] == 0 and r["mismatches"] == 0 and r["bitwise_equal"] == 0
        assert r["passed"] == 0
    assert summ == {"n_candidates": 7, "n_passed": 2, "n_rejected": 5, "n_failed": 0,
                    "first_passed": 0, "first_failed": 1}
    orc = oracle_records(ref, [good, cands[6]], 1e-5, 1e-5)
    assert_records_match([recs[0], recs[6]], orc, "gate survivors")


def test_all_rejected_and_empty(dev):
    say("all rejected / empty")
    ref = torch.zeros(16, device=dev)
    recs, summ = kb.screen(ref, [None, ref.half()], 0.0, 0.0)
    assert [r["status"] for r in recs] == [kb.KB_REJECT_NULL, kb.KB_REJECT_DTYPE]
    assert summ["n_rejected"] == 2
    e = torch.empty(0, device=dev)
    recs, summ = kb.screen(e, [e.clone(), e.clone()], 1e-5, 1e-5)
    for r in recs:
        assert r["status"] == 0 and r["numel"] == 0 and r["bitwise_equal"] == 1 and r["passed"] == 1
    assert summ["n_passed"] == 2


# --------------------------------------------------- determinism & reuse ---

def test_determinism_and_workspace_reuse(dev):
    say("determinism")
    w, _ = oracle_workload("c2", dev, seed=1, scale=1 / 16)
    K = len(w.cands)
    ws = kb.alloc_workspace(K, w.numel, kb.KB_BF16, dev)
    st = kb.alloc_stats(K, dev)
    first = None
    for it in range(20):
        if it % 5 == 4:
            # a dirtied workspace is usable again after re-initialisation
            ws.fill_(0xFF if it % 2 else 0x5A)
            kb.kb_screen_workspace_init(ws)
        kb.kb_screen(w.ref, w.cands, w.atol, w.rtol, 0, ws, st)
        recs, _ = kb.kb_screen_stats(st, K)
        if first is None:
            first = recs
        else:
            assert recs == first, it
    assert_records_match(first, oracle_records(w.ref, w.cands, w.atol, w.rtol), "c2 1/16")


@pytest.mark.parametrize("mode", ["plain", "fail_fast", "positions"])
def test_dirty_workspace_is_reported(dev, mode):
    """Workspaces that break the zero-fill contract: filled with 0xFF bytes,
    with random bytes, and used for other sizes without a new zero-fill
    (the partials of one call then lie where the next call's counters are).
    Every call's readback must either be the oracle's records (and, with
    positions, the oracle's positions) or raise KB_ERR_WORKSPACE -- never
    wrong records -- and the garbage fills must be caught.  After
    kb_screen_workspace_init every call is exact again."""
    flags = kb.KB_FAIL_FAST if mode == "fail_fast" else 0
    big, _ = oracle_workload("c4", dev, seed=2, scale=1 / 256, K=40)
    small, _ = oracle_workload("c1", dev, seed=2)
    plan = kb.kb_screen_launch(40, big.numel, kb.KB_F16)
    say("dirty workspace", mode, plan)
    assert plan["n_groups"] > 1 and plan["blocks_per_group"] > 16, plan  # two-level finish
    size = kb.kb_screen_positions_workspace_bytes if mode == "positions" else kb.kb_screen_workspace_bytes
    nbytes = max(size(40, big.numel, kb.KB_F16), size(4, small.numel, kb.KB_F32))
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    orcs = {w.name: oracle_records(w.ref, w.cands, w.atol, w.rtol) for w in (big, small)}
    locs = {}
    if mode == "positions":
        for w in (big, small):
            r = storage(w.ref)
            locs[w.name] = []
            for c, o in zip(w.cands, orcs[w.name]):
                fm, ai, ri = oracle.locate(r, storage(c), dtype_name(w.ref), w.atol, w.rtol, o["max_abs_err"],
                                           o["max_rel_err"])
                locs[w.name].append({"first_mismatch": fm, "max_abs_index": ai, "max_rel_index": ri})
    g = torch.Generator(device=dev).manual_seed(99)

    def run(w):
        st = kb.alloc_stats(len(w.cands), dev)
        d_loc = kb.alloc_locate(len(w.cands), dev) if mode == "positions" else None
        kb.kb_screen(w.ref, w.cands, w.atol, w.rtol, flags, ws, st, d_loc=d_loc)
        try:
            recs, _ = kb.kb_screen_stats(st, len(w.cands))
        except kb.KbError as e:
            assert e.code == kb.KB_ERR_WORKSPACE, e
            return None
        orc = orcs[w.name]
        if d_loc is not None:
            assert kb.read_locate(d_loc, len(w.cands)) == locs[w.name], w.name
        if flags == 0:
            assert_records_match(recs, orc, w.name)
        else:
            assert [r["passed"] for r in recs] == [o["passed"] for o in orc], w.name
            assert_records_match([r for r, o in zip(recs, orc) if o["passed"]],
                                 [o for o in orc if o["passed"]], w.name)
        return recs

    ws.fill_(0xFF)
    assert run(big) is None, "0xFF workspace not reported"
    ws.copy_(torch.randint(0, 256, (nbytes,), generator=g, device=dev, dtype=torch.uint8))
    assert run(big) is None, "random workspace not reported"
    kb.kb_screen_workspace_init(ws)
    assert run(big) is not None
    assert run(big) is not None  # consecutive calls of one size need nothing
    run(small)  # other sizes without a new zero-fill: exact, or reported
    run(big)
    kb.kb_screen_workspace_init(ws)
    assert run(small) is not None
    kb.kb_screen_workspace_init(ws)
    assert run(big) is not None


def test_pinned_host_records_pipeline(dev):
    say("pinned host records")
    w, _ = oracle_workload("c2", dev, seed=4, scale=1 / 64)
    scr = kb.Screener(w.ref, w.cands, w.atol, w.rtol, host_slots=2)
    ev = [torch.cuda.Event(), torch.cuda.Event()]
    seen = []
    for i in range(6):
        scr.launch(i % 2)
        ev[i % 2].record()
        if i > 0:
            ev[(i - 1) % 2].synchronize()
            seen.append((scr.summarize((i - 1) % 2).as_dict(), scr.records((i - 1) % 2)))
    ev[5 % 2].synchronize()
    seen.append((scr.summarize(5 % 2).as_dict(), scr.records(5 % 2)))
    orc = oracle_records(w.ref, w.cands, w.atol, w.rtol)
    for summ, recs in seen:
        assert_records_match(recs, orc, "pinned slot")
        assert summ == kb.kb_summarize(recs)


def test_stream_ordering_with_side_stream(dev):
    say("side stream")
    s = torch.cuda.Stream()
    w, _ = oracle_workload("c1", dev, seed=3)
    with torch.cuda.stream(s):
        recs, _ = kb.screen(w.ref, w.cands, w.atol, w.rtol, stream=s)
    assert_records_match(recs, oracle_records(w.ref, w.cands, w.atol, w.rtol), "side stream")


def test_two_streams_concurrent_screens(dev):
    """Screens of the same candidates alternating over two streams, each
    with its own workspace and ring of pinned record slots, overlapping on
    the device (the pipelined bench loop): every record is the oracle's."""
    say("two streams")
    w, _ = oracle_workload("c2", dev, seed=6, scale=1 / 16)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    scrs = [kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st, host_slots=4) for st in streams]
    for i in range(16):
        scrs[i % 2].launch((i // 2) % 4)
    torch.cuda.synchronize()
    orc = oracle_records(w.ref, w.cands, w.atol, w.rtol)
    for sc in scrs:
        for slot in range(4):
            assert_records_match(sc.records(slot), orc, "two streams slot %d" % slot)


def test_host_threads_each_on_its_own_stream(dev):
    """Four host threads use the library at once, each on its own stream with
    its own workload (one of more than 128 candidates, so a host launch
    table; one with positions in the screening pass): every call of every
    thread gives the records and positions of a call made alone."""
    say("host threads")
    cases = [("c2", 1 / 64, 16, False), ("c3", 1 / 16, 200, False), ("c4", 1 / 256, 40, True),
             ("c5", 1 / 1024, 8, False)]
    work, alone = [], []
    for name, scale, K, pos in cases:
        w, _ = oracle_workload(name, dev, seed=9, scale=scale, K=K)
        if pos:
            recs, locs = kb.screen_positions(w.ref, w.cands, w.atol, w.rtol)
        else:
            (recs, _), locs = kb.screen(w.ref, w.cands, w.atol, w.rtol), None
        assert_records_match(recs, oracle_records(w.ref, w.cands, w.atol, w.rtol), name + " alone")
        work.append((w, pos))
        alone.append((recs, locs))
    torch.cuda.synchronize()

    def run(t):
        w, pos = work[t]
        st = torch.cuda.Stream()
        with torch.cuda.stream(st):
            for i in range(12):
                if pos:
                    recs, locs = kb.screen_positions(w.ref, w.cands, w.atol, w.rtol, stream=st)
                else:
                    (recs, _), locs = kb.screen(w.ref, w.cands, w.atol, w.rtol, stream=st), None
                # (repr: the same bits, NaN fields included)
                if repr((recs, locs)) != repr(alone[t]):
                    return (t, i)
        return None

    with ThreadPoolExecutor(len(cases)) as ex:
        bad = [r for r in ex.map(run, range(len(cases))) if r is not None]
    assert not bad, bad


# ------------------------------------------------ exhaustive 16-bit pairs ---

@pytest.mark.parametrize("dt,tol", [("f16", 1e-3), ("bf16", 1e-2)])
def test_exhaustive_16bit_pairs(dev, dt, tol):
    """All 2^16 x 2^16 (candidate, reference) bit patterns: the reference holds
    every pattern once; candidate k is the constant pattern k."""
    say("exhaustive", dt)
    allbits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = to_dev(allbits, dt, dev)
    batch = 4096
    bits_dev = torch.from_numpy(allbits.view(np.int16)).to(dev)
    for b0 in range(0, 1 << 16, batch):
        rows = bits_dev[b0:b0 + batch].view(-1, 1).expand(-1, 1 << 16).contiguous()
        cands = [rows[i].view(TORCH_DT[dt]) for i in range(rows.shape[0])]
        recs, _ = kb.screen(ref, cands, tol, tol)

        def one(i):
            return oracle.screen(allbits, np.full(1 << 16, b0 + i, dtype=np.uint16), dt, tol, tol)

        with ThreadPoolExecutor(THREADS) as ex:
            orc = list(ex.map(one, range(rows.shape[0])))
        assert_records_match(recs, orc, "%s exhaustive batch %d" % (dt, b0))
