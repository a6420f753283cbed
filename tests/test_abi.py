"""The C interface without a GPU: library loading, exported symbols, and the
argument checks and policy gate that run on the host before any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2608_02611_amd as kb
from tests.helpers import ensure_built

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    ensure_built()
    return kb.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "kb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kb_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported(L):
    names = declared_functions()
    assert set(kb.EXPORTS) <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_version(L):
    assert kb.kb_version() == 20000


def desc(data, dtype, shape, strides=None):
    t = kb.KbTensor()
    t.data = data
    t.dtype = dtype
    t.ndim = len(shape)
    if strides is None:
        strides, acc = [], 1
        for s in reversed(shape):
            strides.insert(0, acc)
            acc *= s
    for i, (s, st) in enumerate(zip(shape, strides)):
        t.shape[i] = s
        t.strides[i] = st
    return t


def gate(ref, cands):
    arr = (kb.KbTensor * len(cands))(*cands)
    st = (ctypes.c_int32 * len(cands))()
    rc = kb.lib().kb_policy_check(ctypes.byref(ref), arr, len(cands), st)
    return rc, list(st)


def test_policy_gate_statuses(L):
    ref = desc(0x10000, kb.KB_F32, (4, 8))
    cands = [
        desc(0x20000, kb.KB_F32, (4, 8)),                     # ok
        desc(None, kb.KB_F32, (4, 8)),                        # null
        desc(0x30000, kb.KB_F16, (4, 8)),                     # dtype
        desc(0x40000, kb.KB_F32, (8, 4)),                     # shape
        desc(0x50000, kb.KB_F32, (32,)),                      # ndim
        desc(0x60000, kb.KB_F32, (4, 8), strides=(16, 2)),    # layout
        desc(0x70000, kb.KB_F32, (4, 8), strides=(1, 4)),     # transposed layout
        desc(0x80000, kb.KB_F32, (4, 1, 8), ),                # ndim differs
    ]
    rc, st = gate(ref, cands)
    assert rc == kb.KB_OK
    assert st == [kb.KB_STATUS_OK, kb.KB_REJECT_NULL, kb.KB_REJECT_DTYPE, kb.KB_REJECT_SHAPE,
                  kb.KB_REJECT_SHAPE, kb.KB_REJECT_LAYOUT, kb.KB_REJECT_LAYOUT,
                  kb.KB_REJECT_SHAPE]


def test_policy_gate_size_one_dims_and_empty(L):
    ref = desc(0x10000, kb.KB_BF16, (1, 5, 1))
    ok = desc(0x20000, kb.KB_BF16, (1, 5, 1), strides=(999, 1, 7))  # size-1 strides free
    rc, st = gate(ref, [ok])
    assert rc == kb.KB_OK and st == [kb.KB_STATUS_OK]
    ref0 = desc(0x10000, kb.KB_F16, (0, 3))
    rc, st = gate(ref0, [desc(0x20000, kb.KB_F16, (0, 3), strides=(5, 5))])
    assert rc == kb.KB_OK and st == [kb.KB_STATUS_OK]


def test_policy_gate_call_errors(L):
    ref = desc(0x10000, kb.KB_U32, (4,))
    rc, _ = gate(ref, [desc(0x20000, kb.KB_U32, (4,))])
    assert rc == kb.KB_ERR_DTYPE and "dtype" in kb.kb_last_error()
    ref = desc(None, kb.KB_F32, (4,))
    rc, _ = gate(ref, [desc(0x20000, kb.KB_F32, (4,))])
    assert rc == kb.KB_ERR_INVALID_ARG


def screen_rc(ref, cands, atol=1e-5, rtol=1e-5, flags=0, ws=0x100000, ws_bytes=1 << 30,
              stats=0x200000):
    arr = (kb.KbTensor * max(1, len(cands)))(*cands)
    return kb.lib().kb_screen(ctypes.byref(ref) if ref is not None else None, arr, len(cands),
                              atol, rtol, flags, ws, ws_bytes, stats, None)


def test_screen_argument_errors(L):
    ref = desc(0x10000, kb.KB_F32, (64,))
    good = [desc(0x20000, kb.KB_F32, (64,))]
    assert screen_rc(None, good) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, []) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, good, atol=-1.0) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, good, rtol=float("nan")) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, good, atol=float("inf")) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, good, flags=4) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(ref, good, stats=None) == kb.KB_ERR_INVALID_ARG
    assert screen_rc(desc(0x10000, kb.KB_U32, (64,)), good) == kb.KB_ERR_DTYPE
    assert screen_rc(ref, good, ws_bytes=16) == kb.KB_ERR_WORKSPACE
    assert screen_rc(ref, good, ws=None) == kb.KB_ERR_WORKSPACE
    assert screen_rc(desc(0x10004, kb.KB_F32, (64,)), good) == kb.KB_ERR_ALIGNMENT
    assert screen_rc(ref, [desc(0x20008, kb.KB_F32, (64,))]) == kb.KB_ERR_ALIGNMENT
    assert screen_rc(ref, good, ws=0x100008) == kb.KB_ERR_ALIGNMENT
    assert screen_rc(ref, good, stats=0x200004) == kb.KB_ERR_ALIGNMENT
    assert screen_rc(desc(0x10000, kb.KB_F32, (8, 8), strides=(1, 8)), good) == kb.KB_ERR_INVALID_ARG
    assert "contiguous" in kb.kb_last_error()


def test_rejected_misaligned_candidate_is_not_an_error_source(L):
    # a candidate that fails the gate is not read, so its pointer may be anything
    ref = desc(0x10000, kb.KB_F32, (64,))
    bad = desc(0x20002, kb.KB_F16, (64,))
    # the call still fails later for lack of a GPU, but not with an alignment error
    rc = screen_rc(ref, [bad], ws_bytes=16)
    assert rc == kb.KB_ERR_WORKSPACE


def test_workspace_and_launch_plan(L):
    for K, n, dt in [(4, 65536, kb.KB_F32), (16, 4096 * 4096, kb.KB_BF16),
                     (1024, 256 * 1024, kb.KB_F32), (64, 8 * 2048 * 4096, kb.KB_F16),
                     (8, 1 << 30, kb.KB_F32), (1, 0, kb.KB_F32), (3, 7, kb.KB_F16)]:
        ws = kb.kb_screen_workspace_bytes(K, n, dt)
        assert ws > 0 and ws % 256 == 0
        plan = kb.kb_screen_launch(K, n, dt)
        assert plan["blocks_per_group"] % 8 == 0
        assert plan["group_size"] * plan["n_groups"] >= K
        assert plan["grid"] == plan["n_groups"] * plan["blocks_per_group"]
        # one work-group never holds 2^31 or more elements of one candidate
        assert n / plan["blocks_per_group"] < 2 ** 31
    assert kb.kb_screen_workspace_bytes(0, 10, kb.KB_F32) == 0
    assert kb.kb_screen_workspace_bytes(4, 10, kb.KB_U32) == 0
    with pytest.raises(kb.KbError):
        kb.kb_screen_launch(4, 10, kb.KB_U32)


def test_gen_argument_errors(L):
    g = kb.lib().kb_gen_inputs
    assert g(0x1000, kb.KB_F32, 16, kb.KB_DIST_U32, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_DTYPE
    assert g(0x1000, kb.KB_U32, 16, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_DTYPE
    assert g(0x1000, 7, 16, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_DTYPE
    assert g(0x1000, kb.KB_F32, 16, 9, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert g(0x1000, kb.KB_F32, 16, kb.KB_DIST_NORMAL, float("nan"), 1.0, 0, 0, 0, 0,
             None) == kb.KB_ERR_INVALID_ARG
    assert g(None, kb.KB_F32, 16, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert g(0x1004, kb.KB_F32, 16, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_ALIGNMENT
    assert g(0x1000, kb.KB_F32, 16, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 2**64 - 4,
             None) == kb.KB_ERR_INVALID_ARG
    # n = 0 is a no-op: no launch, no error
    assert g(None, kb.KB_F32, 0, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_OK


def test_noalloc_argument_errors(L):
    """kb_screen_noalloc refuses, before any device work, what kb_screen
    refuses, and more than KB_INLINE_CANDS candidates."""
    ref = desc(0x10000, kb.KB_F32, (64,))
    f = kb.lib().kb_screen_noalloc

    def call(cands, atol=1e-5, stats=0x200000, flags=0):
        arr = (kb.KbTensor * max(1, len(cands)))(*cands)
        return f(ctypes.byref(ref), arr, len(cands), atol, 1e-5, flags, stats, None)

    good = [desc(0x20000, kb.KB_F32, (64,))]
    assert call([]) == kb.KB_ERR_INVALID_ARG
    assert call(good, atol=-1.0) == kb.KB_ERR_INVALID_ARG
    assert call(good, stats=None) == kb.KB_ERR_INVALID_ARG
    assert call(good, flags=8) == kb.KB_ERR_INVALID_ARG
    assert call(good * (kb.KB_INLINE_CANDS + 1)) == kb.KB_ERR_INVALID_ARG
    assert "at most" in kb.kb_last_error()
    assert kb.NOALLOC_SCRATCH_BYTES >= max(kb.kb_screen_workspace_bytes(kb.KB_INLINE_CANDS, 1 << 32, dt)
                                           for dt in (kb.KB_F32, kb.KB_F16, kb.KB_BF16))


def test_derived_generator_argument_errors(L):
    """The derived-input calls refuse bad arguments before any device work."""
    sm, ix, pt, sc = (kb.lib().kb_gen_softmax_rows, kb.lib().kb_gen_indices, kb.lib().kb_gen_perturb,
                      kb.lib().kb_gen_scatter)
    assert sm(0x1000, kb.KB_F16, 4, 4, 2.0, 0, 0, 0, None) == kb.KB_ERR_DTYPE
    assert sm(0x1000, kb.KB_F32, 4, 0, 2.0, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert sm(0x1000, kb.KB_F32, 4, 4, float("inf"), 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert sm(0x1008, kb.KB_F32, 4, 4, 2.0, 0, 0, 0, None) == kb.KB_ERR_ALIGNMENT
    assert sm(None, kb.KB_F32, 0, 4, 2.0, 0, 0, 0, None) == kb.KB_OK  # no rows: nothing to do
    assert ix(0x1000, 0, 100, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert ix(0x1000, 6, 11, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG  # 2 m > n
    assert ix(0x1000, kb.KB_MAX_INDICES + 1, 1 << 40, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert ix(None, 5, 100, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG
    assert ix(0x1008, 5, 100, 0, 0, 0, None) == kb.KB_ERR_ALIGNMENT
    ok = (0x1000, 0x2000, kb.KB_F32, 16, kb.KB_PERTURB_ADD_UNIFORM, 0.0, 1.0, 0.5, 0, 0, 0, 0, None)

    def perturb(**kw):
        a = list(ok)
        for i, k in enumerate(("dst", "src", "dtype", "n", "op", "a", "b", "p")):
            if k in kw:
                a[i] = kw[k]
        return pt(*a)

    assert perturb(op=0) == kb.KB_ERR_INVALID_ARG and perturb(op=8) == kb.KB_ERR_INVALID_ARG
    assert perturb(dtype=kb.KB_U32) == kb.KB_ERR_DTYPE
    assert perturb(dtype=kb.KB_F16, op=kb.KB_PERTURB_SPECIALS) == kb.KB_ERR_DTYPE
    assert perturb(p=float("nan")) == kb.KB_ERR_INVALID_ARG
    assert perturb(src=None) == kb.KB_ERR_INVALID_ARG
    assert perturb(dst=0x1004) == kb.KB_ERR_ALIGNMENT
    assert perturb(dst=None, src=None, n=0) == kb.KB_OK
    assert pt(0x1000, 0x2000, kb.KB_F32, 16, 1, 0.0, 1.0, 0.0, 0, 0, 0, 2 ** 64 - 8, None) == kb.KB_ERR_INVALID_ARG
    assert sc(0x1000, 0x2000, kb.KB_F32, 16, 0x3000, 4, 3, None) == kb.KB_ERR_INVALID_ARG
    assert sc(0x1000, 0x2000, kb.KB_U32, 16, 0x3000, 4, 1, None) == kb.KB_ERR_DTYPE
    assert sc(0x1000, None, kb.KB_F32, 16, 0x3000, 4, 1, None) == kb.KB_ERR_INVALID_ARG
    assert sc(0x1000, 0x2000, kb.KB_F32, 16, 0x3004, 4, 1, None) == kb.KB_ERR_ALIGNMENT
    g = kb.lib().kb_gen_inputs
    assert g(0x1000, kb.KB_U32, 16, kb.KB_DIST_STUDENT_T3, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_DTYPE
    assert g(0x1000, kb.KB_F32, 16, 4, 0.0, 1.0, 0, 0, 0, 0, None) == kb.KB_ERR_INVALID_ARG


def test_stats_argument_errors(L):
    assert kb.lib().kb_screen_stats(None, 4, None, None, None, None) == kb.KB_ERR_INVALID_ARG
    assert kb.lib().kb_screen_stats(0x1000, -1, None, None, None, None) == kb.KB_ERR_INVALID_ARG


def test_large_calls_need_a_host_table(L):
    """More than KB_INLINE_CANDS candidates: the launch table lives in the
    caller's pinned host memory, so kb_screen (no options) refuses, and
    kb_screen_ex refuses a missing, short or misaligned table -- all before
    any device work."""
    assert kb.lib().kb_screen_host_table_bytes(1) == 0
    assert kb.lib().kb_screen_host_table_bytes(kb.KB_INLINE_CANDS) == 0
    assert kb.lib().kb_screen_host_table_bytes(0) == 0
    need = kb.lib().kb_screen_host_table_bytes(kb.KB_INLINE_CANDS + 1)
    assert need >= 16 * (kb.KB_INLINE_CANDS + 1) and need % 256 == 0
    assert kb.lib().kb_screen_host_table_bytes(1024) >= 16 * 1024
    assert kb.lib().kb_screen_multi_host_table_bytes(3, 1024) == 3 * kb.lib().kb_screen_host_table_bytes(1024)
    assert kb.lib().kb_screen_multi_host_table_bytes(3, 100) == 0
    n = 300
    ref = desc(0x10000, kb.KB_F32, (64,))
    cands = [desc(0x20000 + 256 * k, kb.KB_F32, (64,)) for k in range(n)]
    assert screen_rc(ref, cands) == kb.KB_ERR_WORKSPACE
    assert "host table" in kb.kb_last_error()
    arr = (kb.KbTensor * n)(*cands)
    buf = (ctypes.c_uint8 * (kb.lib().kb_screen_host_table_bytes(n) + 32))()
    base = ctypes.addressof(buf)
    aligned = (base + 15) // 16 * 16

    def ex(ptr, nbytes):
        opts = kb.KbScreenOpts(ptr, nbytes)
        return kb.lib().kb_screen_ex(ctypes.byref(ref), arr, n, 1e-5, 1e-5, 0, 0x100000, 1 << 30,
                                     0x200000, ctypes.byref(opts), None)

    assert ex(None, 1 << 20) == kb.KB_ERR_WORKSPACE
    assert ex(aligned, 256) == kb.KB_ERR_WORKSPACE
    assert ex(aligned + 8, kb.lib().kb_screen_host_table_bytes(n)) == kb.KB_ERR_ALIGNMENT
    # a 2-candidate call ignores the options entirely (inline table)
    assert kb.lib().kb_screen_ex(ctypes.byref(ref), arr, 2, 1e-5, 1e-5, 0, 0x100000, 16, 0x200000,
                                 ctypes.byref(kb.KbScreenOpts(None, 0)), None) == kb.KB_ERR_WORKSPACE
    assert "workspace of 16 bytes" in kb.kb_last_error()


def test_positions_argument_errors(L):
    """kb_screen_ex with positions (opts.d_loc): its own workspace size, and
    the refusals that come before any device work."""
    for dt in (kb.KB_F32, kb.KB_F16, kb.KB_BF16):
        for n, numel in ((1, 1), (16, 1 << 24), (300, 1 << 18), (128, 1 << 32)):
            plain = kb.kb_screen_workspace_bytes(n, numel, dt)
            pos = kb.kb_screen_positions_workspace_bytes(n, numel, dt)
            assert plain > 0 and pos > plain and pos % 256 == 0, (dt, n, numel)
    assert kb.kb_screen_positions_workspace_bytes(0, 64, kb.KB_F32) == 0
    assert kb.kb_screen_positions_workspace_bytes(4, 64, kb.KB_U32) == 0
    ref = desc(0x10000, kb.KB_F32, (4096,))
    cands = [desc(0x20000 + 0x4000 * k, kb.KB_F32, (4096,)) for k in range(3)]
    arr = (kb.KbTensor * 3)(*cands)
    pos = kb.kb_screen_positions_workspace_bytes(3, 4096, kb.KB_F32)
    plain = kb.kb_screen_workspace_bytes(3, 4096, kb.KB_F32)

    def ex(loc, ws_bytes=pos, flags=0):
        opts = kb.KbScreenOpts(None, 0, loc)
        return kb.lib().kb_screen_ex(ctypes.byref(ref), arr, 3, 1e-5, 1e-5, flags, 0x100000, ws_bytes,
                                     0x200000, ctypes.byref(opts), None)

    assert ex(0x300000, flags=kb.KB_FAIL_FAST) == kb.KB_ERR_INVALID_ARG
    assert "KB_FAIL_FAST" in kb.kb_last_error()
    assert ex(0x300000, ws_bytes=plain) == kb.KB_ERR_WORKSPACE
    assert ex(0x300008) == kb.KB_ERR_ALIGNMENT
    # multi-output calls take no positions
    o = kb.KbScreenOpts(None, 0, 0x300000)
    at = (ctypes.c_float * 1)(1e-5)
    assert kb.lib().kb_screen_multi(ctypes.byref(ref), 1, arr, 3, at, at, 0, 0x100000, 1 << 30, 0x200000,
                                    ctypes.byref(o), None) == kb.KB_ERR_INVALID_ARG


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(kb, "_lib", None)
    monkeypatch.setattr(kb, "LIB_PATH", "/nonexistent/libkb.so")
    with pytest.raises(kb.KbError):
        kb.lib()


def test_summarize_on_host(L):
    recs = []
    for status, mism in ((0, 0), (kb.KB_REJECT_DTYPE, 0), (0, 3), (0, 0), (kb.KB_REJECT_NULL, 0)):
        r = {name: 0 for name, _ in kb.KbStats._fields_}
        r["status"], r["mismatches"] = status, mism
        recs.append(r)
    assert kb.kb_summarize(recs) == {"n_candidates": 5, "n_passed": 2, "n_rejected": 2,
                                     "n_failed": 1, "first_passed": 0, "first_failed": 1}
    assert kb.kb_summarize([])["n_candidates"] == 0
    assert kb.lib().kb_summarize(None, 3, None, None) == kb.KB_ERR_INVALID_ARG
    # the per-candidate verdicts come from the library
    arr = (kb.KbStats * 5)()
    for k, r in enumerate(recs):
        for name, _ in kb.KbStats._fields_:
            setattr(arr[k], name, r[name])
    passed = (ctypes.c_int32 * 5)(*([7] * 5))
    assert kb.lib().kb_summarize(arr, 5, None, passed) == kb.KB_OK
    assert list(passed) == [1, 0, 0, 1, 0]
    # a record written by a call that found its workspace not clean makes the
    # verdict an error, not a rejection
    arr[3].status = kb.KB_ERR_WORKSPACE
    assert kb.lib().kb_summarize(arr, 5, None, passed) == kb.KB_ERR_WORKSPACE
    assert "not clean" in kb.kb_last_error()
    assert kb.lib().kb_summarize_multi(arr, 1, 5, ctypes.byref(kb.KbSummary()), None) == kb.KB_ERR_WORKSPACE


def test_summarize_matches_the_verdict_rule(L):
    """The verdict: a candidate passes iff the gate accepted it and it has no
    mismatch (one is enough to fail, and counts past 2^32 are counts);
    first_failed is the first candidate that did not pass."""
    import numpy as np
    rng = np.random.default_rng(3)
    statuses = [kb.KB_STATUS_OK] * 4 + [kb.KB_REJECT_NULL, kb.KB_REJECT_DTYPE, kb.KB_REJECT_SHAPE,
                                        kb.KB_REJECT_LAYOUT]
    for trial in range(200):
        n = int(rng.integers(1, 40))
        recs = []
        for _ in range(n):
            r = {name: 0 for name, _ in kb.KbStats._fields_}
            r["status"] = statuses[int(rng.integers(0, len(statuses)))]
            r["mismatches"] = int(rng.choice([0, 0, 1, 2, 1 << 32, (1 << 40) + 1]))
            recs.append(r)
        ok = [r["status"] == kb.KB_STATUS_OK and r["mismatches"] == 0 for r in recs]
        rej = [r["status"] != kb.KB_STATUS_OK for r in recs]
        want = {"n_candidates": n, "n_passed": sum(ok), "n_rejected": sum(rej),
                "n_failed": n - sum(ok) - sum(rej),
                "first_passed": ok.index(True) if any(ok) else -1,
                "first_failed": ok.index(False) if not all(ok) else -1}
        assert kb.kb_summarize(recs) == want, (trial, recs)
        arr = (kb.KbStats * n)()
        for k, r in enumerate(recs):
            for name, _ in kb.KbStats._fields_:
                setattr(arr[k], name, r[name])
        passed = (ctypes.c_int32 * n)()
        assert kb.lib().kb_summarize(arr, n, None, passed) == kb.KB_OK
        assert [bool(x) for x in passed] == ok, (trial, recs)


def test_workspace_init_argument_errors(L):
    f = kb.lib().kb_screen_workspace_init
    assert f(None, 256, None) == kb.KB_ERR_WORKSPACE
    assert f(0x1000, 0, None) == kb.KB_ERR_WORKSPACE
    assert f(0x1008, 256, None) == kb.KB_ERR_ALIGNMENT
    assert f(0x1000, 250, None) == kb.KB_ERR_ALIGNMENT


def test_locate_argument_errors(L):
    ref = desc(0x10000, kb.KB_F32, (64,))
    arr = (kb.KbTensor * 1)(desc(0x20000, kb.KB_F32, (64,)))
    f = kb.lib().kb_screen_locate
    assert f(None, arr, 1, 1e-5, 1e-5, 0, 0x3000, 0x4000, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 0, 1e-5, 1e-5, 0, 0x3000, 0x4000, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 1, -1.0, 1e-5, 0, 0x3000, 0x4000, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 1, 1e-5, 1e-5, 4, 0x3000, 0x4000, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 1, 1e-5, 1e-5, 0, None, 0x4000, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 1, 1e-5, 1e-5, 0, 0x3000, None, None) == kb.KB_ERR_INVALID_ARG
    assert f(ctypes.byref(ref), arr, 1, 1e-5, 1e-5, 0, 0x3000, 0x4008, None) == kb.KB_ERR_ALIGNMENT
    bad = desc(0x10000, kb.KB_U32, (64,))
    assert f(ctypes.byref(bad), arr, 1, 1e-5, 1e-5, 0, 0x3000, 0x4000, None) == kb.KB_ERR_DTYPE


def test_rung_argument_errors(L):
    f = kb.lib().kb_rung_stats
    ok = dict(samples=0x10000, C=3, S=2, N=16, base=0, rung=1, budget=16.0, alpha=0.02, beta=0.01,
              rows=0x20000, scores=0x30000)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["samples"], a["C"], a["S"], a["N"], a["base"], a["rung"], a["budget"], a["alpha"],
                 a["beta"], a["rows"], a["scores"], None)

    assert call(samples=None) == kb.KB_ERR_INVALID_ARG
    assert call(rows=None) == kb.KB_ERR_INVALID_ARG
    assert call(scores=None) == kb.KB_ERR_INVALID_ARG
    assert call(C=0) == kb.KB_ERR_INVALID_ARG
    assert call(S=0) == kb.KB_ERR_INVALID_ARG
    assert call(N=0) == kb.KB_ERR_INVALID_ARG
    assert call(N=kb.RUNG_MAX_ITER + 1) == kb.KB_ERR_INVALID_ARG
    assert call(base=3) == kb.KB_ERR_INVALID_ARG
    assert call(base=-2) == kb.KB_ERR_INVALID_ARG
    assert call(rung=-1) == kb.KB_ERR_INVALID_ARG
    assert call(budget=-1.0) == kb.KB_ERR_INVALID_ARG
    assert call(budget=float("inf")) == kb.KB_ERR_INVALID_ARG
    assert call(alpha=float("nan")) == kb.KB_ERR_INVALID_ARG
    assert call(samples=0x10004) == kb.KB_ERR_ALIGNMENT
    assert call(rows=0x20004) == kb.KB_ERR_ALIGNMENT
    assert call(scores=0x30002) == kb.KB_ERR_ALIGNMENT
    assert "kb_rung_stats" in kb.kb_last_error()


def test_promote_argument_errors(L):
    f = kb.lib().kb_rung_promote
    ok = dict(sc=0x10000, n=5, base=0, num=2, den=5, rank=0x20000, order=0x30000, prom=0x40000)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["sc"], a["n"], a["base"], a["num"], a["den"], a["rank"], a["order"], a["prom"], None)

    assert call(sc=None) == kb.KB_ERR_INVALID_ARG
    assert call(rank=None) == kb.KB_ERR_INVALID_ARG
    assert call(order=None) == kb.KB_ERR_INVALID_ARG
    assert call(prom=None) == kb.KB_ERR_INVALID_ARG
    assert call(n=0) == kb.KB_ERR_INVALID_ARG
    assert call(n=kb.PROMOTE_MAX + 1) == kb.KB_ERR_INVALID_ARG
    assert call(base=5) == kb.KB_ERR_INVALID_ARG
    assert call(base=-2) == kb.KB_ERR_INVALID_ARG
    assert call(den=0) == kb.KB_ERR_INVALID_ARG
    assert call(num=-1) == kb.KB_ERR_INVALID_ARG
    assert call(num=6) == kb.KB_ERR_INVALID_ARG
    assert call(sc=0x10004) == kb.KB_ERR_ALIGNMENT
    assert call(order=0x30002) == kb.KB_ERR_ALIGNMENT
    assert "kb_rung_promote" in kb.kb_last_error()


def test_survival_host_function(L):
    """The library's survival accounting against the oracle's (host only)."""
    import oracle
    cases = [([21, 7, 3], [5, 2, 0], [7, 3, 3], 21), ([31, 8, 3], [5, 2, 0], [8, 3, 3], 31),
             ([26, 6], [5, 0], [6, 4], 26), ([1], [0], [0], 1), ([0, 0], [0, 0], [0, 0], 5)]
    for entering, failed, promoted, orig in cases:
        g = kb.kb_rung_survival(entering, failed, promoted, orig)
        o = oracle.rung_survival(entering, failed, promoted, orig)
        assert g[0] == list(o[0]) and g[1] == list(o[1])
    fail, promo = kb.kb_rung_survival([21, 7], [5, 2], [7, 3], 21)
    assert [round(x, 1) for x in fail + promo] == [23.8, 28.6, 33.3, 14.3]
    with pytest.raises(kb.KbError):
        kb.kb_rung_survival([3], [4], [0], 3)
    with pytest.raises(kb.KbError):
        kb.kb_rung_survival([3], [1], [1], 0)


def test_gate_matches_the_oracle_on_random_views(L):
    """kb_policy_check (library host code) against the oracle's gate on
    random descriptors: dtypes, shapes, strides, null data."""
    import random
    import oracle
    rnd = random.Random(2024)

    def rand_meta(base):
        shape = list(base["shape"])
        kind = rnd.random()
        if kind < 0.15:
            shape = [max(0, d + rnd.choice([-1, 1])) for d in shape]
        elif kind < 0.2:
            shape = shape + [1]
        dtype = base["dtype"] if rnd.random() > 0.15 else rnd.choice([0, 1, 2])
        strides, acc = [], 1
        for d in reversed(shape):
            strides.append(acc)
            acc *= d
        strides = list(reversed(strides))
        if rnd.random() < 0.25 and len(shape) > 1:
            i = rnd.randrange(len(shape))
            strides[i] = rnd.choice([0, 1, 2, 3, strides[i] * 2, strides[i] + 1])
        return {"null": rnd.random() < 0.1, "dtype": dtype, "shape": tuple(shape),
                "strides": tuple(strides)}

    def desc_of(m):
        return desc(None if m["null"] else 0x20000, m["dtype"], m["shape"], m["strides"])

    for trial in range(2000):
        nd = rnd.randrange(0, 4)
        shape = tuple(rnd.choice([0, 1, 2, 3, 5]) for _ in range(nd))
        ref_m = {"null": False, "dtype": rnd.choice([0, 1, 2]), "shape": shape, "strides": None}
        strides, acc = [], 1
        for d in reversed(shape):
            strides.append(acc)
            acc *= d
        ref_m["strides"] = tuple(reversed(strides))
        cands = [rand_meta(ref_m) for _ in range(4)]
        rc, st = gate(desc(0x10000, ref_m["dtype"], shape, ref_m["strides"]),
                      [desc_of(m) for m in cands])
        assert rc == kb.KB_OK
        assert list(st) == [oracle.gate_status(ref_m, m) for m in cands], (ref_m, cands)


def test_error_text_belongs_to_the_calling_thread(L):
    """The error text is the only state a call leaves, and it is per thread:
    threads that fail with their own message, interleaved with threads whose
    successful calls clear theirs, each read back exactly their own."""
    from concurrent.futures import ThreadPoolExecutor
    L.kb_last_error.restype = ctypes.c_char_p
    arr = (kb.KbStats * 4)()
    passed = (ctypes.c_int32 * 4)()

    def failing(t):
        dtype = 100 + t
        want = ("unknown dtype %d" % dtype).encode()
        for _ in range(3000):
            rc = L.kb_gen_inputs(None, dtype, ctypes.c_uint64(10), 1, ctypes.c_float(0.0), ctypes.c_float(1.0),
                                 ctypes.c_uint64(0), 0, 0, ctypes.c_uint64(0), None)
            msg = L.kb_last_error()
            if rc != kb.KB_ERR_DTYPE or want not in msg:
                return (t, rc, msg)
        return None

    def succeeding(t):
        for _ in range(3000):
            if L.kb_summarize(arr, 4, None, passed) != kb.KB_OK or L.kb_last_error() not in (b"", None):
                return (t, L.kb_last_error())
        return None

    with ThreadPoolExecutor(8) as ex:
        futs = [ex.submit(failing if t % 2 == 0 else succeeding, t) for t in range(8)]
        bad = [f.result() for f in futs if f.result() is not None]
    assert not bad, bad
