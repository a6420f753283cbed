"""Parity of the library's derived seeded inputs with the oracle (GPU):
Student-t values, softmax rows, index draws, planted changes, scatters, and
the five screening workloads built from them.

The bar: bit-exact where only uniform words enter (index draws, masks,
uniform noise, flips, scatters, the planted specials); where binary64
normals enter (Box-Muller, Student-t, softmax), within 1e-6 relative of the
oracle in binary32 -- the device's log/sin/cos/exp and the host's may differ
in the last binary64 place, which very rarely moves a binary32 rounding --
and then at most one unit of the storage type's last place apart after a
16-bit rounding, with nearly every element bit-identical (the count is
printed).  Inputs of the changes come from the oracle (host arrays copied to
the device), never from the library."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
import synth
from oracle import workloads
from tests.helpers import ensure_built, storage, to_device

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
CODE = {"f32": kb.KB_F32, "f16": kb.KB_F16, "bf16": kb.KB_BF16}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def widen(bits, dt):
    if dt == "f32":
        return bits.view(np.float32).astype(np.float64)
    if dt == "f16":
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def ordinal(bits, dt):
    """Storage bits -> integers in value order (adjacent values differ by 1)."""
    if dt == "f32":
        u = bits.view(np.uint32).astype(np.int64)
        sign, mag = u >> 31, u & 0x7FFFFFFF
    else:
        u = bits.view(np.uint16).astype(np.int64)
        sign, mag = u >> 15, u & 0x7FFF
    return np.where(sign == 1, -mag, mag)


def assert_normals_close(got, want, dt, label, min_identical=0.999):
    """got, want: storage arrays of dtype dt computed from binary64 normals.
    Identical, or (binary32) within 1e-6 relative, or (16-bit) one unit in
    the last place apart; NaN where NaN; nearly all identical."""
    got = np.ascontiguousarray(got).reshape(-1)
    want = np.ascontiguousarray(want).reshape(-1)
    assert got.shape == want.shape, label
    gb = got.view(np.uint32 if dt == "f32" else np.uint16)
    wb = want.view(np.uint32 if dt == "f32" else np.uint16)
    same = gb == wb
    diff = ~same
    n_diff = int(diff.sum())
    if n_diff:
        g, w = widen(gb[diff], dt), widen(wb[diff], dt)
        assert not np.isnan(g).any() and not np.isnan(w).any(), (label, "NaN differs")
        if dt == "f32":
            bad = np.abs(g - w) > 1e-6 * np.abs(w)
        else:
            bad = np.abs(ordinal(gb[diff], dt) - ordinal(wb[diff], dt)) > 1
        assert not bad.any(), (label, g[bad][:5], w[bad][:5])
    say("  %s: %d of %d elements bit-identical" % (label, got.size - n_diff, got.size))
    assert got.size - n_diff >= min_identical * got.size, (label, n_diff)


def host(t):
    return storage(t)


# ------------------------------------------------------------- Student-t ---

@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n,offset", [(1, 0), (1000, 3), (65537, 0), ((1 << 20) + 5, (1 << 33) + 7)])
def test_student_t(dev, dt, n, offset):
    out = torch.empty(n, dtype=TORCH_DT[dt], device=dev)
    kb.kb_gen_inputs(out, kb.KB_DIST_STUDENT_T3, 0.0, 1.0, seed=0, stream_id=(5 << 8), sub=0, offset=offset)
    want = oracle.gen(dt, n, oracle.DIST_STUDENT_T3, 0.0, 1.0, seed=0, stream_id=(5 << 8), sub=0, offset=offset)
    assert_normals_close(host(out), want, dt, "t3 %s n=%d off=%d" % (dt, n, offset))
    # location and scale
    kb.kb_gen_inputs(out, kb.KB_DIST_STUDENT_T3, -2.0, 0.5, seed=7, stream_id=11, sub=3, offset=offset)
    want = oracle.gen(dt, n, oracle.DIST_STUDENT_T3, -2.0, 0.5, seed=7, stream_id=11, sub=3, offset=offset)
    assert_normals_close(host(out), want, dt, "t3 loc/scale %s n=%d" % (dt, n))


def test_student_t_sampled_at_full_size(dev):
    """The five-gigabyte workload's 2^30 Student-t values, sampled: the
    oracle computes any element on its own (random access)."""
    n = 1 << 30
    out = torch.empty(n, dtype=torch.float32, device=dev)
    kb.kb_gen_inputs(out, kb.KB_DIST_STUDENT_T3, 0.0, 1.0, seed=0, stream_id=(5 << 8), sub=0)
    rng = np.random.default_rng(5)
    starts = np.concatenate([[0, n - 4096], rng.integers(0, n - 4096, 30)])
    for s in starts:
        got = host(out[int(s):int(s) + 4096])
        want = oracle.gen("f32", 4096, oracle.DIST_STUDENT_T3, 0.0, 1.0, seed=0, stream_id=(5 << 8), sub=0,
                          offset=int(s))
        assert_normals_close(got, want, "f32", "t3 full-size @%d" % s)
    del out
    torch.cuda.empty_cache()


# --------------------------------------------------------------- softmax ---

@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 5), (7, 1000), (256, 1024), (2, 4097), (70000, 3)])
def test_softmax_rows(dev, rows, cols):
    out = torch.empty(rows, cols, dtype=torch.float32, device=dev)
    kb.kb_gen_softmax_rows(out, 2.0, seed=0, stream_id=(3 << 8), sub=0)
    got = host(out).reshape(rows, cols)
    want = oracle.gen_softmax_rows(rows, cols, 2.0, seed=0, stream_id=(3 << 8), sub=0)
    assert_normals_close(got, want, "f32", "softmax %dx%d" % (rows, cols), min_identical=0.99)
    assert np.all(got > 0)
    assert np.max(np.abs(got.astype(np.float64).sum(axis=1) - 1.0)) <= max(1, cols) * 2.0 ** -24
    # the same bits on every call (a fixed summation tree)
    again = torch.empty_like(out)
    kb.kb_gen_softmax_rows(again, 2.0, seed=0, stream_id=(3 << 8), sub=0)
    assert torch.equal(again.view(torch.int32), out.view(torch.int32))


# ----------------------------------------------------------- index draws ---

@pytest.mark.parametrize("m,n,stream_id,sub", [(5, 65536, (1 << 8) | 3, 2), (64, 8 * 2048 * 4096, (4 << 8) | 3, 6),
                                               (1, 2, 9, 0), (100, 200, 9, 1), (kb.KB_MAX_INDICES, 1 << 40, 5, 5),
                                               (kb.KB_MAX_INDICES, 2 * kb.KB_MAX_INDICES, 77, 3)])
def test_index_draws_exact(dev, m, n, stream_id, sub):
    got = kb.kb_gen_indices(m, n, dev, seed=0, stream_id=stream_id, sub=sub).cpu().numpy().astype(np.uint64)
    want = oracle.gen_indices(m, n, seed=0, stream_id=stream_id, sub=sub)
    assert np.array_equal(got, want), (m, n)


def test_index_draw_limits(dev):
    for m, n in ((0, 10), (kb.KB_MAX_INDICES + 1, 1 << 40), (6, 11)):
        with pytest.raises(kb.KbError):
            kb.kb_gen_indices(m, n, dev)


# ------------------------------------------------------- planted changes ---

def _src(dt, n, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(n) * np.exp(rng.uniform(-4, 4, n))).astype(np.float32)
    x[:: 101] = 0.0
    x[1:: 211] = -0.0
    x[2:: 307] = np.float32(2.0 ** -140)
    x[3:: 401] = -np.float32(2.0 ** -130)
    x[4:: 997] = np.inf
    if dt == "f32":
        return x
    return oracle.f32_to_f16_n(x) if dt == "f16" else oracle.f32_to_bf16_n(x)


EXACT_OPS = [(kb.KB_PERTURB_ADD_UNIFORM, -1e-3, 2e-3, 0.0), (kb.KB_PERTURB_REL_UNIFORM, -2.0 ** -6, 2.0 ** -6, 0.0),
             (kb.KB_PERTURB_SCALE_WHERE, 1.01, 0.0, 0.01), (kb.KB_PERTURB_FLIP_LSB_WHERE, 0.0, 0.0, 0.001),
             (kb.KB_PERTURB_FLIP_LSB_WHERE, 0.0, 0.0, 1.0), (kb.KB_PERTURB_SCALE_WHERE, 0.5, 0.0, 1.0)]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n,offset", [(1, 0), (4099, 13), ((1 << 20) + 3, (1 << 32) + 1)])
def test_perturb_uniform_ops_exact(dev, dt, n, offset):
    """Changes driven by uniform words only: bit-exact, in place too."""
    src = _src(dt, n, n)
    d_src = to_device(src, dt, dev)
    bits = (lambda a: a.view(np.uint32)) if dt == "f32" else (lambda a: a)
    for op, a, b, p in EXACT_OPS:
        want = oracle.perturb(src, dt, op, a, b, p, seed=3, stream_id=41, sub=2, offset=offset)
        out = torch.empty_like(d_src)
        kb.kb_gen_perturb(out, d_src, op, a, b, p, seed=3, stream_id=41, sub=2, offset=offset)
        got = bits(host(out))
        bad = np.nonzero(got != bits(want))[0]
        assert bad.size == 0, (dt, op, n, offset, bad.size, [(int(i), hex(int(bits(src)[i])), hex(int(got[i])),
                                                              hex(int(bits(want)[i]))) for i in bad[:6]])
        inplace = d_src.clone()
        kb.kb_gen_perturb(inplace, inplace, op, a, b, p, seed=3, stream_id=41, sub=2, offset=offset)
        assert torch.equal(inplace.view(torch.int16 if dt != "f32" else torch.int32),
                           out.view(torch.int16 if dt != "f32" else torch.int32))


@pytest.mark.parametrize("n,offset", [(1, 0), (5000, 7), ((1 << 20) + 1, (1 << 31) - 3)])
def test_perturb_block_ops_exact(dev, n, offset):
    """The planted specials and the zero/subnormal/relative changes (whole
    blocks of words per element, binary32): bit-exact."""
    src = _src("f32", n, n + 1)
    d_src = to_device(src, "f32", dev)
    for op, a, b, p in ((kb.KB_PERTURB_SPECIALS, 2.0 ** -10, 2.0 ** -9, 2.0 ** -9 + 2.0 ** -20),
                        (kb.KB_PERTURB_SPECIALS, 0.3, 0.6, 0.9),
                        (kb.KB_PERTURB_ZERO_SUBNORMAL_REL, -1e-7, 1e-7, 0.5),
                        (kb.KB_PERTURB_ZERO_SUBNORMAL_REL, -0.25, 0.5, 1.0)):
        want = oracle.perturb(src, "f32", op, a, b, p, seed=0, stream_id=(5 << 8) | 1, sub=4, offset=offset)
        out = torch.empty_like(d_src)
        kb.kb_gen_perturb(out, d_src, op, a, b, p, seed=0, stream_id=(5 << 8) | 1, sub=4, offset=offset)
        assert np.array_equal(host(out).view(np.uint32), want.view(np.uint32)), (op, n, offset)
    with pytest.raises(kb.KbError):
        h = torch.zeros(8, dtype=torch.float16, device=dev)
        kb.kb_gen_perturb(h, h, kb.KB_PERTURB_SPECIALS, 0.1, 0.2, 0.3)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_perturb_add_normal(dev, dt):
    n = (1 << 18) + 9
    src = _src(dt, n, 3)
    d_src = to_device(src, dt, dev)
    out = torch.empty_like(d_src)
    kb.kb_gen_perturb(out, d_src, kb.KB_PERTURB_ADD_NORMAL, 1e-3, 0.0, 0.0, seed=0, stream_id=(3 << 8) | 1,
                      sub=9, offset=5)
    want = oracle.perturb(src, dt, oracle.PERTURB_ADD_NORMAL, 1e-3, 0.0, 0.0, seed=0, stream_id=(3 << 8) | 1,
                          sub=9, offset=5)
    assert_normals_close(host(out), want, dt, "add normal %s" % dt)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_scatter(dev, dt):
    n = 70001
    src = _src(dt, n, 4)
    d_ref = to_device(src, dt, dev)
    idx = kb.kb_gen_indices(64, n, dev, seed=0, stream_id=(4 << 8) | 3, sub=2)
    h_idx = oracle.gen_indices(64, n, seed=0, stream_id=(4 << 8) | 3, sub=2)
    for mode in (kb.KB_SCATTER_NAN, kb.KB_SCATTER_INF_SIGN_OF_REF):
        out = d_ref.clone()
        kb.kb_gen_scatter(out, d_ref, idx, mode)
        want = src.copy()
        oracle.scatter(want, src, dt, h_idx, mode)
        assert np.array_equal(host(out).view(np.uint32 if dt == "f32" else np.uint16),
                              want.view(np.uint32 if dt == "f32" else np.uint16)), (dt, mode)


# -------------------------------------------------------- the workloads ---

def compare_workloads(gw, ow, label):
    """A workload built on the GPU by the library against the oracle's."""
    assert gw.meta == ow.meta, (label, gw.meta, ow.meta)  # index sets and tiles: exact
    assert_normals_close(host(gw.ref), ow.ref, ow.dtype, label + " ref")
    for k, (g, o) in enumerate(zip(gw.cands, ow.cands)):
        # each candidate is derived from the reference of its own side, so it
        # differs only where the two references differ
        assert_normals_close(host(g), o, ow.dtype, label + " cand %d" % k)


@pytest.mark.parametrize("name,scale,K", [("c1", 1.0, None), ("c2", 1 / 64, None), ("c3", 1.0, 64),
                                          ("c4", 1 / 256, 16), ("c5", 1 / 256, None)])
def test_workloads_scaled_built_alike(dev, name, scale, K):
    say("workload built alike", name, scale, K)
    gw = synth.build(name, dev, seed=0, scale=scale, K=K)
    ow = workloads.build(name, seed=0, scale=scale, K=K)
    compare_workloads(gw, ow, name)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workloads_full_size_built_alike(dev, name):
    """The exact workloads the benchmark screens, built by the library,
    against the oracle's, tensor by tensor over every element."""
    say("full-size workload built alike", name)
    gw = synth.build(name, dev, seed=0)
    torch.cuda.synchronize()
    ow = workloads.build(name, seed=0)
    compare_workloads(gw, ow, name + " full")
    del gw, ow
    torch.cuda.empty_cache()
