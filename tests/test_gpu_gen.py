"""Parity of the HIP generator with the CPU oracle (GPU).

u32 words and uniform values must be bit-identical; normal values (binary64
Box-Muller on both sides, with different math libraries) within 1e-6
relative, and the count of bit-identical values is reported.  Full-size
streams are checked on sampled indices, which the oracle regenerates one by
one (random access by global index).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
from tests.helpers import ensure_built, storage

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16, "u32": torch.int32}
DIST = {"u32": kb.KB_DIST_U32, "uniform": kb.KB_DIST_UNIFORM, "normal": kb.KB_DIST_NORMAL}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_gen(dev, dt, n, dist, p0, p1, seed, sid, sub, offset):
    out = torch.empty(n, dtype=TORCH_DT[dt], device=dev)
    kb.kb_gen_inputs(out, DIST[dist], p0, p1, seed, sid, sub, offset)
    torch.cuda.synchronize()
    if dt == "u32":
        return out.cpu().numpy().view(np.uint32)
    return storage(out)


CASES = [
    # (n, seed, stream_id, sub, offset)
    (1, 0, 0, 0, 0), (3, 0, 1, 0, 1), (4, 7, 2, 3, 4), (5, 7, 2, 3, 2), (257, 9, 0x0105, 1, 3),
    (4096, 2**40 + 5, 0xFFFF_FFFF, 0xFFFF_FFFF, 2**34 + 1), (65537, 0, 0x0101, 0, 0),
    ((1 << 20) + 6, 123, 0x0300, 17, 12345),
]


@pytest.mark.parametrize("case", CASES)
def test_u32_bit_exact(dev, case):
    n, seed, sid, sub, off = case
    say("u32", case)
    got = gpu_gen(dev, "u32", n, "u32", 0.0, 1.0, seed, sid, sub, off)
    want = oracle.gen("u32", n, oracle.DIST_U32, 0.0, 1.0, seed, sid, sub, off)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("case", CASES)
def test_uniform_bit_exact(dev, dt, case):
    n, seed, sid, sub, off = case
    for a, b in ((-1e-6, 1e-6), (0.0, 1.0), (-3.0, 7.5)):
        say("uniform", dt, case, a, b)
        got = gpu_gen(dev, dt, n, "uniform", a, b, seed, sid, sub, off)
        want = oracle.gen(dt, n, oracle.DIST_UNIFORM, a, b, seed, sid, sub, off)
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8))


@pytest.mark.parametrize("case", CASES)
def test_normal_within_1e6(dev, case):
    n, seed, sid, sub, off = case
    say("normal f32", case)
    for mean, std in ((0.0, 1.0), (0.0, 64.0), (3.0, 0.5)):
        got = gpu_gen(dev, "f32", n, "normal", mean, std, seed, sid, sub, off)
        want = oracle.gen("f32", n, oracle.DIST_NORMAL, mean, std, seed, sid, sub, off)
        diff = np.abs(got.astype(np.float64) - want.astype(np.float64))
        assert np.all(diff <= 1e-6 * np.abs(want.astype(np.float64))), (np.max(diff))
        exact = int(np.sum(got.view(np.uint32) == want.view(np.uint32)))
        say("  bit-identical normals: %d of %d" % (exact, n))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_normal_16bit_rounds_the_same_binary32_value(dev, dt):
    n, seed, sid, sub, off = (1 << 18) + 3, 4, 0x0402, 5, 7
    say("normal", dt)
    g16 = gpu_gen(dev, dt, n, "normal", 0.0, 64.0, seed, sid, sub, off)
    g32 = gpu_gen(dev, "f32", n, "normal", 0.0, 64.0, seed, sid, sub, off)
    o16 = oracle.gen(dt, n, oracle.DIST_NORMAL, 0.0, 64.0, seed, sid, sub, off)
    o32 = oracle.gen("f32", n, oracle.DIST_NORMAL, 0.0, 64.0, seed, sid, sub, off)
    conv = oracle.f32_to_f16_n if dt == "f16" else oracle.f32_to_bf16_n
    # the GPU's 16-bit value is the RNE of its own binary32 value ...
    assert np.array_equal(g16, conv(g32))
    # ... so wherever the binary32 values agree the 16-bit values agree
    same = g32.view(np.uint32) == o32.view(np.uint32)
    assert np.array_equal(g16[same], o16[same])
    assert np.all(np.abs(g16[~same].astype(np.int32) - o16[~same].astype(np.int32)) <= 1)


@pytest.mark.parametrize("dist,dt,n", [("normal", "f32", 1 << 30), ("uniform", "f32", 1 << 30),
                                       ("normal", "bf16", 4096 * 4096), ("u32", "u32", 1 << 28)])
def test_full_size_sampled(dev, dist, dt, n):
    say("full-size stream", dist, dt, n)
    seed, sid, sub = 0, 0x0500, 0
    out = torch.empty(n, dtype=TORCH_DT[dt], device=dev)
    p0, p1 = (0.0, 1.0) if dist != "uniform" else (-1e-7, 1e-7)
    kb.kb_gen_inputs(out, DIST[dist], p0, p1, seed, sid, sub, 0)
    torch.cuda.synchronize()
    rng = np.random.default_rng(99)
    idx = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n),
                                    rng.integers(0, n, size=20000)]))
    sel = out[torch.from_numpy(idx).to(dev)]
    got = sel.cpu().numpy().view(np.uint32) if dt == "u32" else storage(sel)
    want = np.concatenate([oracle.gen(dt, 1, DIST[dist], p0, p1, seed, sid, sub, int(g))
                           for g in idx])
    if dist == "normal" and dt == "f32":
        d = np.abs(got.astype(np.float64) - want.astype(np.float64))
        assert np.all(d <= 1e-6 * np.abs(want.astype(np.float64)))
    elif dist == "normal":
        assert np.all(np.abs(got.astype(np.int32) - want.astype(np.int32)) <= 1)
    else:
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8))
    del out
    torch.cuda.empty_cache()
