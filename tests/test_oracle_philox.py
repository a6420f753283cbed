"""Pins for the oracle's Philox4x32-10 stream (CPU only).

The block function and the stream layout are pinned to an independent
implementation run on the host: rocRAND's Philox4x32-10 engine, compiled
from its installed header at test time (its source shares nothing with the
oracle).  Canonical counters (all zeros, all ones, digits of pi) and random
ones are compared word for word.  The stream layout -- key = seed, counter =
(lo32(b), hi32(b), sub, stream_id), element g = word g mod 4 of block g / 4
-- is rocRAND's (seed, subsequence, offset) addressing with subsequence =
(stream_id << 32) | sub and offset = g.  Structural properties (a bijection
on a counter sweep, balanced bits) pin it further without any stored value.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

# Canonical inputs of the block function: (counter x0..x3, key k0 k1).
CANONICAL = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000)),
    ((0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0)),
]


@pytest.fixture(scope="module")
def rocrand_stream(tmp_path_factory):
    src = os.path.join(HERE, "xcheck", "rocrand_philox_stream.cpp")
    inc = "/opt/rocm/include"
    if not os.path.exists(os.path.join(inc, "rocrand", "rocrand_philox4x32_10.h")):
        pytest.skip("rocRAND headers not installed")
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path_factory.mktemp("xcheck") / "rocrand_philox_stream")
    subprocess.run([cxx, "-O1", "-D__HIP_PLATFORM_AMD__", "-I" + inc, src, "-o", exe],
                   check=True)

    def run(queries):
        text = "".join("%x %x %x %x\n" % q for q in queries)
        out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True)
        return [tuple(int(t, 16) for t in line.split()) for line in out.stdout.splitlines()]

    return run


def test_philox_canonical_counters_match_rocrand(rocrand_stream):
    # rocRAND's engine with key = seed and the counter split across
    # (offset, subsequence) evaluates the block function at any counter.
    queries, got = [], []
    for ctr, key in CANONICAL:
        seed = (key[1] << 32) | key[0]
        subseq = (ctr[3] << 32) | ctr[2]
        queries.append((seed, subseq, ctr[0], ctr[1]))
        got.append(oracle.philox4x32_10(ctr, key))
    assert got == rocrand_stream(queries)


def test_philox_random_counters_and_keys_match_rocrand(rocrand_stream):
    rng = np.random.default_rng(11)
    queries, got = [], []
    for _ in range(300):
        ctr = tuple(int(v) for v in rng.integers(0, 2**32, 4))
        key = tuple(int(v) for v in rng.integers(0, 2**32, 2))
        queries.append(((key[1] << 32) | key[0], (ctr[3] << 32) | ctr[2], ctr[0], ctr[1]))
        got.append(oracle.philox4x32_10(ctr, key))
    assert got == rocrand_stream(queries)


def test_stream_layout_matches_rocrand(rocrand_stream):
    rng = np.random.default_rng(2608)
    cases = []
    for _ in range(400):
        seed = int(rng.integers(0, 2**64, dtype=np.uint64))
        stream_id = int(rng.integers(0, 2**32))
        sub = int(rng.integers(0, 2**32))
        b = int(rng.integers(0, 2**64, dtype=np.uint64))
        cases.append((seed, stream_id, sub, b))
    # edge counters: carries between counter words
    cases += [(0, 0, 0, 0), (0, 7, 3, 2**32 - 1), (1, 0, 0, 2**32), (2**64 - 1, 2**32 - 1, 2**32 - 1, 2**64 - 1)]
    got = [oracle.stream_block(s, sid, sub, b) for s, sid, sub, b in cases]
    queries = [(s, (sid << 32) | sub, b & 0xFFFFFFFF, b >> 32) for s, sid, sub, b in cases]
    assert got == rocrand_stream(queries)


def test_gen_u32_addresses_words_by_global_index():
    seed, sid, sub = 0x1234_5678_9ABC_DEF0, 0x0102, 77
    for offset in (0, 1, 2, 3, 5, 2**33 + 3):
        n = 23
        got = oracle.gen("u32", n, oracle.DIST_U32, seed=seed, stream_id=sid, sub=sub, offset=offset)
        want = []
        for g in range(offset, offset + n):
            want.append(oracle.stream_block(seed, sid, sub, g // 4)[g % 4])
        assert got.tolist() == want


def test_philox_is_a_bijection_on_a_counter_sweep():
    # For a fixed key the block function is a permutation of the counter
    # space: 2^16 consecutive counters give 2^16 distinct outputs and
    # roughly balanced bits.
    key = (0xDEADBEEF, 0x01234567)
    outs = np.array([oracle.philox4x32_10((i, 0, 0, 0), key) for i in range(1 << 16)],
                    dtype=np.uint32)
    packed = outs.view(np.uint64)  # two 64-bit halves per block
    assert len({tuple(r) for r in packed.reshape(-1, 2).tolist()}) == 1 << 16
    bits = np.unpackbits(outs.view(np.uint8))
    assert abs(bits.mean() - 0.5) < 0.002


def test_gen_rejects_bad_dtype_dist_pairs():
    with pytest.raises(ValueError):
        oracle.gen("f32", 4, oracle.DIST_U32)
    with pytest.raises(ValueError):
        oracle.gen("u32", 4, oracle.DIST_NORMAL)
