"""Pins for the oracle's Philox4x32-10 stream (CPU only).

The block function is pinned to the published known-answer vectors
(tests/golden/philox4x32_10_kat.txt) and to an independent implementation run
on the host (rocRAND's engine, compiled from its header at test time).  The
stream layout -- key = seed, counter = (lo32(b), hi32(b), sub, stream_id),
element g = word g mod 4 of block g / 4 -- is pinned by the same rocRAND
engine, whose (seed, subsequence, offset) addressing is that layout when
subsequence = (stream_id << 32) | sub and offset = g.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


@pytest.mark.parametrize("ctr,key,want", _kat_rows())
def test_philox_known_answer_vectors(ctr, key, want):
    assert oracle.philox4x32_10(ctr, key) == want


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


def test_philox_kat_through_rocrand(rocrand_stream):
    # rocRAND reproduces the known-answer vectors with key = seed and the
    # counter split across (offset, subsequence): both oracles agree on them.
    queries, wants = [], []
    for ctr, key, want in _kat_rows():
        seed = (key[1] << 32) | key[0]
        subseq = (ctr[3] << 32) | ctr[2]
        queries.append((seed, subseq, ctr[0], ctr[1]))
        wants.append(want)
    assert rocrand_stream(queries) == wants


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
