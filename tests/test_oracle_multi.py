"""Pins of the oracle's multi-output screen and of its policy gate (CPU).

The gate follows the definition of the policy check (Section 3.2: output
shape and dtype against the reference) plus the two checks a view needs to
be read; the hand cases below are read off that definition.  The
multi-output screen must reduce to the single-output one, take the verdict
as the AND over outputs, and report the first failing output's status."""
import numpy as np
import pytest

import oracle


def meta(shape, dtype=0, strides=None, null=False):
    if strides is None:
        strides, acc = [], 1
        for d in reversed(shape):
            strides.append(acc)
            acc *= d
        strides = tuple(reversed(strides))
    return {"null": null, "dtype": dtype, "shape": tuple(shape), "strides": tuple(strides)}


REF = meta((4, 8))


@pytest.mark.parametrize("cand,want", [
    (meta((4, 8)), oracle.STATUS_OK),
    (None, oracle.REJECT_NULL),
    (meta((4, 8), null=True), oracle.REJECT_NULL),
    (meta((4, 8), dtype=1), oracle.REJECT_DTYPE),
    (meta((4, 8), dtype=2, strides=(1, 4)), oracle.REJECT_DTYPE),  # dtype is checked before layout
    (meta((8, 4)), oracle.REJECT_SHAPE),
    (meta((4, 8, 1)), oracle.REJECT_SHAPE),
    (meta((32,)), oracle.REJECT_SHAPE),
    (meta((4, 8), strides=(1, 4)), oracle.REJECT_LAYOUT),      # a transposed view
    (meta((4, 8), strides=(16, 1)), oracle.REJECT_LAYOUT),     # a strided slice
    (meta((4, 8), strides=(8, 2)), oracle.REJECT_LAYOUT),
])
def test_gate_hand_cases(cand, want):
    assert oracle.gate_status(REF, cand) == want


def test_gate_size_one_and_empty():
    # a size-1 dimension's stride is irrelevant; an empty tensor is dense
    assert oracle.gate_status(meta((1, 8)), meta((1, 8), strides=(999, 1))) == oracle.STATUS_OK
    assert oracle.gate_status(meta((4, 1)), meta((4, 1), strides=(1, 77))) == oracle.STATUS_OK
    e = meta((0, 8))
    assert oracle.gate_status(e, meta((0, 8), null=True, strides=(3, 5))) == oracle.STATUS_OK
    assert oracle.gate_status(e, meta((1, 8), null=True)) == oracle.REJECT_NULL


def _out(n, seed, dtype="f32"):
    rng = np.random.default_rng(seed)
    return rng.standard_normal(n).astype(np.float32)


def test_multi_reduces_to_single_and_ands_the_verdict():
    n = 1000
    r0, r1 = _out(n, 1), _out(n, 2)
    refs = [(meta((n,)), r0, "f32"), (meta((n,)), r1, "f32")]
    good0, good1 = r0.copy(), r1.copy()
    bad1 = r1.copy()
    bad1[7] += 1.0
    cands = [[(meta((n,)), good0), (meta((n,)), good1)],
             [(meta((n,)), good0), (meta((n,)), bad1)]]
    recs, passed = oracle.screen_multi(refs, cands, [1e-5, 1e-5], [1e-5, 1e-5])
    assert passed == [1, 0]
    for o, ref in enumerate((r0, r1)):
        for k in range(2):
            single = oracle.screen(ref, cands[k][o][1], "f32", 1e-5, 1e-5)
            assert {f: recs[o][k][f] for f in single} == single
    assert recs[1][1]["mismatches"] == 1 and recs[0][1]["mismatches"] == 0


def test_multi_status_comes_from_the_first_failing_output():
    n = 64
    r0, r1 = _out(n, 3), _out(n, 4)
    refs = [(meta((n,)), r0, "f32"), (meta((n,)), r1, "f32")]
    cands = [
        [(meta((n + 1,)), None), (meta((n,), dtype=1), None)],  # shape in 0, dtype in 1 -> SHAPE
        [(meta((n,)), r0.copy()), (None, None)],                 # output 1 missing -> NULL
        [(meta((n,), dtype=2), None), (meta((n,)), r1.copy())],  # dtype in 0 -> DTYPE
    ]
    recs, passed = oracle.screen_multi(refs, cands, [0.0, 0.0], [0.0, 0.0])
    want = [oracle.REJECT_SHAPE, oracle.REJECT_NULL, oracle.REJECT_DTYPE]
    for k, st in enumerate(want):
        for o in range(2):
            assert recs[o][k]["status"] == st and recs[o][k]["numel"] == 0
    assert passed == [0, 0, 0]
