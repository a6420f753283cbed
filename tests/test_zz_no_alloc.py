"""kb_screen_noalloc, the screening entry point for callers that cannot
allocate (GPU): its records against kb_screen's on the same inputs, on two
calls in a row on the library's shared scratch, the second smaller, and its
argument limits."""
import sys

import pytest
import torch

import paper_2608_02611_amd as kb
from tests.helpers import assert_records_match, ensure_built, oracle_records

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def case(dev, seed, K, n, dtype):
    """A reference and K candidates: copies, in-tolerance noise, and a few
    with mismatches, NaNs and infinities."""
    g = torch.Generator(device=dev).manual_seed(seed)
    ref = torch.randn(n, generator=g, device=dev).to(dtype)
    cands = []
    for k in range(K):
        c = ref.float() * (1 + 2e-4 * torch.randn(n, generator=g, device=dev))
        if k % 5 == 1:
            c[(k * 7919) % n] += 3.0
        if k % 7 == 2:
            c[(k * 104729) % n] = float("nan")
            c[(k * 13) % n] = float("inf")
        cands.append(c.to(dtype) if k % 3 else ref.clone())
    return ref, cands


def noalloc_records(ref, cands, atol, rtol, flags=0):
    st = kb.kb_screen_noalloc(ref, cands, atol, rtol, flags)
    return kb.kb_screen_stats(st, len(cands))


def test_noalloc_matches_kb_screen_twice(dev):
    # first: 40 fp16 candidates of 2^18 + 77 elements (five groups, a
    # two-level finish); second, smaller: 4 fp32 candidates of 5000 elements
    for seed, K, n, dtype, tol in ((1, 40, (1 << 18) + 77, torch.float16, 1e-3),
                                   (2, 4, 5000, torch.float32, 1e-5)):
        ref, cands = case(dev, seed, K, n, dtype)
        say("noalloc", K, n, dtype, kb.kb_screen_launch(K, n, kb.dtype_code(ref)))
        got, gsum = noalloc_records(ref, cands, tol, tol)
        want, wsum = kb.screen(ref, cands, tol, tol)
        assert_records_match(got, want, "noalloc vs kb_screen K=%d" % K)
        assert gsum == wsum
        assert_records_match(got, oracle_records(ref, cands, tol, tol), "noalloc vs oracle K=%d" % K)
        assert 0 < gsum["n_passed"] < K and gsum["n_failed"] > 0, gsum


def test_noalloc_fail_fast_and_limits(dev):
    ref, cands = case(dev, 3, 16, (1 << 20) + 5, torch.bfloat16)
    got, gsum = noalloc_records(ref, cands, 1e-2, 1e-2, kb.KB_FAIL_FAST)
    want, wsum = kb.screen(ref, cands, 1e-2, 1e-2, kb.KB_FAIL_FAST)
    assert [r["passed"] for r in got] == [r["passed"] for r in want]
    assert gsum == wsum
    assert_records_match([r for r in got if r["passed"]], [r for r in want if r["passed"]], "noalloc ff")
    with pytest.raises(kb.KbError) as e:
        kb.kb_screen_noalloc(ref, [ref] * (kb.KB_INLINE_CANDS + 1), 1e-2, 1e-2)
    assert e.value.code == kb.KB_ERR_INVALID_ARG
    # the earlier calls' records are still there: nothing ran for the error
    again, _ = noalloc_records(ref, cands, 1e-2, 1e-2)
    plain, _ = kb.screen(ref, cands, 1e-2, 1e-2)
    assert_records_match(again, plain, "noalloc after an error")
