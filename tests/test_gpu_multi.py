"""Multi-output candidates (kb_screen_multi) against the oracle (GPU).

Candidates return a tuple of tensors -- here an attention-style pair (the
output in bf16 and the log-sum-exp in fp32) and a third fp16 tensor.  One
gate covers all outputs; accepted candidates get one record per output,
rejected ones the first failing status in every record."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_02611_amd as kb
from tests.helpers import assert_records_match, ensure_built, storage, dtype_name

pytestmark = pytest.mark.gpu

CODES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def meta(t):
    if t is None:
        return None
    return {"null": t.numel() == 0 and t.data_ptr() == 0, "dtype": CODES.get(t.dtype, 3),
            "shape": tuple(t.shape), "strides": tuple(t.stride())}


def oracle_side(refs, cands, atol, rtol, flags):
    o_refs = [(meta(r), storage(r), dtype_name(r)) for r in refs]
    o_cands = []
    for row in cands:
        o_row = []
        for o, c in enumerate(row):
            ok = c is not None and oracle.gate_status(o_refs[o][0], meta(c)) == oracle.STATUS_OK
            o_row.append((meta(c), storage(c) if ok else None))
        o_cands.append(o_row)
    return oracle.screen_multi(o_refs, o_cands, atol, rtol, flags)


def compare(refs, cands, atol, rtol, flags=0, label=""):
    g_recs, g_summ, g_passed = kb.screen_multi(refs, cands, atol, rtol, flags)
    o_recs, o_passed = oracle_side(refs, cands, atol, rtol, flags & kb.KB_EQUAL_NAN)
    assert g_passed == o_passed, (label, g_passed, o_passed)
    for o in range(len(refs)):
        for k in range(len(cands)):
            g, w = g_recs[o][k], o_recs[o][k]
            assert g["status"] == w["status"], (label, o, k, g, w)
            if w["status"] != 0:
                assert g["numel"] == 0 and g["mismatches"] == 0 and g["passed"] == 0, (label, o, k, g)
            elif not (flags & kb.KB_FAIL_FAST) or w["mismatches"] == 0:
                assert_records_match([g], [w], "%s out %d cand %d" % (label, o, k))
    assert g_summ["n_passed"] == sum(o_passed)
    return g_recs, g_summ, g_passed


def attention_like(dev, B=2, H=4, S=256, D=64, seed=0):
    g = torch.Generator(device=dev).manual_seed(seed)
    out = torch.randn(B, H, S, D, generator=g, device=dev).to(torch.bfloat16)
    lse = torch.randn(B, H, S, generator=g, device=dev) * 3.0 + 10.0
    aux = torch.randn(S, 37, generator=g, device=dev).half()
    return [out, lse, aux]


def perturb(t, scale, seed):
    g = torch.Generator(device=t.device).manual_seed(seed)
    return (t.float() * (1 + scale * torch.randn(t.shape, generator=g, device=t.device))).to(t.dtype)


def test_gate_and_verdicts(dev):
    refs = attention_like(dev)
    out, lse, aux = refs
    atol, rtol = [1e-2, 1e-4, 1e-3], [1e-2, 1e-4, 1e-3]
    wrong_lse = lse.clone()
    wrong_lse[1, 2, 100] += 1.0
    cands = [
        [perturb(out, 1e-3, 1), lse.clone(), aux.clone()],              # pass
        [out.clone(), wrong_lse, aux.clone()],                          # fail in lse only
        [out.clone(), lse[:, :, :255].clone(), aux.clone()],            # shape (output 1)
        [out.half(), lse.clone(), aux.clone()],                         # dtype (output 0)
        [out.transpose(2, 3).contiguous().transpose(2, 3), lse.clone(), aux.clone()],  # layout
        [out.clone(), None, aux.clone()],                               # missing output
        [perturb(out, 0.5, 2), perturb(lse, 1e-2, 3), perturb(aux, 0.1, 4)],  # fail everywhere
        [out.clone(), lse.clone(), aux.clone()],                        # bit-identical
        [out.clone(), lse.clone(), aux.t().contiguous().t()],           # layout in the last output
        [out.half(), lse[:, :, :255].clone(), aux.clone()],             # dtype (0), then shape (1)
        [out.clone(), None, aux.t().contiguous().t()],                  # missing (1), then layout (2)
    ]
    recs, summ, passed = compare(refs, cands, atol, rtol, 0, "gate")
    assert passed == [1, 0, 0, 0, 0, 0, 0, 1, 0, 0, 0]
    assert [recs[0][k]["status"] for k in range(11)] == [0, 0, 3, 2, 4, 1, 0, 0, 4, 2, 1]
    # a candidate that fails the gate on several outputs carries the first
    # failing check, in output order, in every output's record
    assert [recs[o][9]["status"] for o in range(3)] == [2, 2, 2]
    assert [recs[o][10]["status"] for o in range(3)] == [1, 1, 1]
    assert summ["n_rejected"] == 7 and summ["n_failed"] == 2 and summ["n_passed"] == 2
    assert recs[1][1]["mismatches"] == 1 and recs[0][1]["mismatches"] == 0
    assert recs[2][7]["bitwise_equal"] == 1


@pytest.mark.parametrize("flags", [0, kb.KB_EQUAL_NAN, kb.KB_FAIL_FAST])
def test_many_candidates(dev, flags):
    """200 candidates (the launch table is uploaded), random mixes of
    passing, failing and gated outputs."""
    refs = attention_like(dev, S=512, seed=5)
    atol, rtol = [1e-2, 1e-4, 1e-3], [1e-2, 1e-4, 1e-3]
    rng = np.random.default_rng(11)
    cands = []
    for k in range(200):
        row = []
        for o, r in enumerate(refs):
            u = rng.uniform()
            if u < 0.03:
                row.append(None)
            elif u < 0.06:
                row.append(r.reshape(-1)[:-1].clone())
            elif u < 0.3:
                row.append(perturb(r, [0.05, 1e-3, 0.01][o], 1000 * k + o))
            else:
                row.append(perturb(r, [1e-3, 1e-6, 1e-4][o], 1000 * k + o) if u < 0.6 else r.clone())
        cands.append(row)
    say("multi 200 flags", flags)
    compare(refs, cands, atol, rtol, flags, "many flags=%d" % flags)


def test_attention_pair_full_size(dev):
    """The output pair the benchmark screens, at its size: out fp16
    [4, 32, 2048, 128] and lse fp32 [4, 32, 2048], 16 candidates with
    in-tolerance noise, two of them wrong in one output.  Every record
    against the oracle's (host threads over chunks of the outputs)."""
    from tests.helpers import oracle_records
    g = torch.Generator(device=dev).manual_seed(3)
    out = torch.randn(4, 32, 2048, 128, generator=g, device=dev).to(torch.float16)
    lse = torch.randn(4, 32, 2048, generator=g, device=dev) + 8.0
    refs = [out, lse]
    atol, rtol = [1e-2, 1e-4], [1e-2, 1e-4]
    cands = []
    for k in range(16):
        gk = torch.Generator(device=dev).manual_seed(100 + k)
        o = (out.float() * (1 + 1e-3 * torch.randn(out.shape, generator=gk, device=dev))).to(torch.float16)
        l = lse + 1e-6 * torch.randn(lse.shape, generator=gk, device=dev)
        cands.append([o, l])
    cands[3][1][1, 7, 1000] += 1.0
    cands[9][0][2, 3, 17, 5] = float("nan")
    say("attention pair full size")
    g_recs, g_summ, g_passed = kb.screen_multi(refs, cands, atol, rtol, 0)
    for o in range(2):
        want = oracle_records(refs[o], [c[o] for c in cands], atol[o], rtol[o], 0)
        assert_records_match(g_recs[o], want, "attention pair output %d" % o)
    assert g_passed == [int(k not in (3, 9)) for k in range(16)], g_passed
    assert g_summ["n_passed"] == 14


def test_single_output_equals_kb_screen(dev):
    ref = torch.randn(70001, device=dev)
    cands = [ref + 1e-6 * torch.randn(70001, device=dev) for _ in range(5)]
    cands[3][500] += 1.0
    recs, _, passed = kb.screen_multi([ref], [[c] for c in cands], 1e-5, 1e-5)
    plain, _ = kb.screen(ref, cands, 1e-5, 1e-5)
    assert recs[0] == plain
    assert passed == [1, 1, 1, 0, 1]


def test_multiscreener_repeated_launches(dev):
    """The pre-marshalled MultiScreener: every launch gives the records of
    kb_screen_multi on the same arguments, call after call on one
    workspace."""
    refs = attention_like(dev, seed=9)
    out, lse, aux = refs
    atol, rtol = [1e-2, 1e-4, 1e-3], [1e-2, 1e-4, 1e-3]
    cands = [[perturb(out, 1e-3, 21), lse.clone(), aux.clone()],
             [out.clone(), perturb(lse, 1e-2, 22), aux.clone()],
             [out.clone(), lse[:, :, :255].clone(), aux.clone()],
             [perturb(out, 0.5, 23), perturb(lse, 1e-6, 24), perturb(aux, 1e-4, 25)]]
    want, _, _ = kb.screen_multi(refs, cands, atol, rtol)
    ms = kb.MultiScreener(refs, cands, atol, rtol)
    for rep in range(3):
        ms.launch()
        got = ms.records()
        assert [got[o * 4:(o + 1) * 4] for o in range(3)] == want, rep


def test_argument_errors(dev):
    refs = attention_like(dev)
    cands = [[r.clone() for r in refs]]
    with pytest.raises(kb.KbError):
        kb.screen_multi(refs, cands, [1e-3, 1e-3], [1e-3, -1.0, 1e-3])
    with pytest.raises(kb.KbError):
        kb.screen_multi(refs, cands, 1e-3, 1e-3, flags=8)
    R = (kb.KbTensor * 3)(*[kb.describe(r) for r in refs])
    assert kb.lib().kb_screen_multi_workspace_bytes(R, 0, 1) == 0
    assert kb.lib().kb_screen_multi_workspace_bytes(R, 3, 0) == 0
    assert kb.lib().kb_screen_multi_workspace_bytes(R, 3, 1) > 0
