"""End to end against stored oracle records: the device generator rebuilds the
inputs of tests/golden/screen_golden.json bit for bit (uniform draws,
binary32 additions, round-to-nearest-even narrowing), the library screens
them, and the records must equal the stored ones (counts, flags and maxima
exactly, sums to 1e-6 relative).  The fixture is written by
tests/golden/make_screen_golden.py, which calls only the CPU oracle."""
import json
import os

import numpy as np
import pytest

import paper_2608_02611_amd as kb
from tests.helpers import ensure_built

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "screen_golden.json")))
STREAM_REF, STREAM_NOISE, STREAM_INDEX = 0x501, 0x502, 0x503
N_SPECIAL = 9


def _torch_dtype(torch, name):
    return {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[name]


def _build(torch, dev, dtype):
    seed, n = GOLDEN["seed"], GOLDEN["n"]
    td = _torch_dtype(torch, dtype)
    ref = kb.kb_gen_inputs(torch.empty(n, dtype=td, device=dev), kb.KB_DIST_UNIFORM, -4.0, 4.0,
                           seed=seed, stream_id=STREAM_REF, sub=0)
    r32 = ref.float()
    cands = [ref.clone()]
    for k in range(1, 6):
        s = float(2.0 ** (-22 + 3 * k))
        noise = kb.kb_gen_inputs(torch.empty(n, dtype=torch.float32, device=dev), kb.KB_DIST_UNIFORM,
                                 -s, s, seed=seed, stream_id=STREAM_NOISE, sub=k)
        cands.append((r32 + noise).to(td))
    pos = kb.kb_gen_inputs(torch.empty(N_SPECIAL, dtype=torch.int32, device=dev), kb.KB_DIST_U32,
                           seed=seed, stream_id=STREAM_INDEX, sub=0)
    pos = [int(v) % n for v in pos.cpu().numpy().view(np.uint32)]
    sp = ref.clone()
    vals = [float("nan")] * 3 + [float("inf")] * 3 + [float("-inf")] * 3
    for p, v in zip(pos, vals):
        sp[p] = v
    cands.append(sp)
    return ref, cands


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_records_equal_stored_oracle_records(dtype):
    ensure_built()
    import torch
    dev = torch.device("cuda:0")
    case = GOLDEN["cases"][dtype]
    ref, cands = _build(torch, dev, dtype)
    recs, _ = kb.screen(ref, cands, case["atol"], case["rtol"])
    assert len(recs) == len(case["records"])
    for k, (got, want) in enumerate(zip(recs, case["records"])):
        for f in ("mismatches", "nan_count", "pos_inf_count", "neg_inf_count", "bitwise_equal"):
            assert got[f] == want[f], (dtype, k, f, got[f], want[f])
        assert int(np.float32(got["max_abs_err"]).view(np.uint32)) == want["max_abs_err_bits"], (dtype, k)
        assert int(np.float32(got["max_rel_err"]).view(np.uint32)) == want["max_rel_err_bits"], (dtype, k)
        for f in ("sum_sq_diff", "sum_sq_ref", "rel_l2"):
            w = want[f]
            assert abs(got[f] - w) <= 1e-6 * abs(w) or got[f] == w, (dtype, k, f, got[f], w)
