#!/usr/bin/env python3
"""Writes tests/golden/screen_golden.json: screening records computed by the
CPU oracle (and nothing else) on inputs that both sides can regenerate bit for
bit from the seeded Philox4x32-10 stream.

Every input is a uniform draw (the uniform map is exact, so the library's
generator reproduces it bit-exactly on the device), combined only by
binary32 additions and round-to-nearest-even narrowing, which are
correctly rounded on both sides:
  reference  r   = U(-4, 4) drawn in the tensor's dtype
  candidate  k=0 = r (copy)
  candidate  k   = narrow(widen(r) + U(-s_k, s_k)),  s_k = 2^(-22 + 3k), k = 1..5
  candidate  6   = r with NaN, +inf and -inf written at drawn positions
The sizes are ragged (not multiples of the 512-element chunk).  Run from the
repository root:  python tests/golden/make_screen_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402

SEED = 2026
N = 70001
CASES = {"f32": (1e-5, 1e-5), "f16": (1e-3, 1e-3), "bf16": (1e-2, 1e-2)}
STREAM_REF, STREAM_NOISE, STREAM_INDEX = 0x501, 0x502, 0x503
N_SPECIAL = 9  # positions for NaN, +inf, -inf (three each)


def widen(dtype, a):
    if dtype == "f32":
        return a.astype(np.float32)
    return oracle.f16_to_f32_n(a) if dtype == "f16" else oracle.bf16_to_f32_n(a)


def narrow(dtype, x):
    if dtype == "f32":
        return x.astype(np.float32)
    return oracle.f32_to_f16_n(x) if dtype == "f16" else oracle.f32_to_bf16_n(x)


def special_positions():
    u = oracle.gen("u32", N_SPECIAL, oracle.DIST_U32, seed=SEED, stream_id=STREAM_INDEX, sub=0)
    return [int(v) % N for v in u]


def build(dtype):
    ref = oracle.gen(dtype, N, oracle.DIST_UNIFORM, -4.0, 4.0, seed=SEED, stream_id=STREAM_REF, sub=0)
    r32 = widen(dtype, ref)
    cands = [ref.copy()]
    for k in range(1, 6):
        s = float(2.0 ** (-22 + 3 * k))
        noise = oracle.gen("f32", N, oracle.DIST_UNIFORM, -s, s, seed=SEED, stream_id=STREAM_NOISE, sub=k)
        cands.append(narrow(dtype, (r32 + noise).astype(np.float32)))
    sp = cands[0].copy()
    pos = special_positions()
    vals = narrow(dtype, np.array([np.nan] * 3 + [np.inf] * 3 + [-np.inf] * 3, dtype=np.float32))
    for p, v in zip(pos, vals):
        sp[p] = v
    cands.append(sp)
    return ref, cands


def main():
    out = {"seed": SEED, "n": N, "cases": {}}
    for dtype, (atol, rtol) in CASES.items():
        ref, cands = build(dtype)
        recs = []
        for c in cands:
            s = oracle.screen(ref, c, dtype, atol, rtol)
            recs.append({
                "mismatches": s["mismatches"], "nan_count": s["nan_count"],
                "pos_inf_count": s["pos_inf_count"], "neg_inf_count": s["neg_inf_count"],
                "bitwise_equal": s["bitwise_equal"],
                "max_abs_err_bits": int(np.float32(s["max_abs_err"]).view(np.uint32)),
                "max_rel_err_bits": int(np.float32(s["max_rel_err"]).view(np.uint32)),
                "sum_sq_diff": float(s["sum_sq_diff"]), "sum_sq_ref": float(s["sum_sq_ref"]),
                "rel_l2": float(s["rel_l2"])})
        out["cases"][dtype] = {"atol": atol, "rtol": rtol, "records": recs}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "screen_golden.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
