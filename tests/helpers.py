"""Shared helpers for the GPU parity tests: building, host copies of device
tensors, chunked oracle screening, and record comparison."""
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

EXACT_FIELDS = ("numel", "mismatches", "nan_count", "pos_inf_count", "neg_inf_count",
                "max_abs_err", "max_rel_err", "bitwise_equal", "passed")
SUM_FIELDS = ("sum_sq_diff", "sum_sq_ref", "rel_l2")
SUM_RTOL = 1e-6  # relative tolerance of the binary64 sums and the relative L2 error
THREADS = min(16, os.cpu_count() or 1)


def to_device(arr, dt, dev):
    """numpy storage (float32, or uint16 bits for f16/bf16) -> device tensor of dtype dt."""
    import torch
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(dev)
    bits = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).to(dev)
    return bits.view({"f16": torch.float16, "bf16": torch.bfloat16}[dt])


def oracle_workload(name, dev, seed=0, scale=1.0, K=None):
    """Workload `name` built by the oracle on the host (oracle.workloads) and
    copied to device `dev`: the inputs of the screening parity tests, none of
    whose bytes come from the HIP path.  Returns (synth.Workload of device
    tensors, the oracle's host workload)."""
    import synth
    from oracle import workloads
    ow = workloads.build(name, seed=seed, scale=scale, K=K)
    ref = to_device(ow.ref, ow.dtype, dev).view(ow.shape)
    cands = [to_device(c, ow.dtype, dev).view(ow.shape) for c in ow.cands]
    return synth.Workload(name, ref, cands, ow.atol, ow.rtol, dict(ow.meta)), ow


def ensure_built():
    import __graft_entry__
    __graft_entry__._ensure_built()


def dtype_name(t):
    import torch
    return {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[t.dtype]


def storage(t):
    """Host numpy array of the raw storage of a (device) tensor."""
    import torch
    t = t.detach().contiguous().view(-1)
    if t.dtype == torch.float32:
        return t.cpu().numpy()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def oracle_records(ref, cands, atol, rtol, flags=0, chunk=1 << 24, dt=None):
    """Oracle statistics of every candidate (chunked over elements and run on
    host threads for large tensors; merged in chunk order).  ref and cands
    are device tensors, or host storage arrays with their dtype name dt."""
    host = isinstance(ref, np.ndarray)
    if host:
        n = ref.size
        get = lambda t, lo, hi: t.reshape(-1)[lo:hi]
    else:
        dt = dtype_name(ref)
        n = ref.numel()
        get = lambda t, lo, hi: storage(t.reshape(-1)[lo:hi])
    if n <= chunk:
        r = get(ref, 0, n)
        return [oracle.screen(r, get(c, 0, n), dt, atol, rtol, flags) for c in cands]
    bounds = [(lo, min(n, lo + chunk)) for lo in range(0, n, chunk)]
    partials = [[None] * len(bounds) for _ in cands]
    with ThreadPoolExecutor(THREADS) as ex:
        for bi, (lo, hi) in enumerate(bounds):
            r = get(ref, lo, hi)
            cs = [get(c, lo, hi) for c in cands]
            futs = [ex.submit(oracle.screen_partial, r, cs[k], dt, atol, rtol, flags)
                    for k in range(len(cands))]
            for k, f in enumerate(futs):
                partials[k][bi] = f.result()
    return [oracle.finalize(oracle.merge(p)) for p in partials]


def oracle_positions_host(ref, cands, dt, atol, rtol, records, flags=0):
    """The oracle's positions (kbo_locate) of every candidate, on host
    storage arrays, with the maxima of the oracle's own records; one host
    thread per candidate."""
    def one(k):
        fm, ai, ri = oracle.locate(ref, cands[k], dt, atol, rtol, records[k]["max_abs_err"],
                                   records[k]["max_rel_err"], flags)
        return {"first_mismatch": fm, "max_abs_index": ai, "max_rel_index": ri}
    with ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(one, range(len(cands))))


def close(a, b, rtol=SUM_RTOL):
    if math.isnan(a) or math.isnan(b):
        return math.isnan(a) and math.isnan(b)
    if math.isinf(a) or math.isinf(b):
        return a == b
    return abs(a - b) <= rtol * abs(b)


def assert_records_match(gpu, orc, label=""):
    assert len(gpu) == len(orc)
    bad = []
    for k, (g, o) in enumerate(zip(gpu, orc)):
        assert g["status"] == 0, (label, k, g)
        for f in EXACT_FIELDS:
            if g[f] != o[f] and not (isinstance(o[f], float) and math.isnan(o[f]) and math.isnan(g[f])):
                bad.append((k, f, g[f], o[f]))
        for f in SUM_FIELDS:
            if not close(g[f], o[f]):
                bad.append((k, f, g[f], o[f]))
    assert not bad, "%s: %d mismatching fields, first %s" % (label, len(bad), bad[:8])


def same_record(a, b):
    """A passing candidate's fail-fast record against its plain record:
    counts, flags and maxima identical, the sums within SUM_RTOL."""
    for f in a:
        if f in SUM_FIELDS:
            if not close(a[f], b[f]):
                return False
        elif a[f] != b[f]:
            return False
    return True


def check_partial(g, o, label):
    """A fail-fast record of a failing candidate against the oracle's record
    over the whole tensor."""
    assert g["status"] == 0, (label, g)
    assert o["mismatches"] > 0, (label, o)
    assert 1 <= g["mismatches"] <= o["mismatches"], (label, g, o)
    assert g["passed"] == 0, (label, g)
    assert 0 < g["numel"] <= o["numel"], (label, g, o)
    assert g["mismatches"] <= g["numel"], (label, g)
    for f in ("nan_count", "pos_inf_count", "neg_inf_count"):
        assert g[f] <= o[f], (label, f, g, o)
    for f in ("max_abs_err", "max_rel_err"):
        assert g[f] <= o[f] or o[f] != o[f], (label, f, g, o)
    for f in ("sum_sq_diff", "sum_sq_ref"):
        assert g[f] <= o[f] * (1 + SUM_RTOL), (label, f, g, o)
    if g["numel"] == o["numel"]:
        # nothing was skipped: the whole record
        assert_records_match([g], [o], label)
