"""The screening workloads built on the CPU by the oracle, from synth's recipes.

TEST INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's
CPU-baseline leg).  synth.build carries out the same recipes on the GPU
through the library; here every step is the oracle's own function
(kbo_gen, kbo_gen_softmax_rows, kbo_gen_indices, kbo_perturb, kbo_scatter),
run over element chunks on host threads (the functions are per element and
take the chunk's offset, so the chunking changes nothing).  The result is
raw storage: float32 arrays for f32, uint16 bit patterns for f16 and bf16.
"""
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

import synth

from . import DIST_U32, NP_STORAGE, DTYPES, gen, gen_indices, gen_softmax_rows, perturb, scatter

CHUNK = 1 << 20  # elements per task
THREADS = min(16, os.cpu_count() or 1)


@dataclass
class OracleWorkload:
    name: str
    dtype: str
    shape: tuple
    ref: np.ndarray
    cands: list
    atol: float
    rtol: float
    meta: dict = field(default_factory=dict)

    @property
    def numel(self):
        return self.ref.size


def _bounds(n, chunk=CHUNK):
    return [(lo, min(n, lo + chunk)) for lo in range(0, n, chunk)]


def _run(ex, steps, arr, ref, rec, meta):
    """Carry out `steps` on the flat storage array `arr`, the first arr.size
    elements of the tensor (ref: the finished reference, as long)."""
    n, dt, full = arr.size, rec.dtype, rec.numel
    for st in steps:
        a = st.args
        if st.kind == "gen":
            def one(b):
                lo, hi = b
                arr[lo:hi] = gen(dt, hi - lo, a["dist"], a["p0"], a["p1"], rec.seed, st.stream_id, st.sub, lo)
            list(ex.map(one, _bounds(n)))
        elif st.kind == "softmax":
            cols = full // rec.shape[0]
            rows = n // cols
            view = arr.reshape(rows, cols)

            def one(b):
                r0, r1 = b
                view[r0:r1] = gen_softmax_rows(r1 - r0, cols, a["sigma"], rec.seed, st.stream_id, st.sub, r0)
            list(ex.map(one, _bounds(rows, max(1, CHUNK // cols))))
        elif st.kind == "perturb":
            def one(b):
                lo, hi = b
                arr[lo:hi] = perturb(arr[lo:hi], dt, a["op"], a["a"], a["b"], a["p"], rec.seed, st.stream_id,
                                     st.sub, lo)
            list(ex.map(one, _bounds(n)))
        elif st.kind == "scatter":
            # drawn over the whole tensor; indices past a prefix are skipped
            idx = gen_indices(a["m"], full, rec.seed, st.stream_id, st.sub)
            scatter(arr, ref, dt, idx, a["mode"])
            meta.setdefault("indices", {})[st.sub] = [int(i) for i in idx]
        elif st.kind == "tile":
            rows, cols = rec.shape
            w = gen("u32", 2, DIST_U32, 0.0, 1.0, rec.seed, st.stream_id, st.sub, 0)
            tr, tc = int(w[0]) % (rows // 64), int(w[1]) % (cols // 64)
            arr.reshape(-1, cols)[64 * tr:64 * tr + 64, 64 * tc:64 * tc + 64] = 0
            meta.setdefault("tiles", {})[st.sub] = (tr, tc)
        else:
            raise ValueError(st.kind)


def build(name, seed=0, scale=1.0, K=None, threads=THREADS, prefix=None):
    """Workload `name` as host storage arrays, built by the oracle.  With
    `prefix`, only the first `prefix` elements of every tensor (whole rows
    for row-shaped tensors): every step is per element (or per row) and
    random-access, so a prefix is exactly the start of the full tensors."""
    rec = synth.recipe(name, seed=seed, scale=scale, K=K)
    meta = {}
    store = NP_STORAGE[DTYPES[rec.dtype]]
    n = rec.numel if prefix is None else min(int(prefix), rec.numel)
    if len(rec.shape) > 1:
        row = rec.numel // rec.shape[0]
        n = max(row, n // row * row)
    with ThreadPoolExecutor(threads) as ex:
        ref = np.empty(n, dtype=store)
        _run(ex, rec.ref, ref, ref, rec, meta)
        cands = []
        for steps in rec.cands:
            c = ref.copy()
            _run(ex, steps, c, ref, rec, meta)
            cands.append(c)
    shape = rec.shape if n == rec.numel else (n,)
    return OracleWorkload(name, rec.dtype, shape, ref, cands, rec.atol, rec.rtol, meta)
