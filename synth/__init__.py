"""Seeded synthetic screening workloads: recipes, and their construction on
the GPU by the library's own seeded generator.

A workload is a reference output and K candidate outputs with planted
differences (the Verifier checks a candidate's output against the
reference's on seeded inputs).  Each tensor is described by a recipe -- a
list of generator steps, each naming a stream (seed, stream_id, sub) of the
Philox4x32-10 counter-based generator and the parameters of one library
call -- so that the same recipe can be carried out by two independent
implementations: `build()` here runs it on the GPU through the library
(kb_gen_inputs, kb_gen_softmax_rows, kb_gen_indices, kb_gen_perturb,
kb_gen_scatter; torch only allocates, copies and zero-fills), and the
oracle package runs it on the CPU (oracle.workloads).  This module holds
no generator or screening arithmetic of its own: only the recipes (stream
ids and parameters) and the calls.

Streams: stream_id = (workload << 8) | purpose, purposes REF 0, NOISE 1,
MASK 2, INDEX 3; sub = the candidate index (0 for the reference); seed 0.

Workloads (the five screening configurations):

  c1  K=4,    N=65,536 fp32,        atol=rtol=1e-5: reference N(0,1) (seed 0);
      c0 a copy; c1 + U(-1e-6, 1e-6); c2 with NaN at 5 drawn indices;
      c3 x 1.01 where u < 0.01;
  c2  K=16,   4096x4096 bf16,       atol=rtol=1e-2: reference bf16(64 z);
      candidate k is bf16(fmaf(r, e, r)), e ~ U(-s_k, s_k), s_k = 2^(-8 + 2k/15),
      and candidates 0 and 1 also get a drawn 64x64 tile set to +0;
  c3  K=1024, 256x1024 fp32,        atol=1e-6, rtol=1e-5: softmax rows of 2 z
      (binary64, rounded once); candidate k adds s_k z, s_k = 10^(-9 + 6k/1023);
  c4  K=64,   8x2048x4096 fp16,     atol=rtol=1e-3: reference fp16(z); by k mod
      4: a copy, last-bit flips where u < 0.001, 64 drawn infinities with the
      sign of r, both;
  c5  K=8,    2^30 fp32,            atol=1e-8, rtol=1e-6: Student-t (3) with
      subnormals (2^-10), signed zeros (2^-10) and infinities (2^-20) planted;
      per element with probability 1/2 a zero-sign flip, a subnormal flush
      or a relative change of up to 1e-7.

Every workload also has a scaled form (`scale` < 1 shrinks N, keeping the
recipe) for the oracle-sized parity cases.
"""
import math
from dataclasses import dataclass, field
from typing import List

SPECS = {
    "c1": dict(K=4, shape=(65536,), dtype="f32", atol=1e-5, rtol=1e-5),
    "c2": dict(K=16, shape=(4096, 4096), dtype="bf16", atol=1e-2, rtol=1e-2),
    "c3": dict(K=1024, shape=(256, 1024), dtype="f32", atol=1e-6, rtol=1e-5),
    "c4": dict(K=64, shape=(8, 2048, 4096), dtype="f16", atol=1e-3, rtol=1e-3),
    "c5": dict(K=8, shape=(1 << 30,), dtype="f32", atol=1e-8, rtol=1e-6),
}
CFG = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}

# purposes of the independent seeded streams
REF, NOISE, MASK, INDEX = 0, 1, 2, 3

# generator codes (the library's and the oracle's, which agree)
DIST_UNIFORM, DIST_NORMAL, DIST_STUDENT_T3 = 1, 2, 3
(ADD_UNIFORM, REL_UNIFORM, ADD_NORMAL, SCALE_WHERE, FLIP_LSB_WHERE, SPECIALS,
 ZERO_SUBNORMAL_REL) = range(1, 8)
SCATTER_NAN, SCATTER_INF_SIGN_OF_REF = 1, 2

# c5's planted specials: cumulative thresholds on u (subnormal, zero, infinity)
SUBNORMAL_P = 2.0 ** -10
ZERO_P = 2.0 ** -9
INF_P = 2.0 ** -9 + 2.0 ** -20


def f32(x):
    """x rounded to binary32 (the parameters both builders are given)."""
    import struct
    return struct.unpack("f", struct.pack("f", x))[0]


@dataclass
class Step:
    """One generator call of a recipe.
      gen       the tensor is the stream's `dist` with (p0, p1)
      softmax   the tensor [rows, cols] is softmax rows of NORMAL(0, sigma)
      perturb   the tensor is op(tensor) (kb_gen_perturb) on the stream
      scatter   m distinct indices drawn from the stream get the mode's value
                (the reference supplies the sign)
      tile      a 64 x 64 tile of the [rows, cols] tensor, at (w0 mod rows/64,
                w1 mod cols/64) from words 0 and 1 of the stream's block 0,
                is set to +0
    """
    kind: str
    stream_id: int
    sub: int = 0
    args: dict = field(default_factory=dict)


@dataclass
class Recipe:
    name: str
    shape: tuple
    dtype: str          # "f32", "f16" or "bf16"
    atol: float
    rtol: float
    seed: int
    ref: List[Step]     # from nothing
    cands: List[List[Step]]  # each from a copy of the reference

    @property
    def numel(self):
        return math.prod(self.shape)

    @property
    def dtype_bytes(self):
        return 4 if self.dtype == "f32" else 2


def _sid(name, purpose):
    return (CFG[name] << 8) | purpose


def scaled_shape(name, scale):
    shape = SPECS[name]["shape"]
    if scale >= 1.0:
        return tuple(shape)
    if name == "c2":
        side = max(64, int(round(math.sqrt(math.prod(shape) * scale))) // 64 * 64)
        return (side, side)
    if name == "c3":
        return (max(1, int(round(shape[0] * scale))), shape[1])
    return (max(1, int(round(math.prod(shape) * scale))),)


def recipe(name, seed=0, scale=1.0, K=None):
    """The recipe of workload `name` (scale < 1 shrinks N; K=None keeps K)."""
    spec = SPECS[name]
    shape = scaled_shape(name, scale)
    K = spec["K"] if (K is None or name == "c1") else K
    n = math.prod(shape)
    ref_s, noise, mask, index = (_sid(name, p) for p in (REF, NOISE, MASK, INDEX))
    cands = []
    if name == "c1":
        ref = [Step("gen", ref_s, 0, dict(dist=DIST_NORMAL, p0=0.0, p1=1.0))]
        cands = [[],
                 [Step("perturb", noise, 1, dict(op=ADD_UNIFORM, a=f32(-1e-6), b=f32(1e-6), p=0.0))],
                 [Step("scatter", index, 2, dict(m=min(5, n // 2), mode=SCATTER_NAN))],
                 [Step("perturb", mask, 3, dict(op=SCALE_WHERE, a=f32(1.01), b=0.0, p=f32(0.01)))]][:K]
    elif name == "c2":
        ref = [Step("gen", ref_s, 0, dict(dist=DIST_NORMAL, p0=0.0, p1=64.0))]
        for k in range(K):
            s = f32(2.0 ** (-8.0 + 2.0 * k / 15.0))
            steps = [Step("perturb", noise, k, dict(op=REL_UNIFORM, a=-s, b=s, p=0.0))]
            if k < 2 and shape[0] >= 64 and shape[1] >= 64:
                steps.append(Step("tile", index, k))
            cands.append(steps)
    elif name == "c3":
        ref = [Step("softmax", ref_s, 0, dict(sigma=2.0))]
        for k in range(K):
            s = f32(10.0 ** (-9.0 + 6.0 * k / max(1, K - 1)))
            cands.append([Step("perturb", noise, k, dict(op=ADD_NORMAL, a=s, b=0.0, p=0.0))])
    elif name == "c4":
        ref = [Step("gen", ref_s, 0, dict(dist=DIST_NORMAL, p0=0.0, p1=1.0))]
        for k in range(K):
            kind, steps = k % 4, []
            if kind in (1, 3):
                steps.append(Step("perturb", mask, k, dict(op=FLIP_LSB_WHERE, a=0.0, b=0.0, p=f32(0.001))))
            if kind in (2, 3):
                steps.append(Step("scatter", index, k, dict(m=min(64, n // 2), mode=SCATTER_INF_SIGN_OF_REF)))
            cands.append(steps)
    elif name == "c5":
        ref = [Step("gen", ref_s, 0, dict(dist=DIST_STUDENT_T3, p0=0.0, p1=1.0)),
               Step("perturb", mask, 0, dict(op=SPECIALS, a=SUBNORMAL_P, b=ZERO_P, p=INF_P))]
        for k in range(K):
            cands.append([Step("perturb", noise, k, dict(op=ZERO_SUBNORMAL_REL, a=f32(-1e-7), b=f32(1e-7),
                                                         p=0.5))])
    else:
        raise KeyError(name)
    return Recipe(name, shape, spec["dtype"], spec["atol"], spec["rtol"], seed, ref, cands)


# ------------------------------------------------------------ on the GPU ---

@dataclass
class Workload:
    name: str
    ref: "object"
    cands: list
    atol: float
    rtol: float
    meta: dict = field(default_factory=dict)

    @property
    def numel(self):
        return self.ref.numel()

    @property
    def dtype_bytes(self):
        return self.ref.element_size()

    def screened_bytes(self):
        return len(self.cands) * self.numel * self.dtype_bytes


def _tile_of(kb, rows, cols, seed, stream_id, sub, device):
    import torch
    w = torch.empty(4, dtype=torch.int32, device=device)
    kb.kb_gen_inputs(w, kb.KB_DIST_U32, seed=seed, stream_id=stream_id, sub=sub)
    w0, w1 = (int(x) & 0xFFFFFFFF for x in w[:2].cpu().tolist())
    return w0 % (rows // 64), w1 % (cols // 64)


def _run_gpu(kb, steps, t, ref, rec, device, meta):
    """Carry out `steps` on device tensor t (ref: the finished reference)."""
    for st in steps:
        a = st.args
        if st.kind == "gen":
            kb.kb_gen_inputs(t, a["dist"], a["p0"], a["p1"], seed=rec.seed, stream_id=st.stream_id, sub=st.sub)
        elif st.kind == "softmax":
            kb.kb_gen_softmax_rows(t.view(rec.shape[0], -1), a["sigma"], seed=rec.seed, stream_id=st.stream_id,
                                   sub=st.sub)
        elif st.kind == "perturb":
            kb.kb_gen_perturb(t, t, a["op"], a["a"], a["b"], a["p"], seed=rec.seed, stream_id=st.stream_id,
                              sub=st.sub)
        elif st.kind == "scatter":
            idx = kb.kb_gen_indices(a["m"], t.numel(), device, seed=rec.seed, stream_id=st.stream_id, sub=st.sub)
            kb.kb_gen_scatter(t, ref, idx, a["mode"])
            meta.setdefault("indices", {})[st.sub] = idx.cpu().tolist()
        elif st.kind == "tile":
            rows, cols = rec.shape
            tr, tc = _tile_of(kb, rows, cols, rec.seed, st.stream_id, st.sub, device)
            t.view(rows, cols)[64 * tr:64 * tr + 64, 64 * tc:64 * tc + 64].zero_()
            meta.setdefault("tiles", {})[st.sub] = (tr, tc)
        else:
            raise ValueError(st.kind)


def build(name, device="cuda:0", seed=0, scale=1.0, K=None):
    """Workload `name` built on `device` by the library's generator calls."""
    import torch

    import paper_2608_02611_amd as kb
    rec = recipe(name, seed=seed, scale=scale, K=K)
    dt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[rec.dtype]
    device = torch.device(device)
    meta = {}
    with torch.no_grad():
        ref = torch.empty(rec.shape, dtype=dt, device=device)
        _run_gpu(kb, rec.ref, ref.view(-1), ref.view(-1), rec, device, meta)
        cands = []
        for steps in rec.cands:
            c = ref.clone()
            _run_gpu(kb, steps, c.view(-1), ref.view(-1), rec, device, meta)
            cands.append(c)
    return Workload(name, ref, cands, rec.atol, rec.rtol, meta)


# ------------------------------------------------------------ timing samples

RUNG_REPEATS = (4, 16, 60)  # timed iterations on rungs 0, 1, 2


def timing_samples(n_cands, n_shapes, n_iter, seed=0, device="cpu", shape_us=None):
    """Seeded synthetic timing samples (us), float64 [n_cands][n_shapes][n_iter].

    Recipe (the shape of the paper's measurements, not its data):
      - shape s has a base latency shape_us[s] (default: 50 us doubling per
        shape, like a sweep over growing sizes);
      - candidate c is slower than the best by a factor spread_c drawn
        log-uniformly from [1, 30] (the rung-0 score spread of Fig. 2 reaches
        about 30x), candidate 0 (the baseline) at 5x;
      - each iteration adds half-normal jitter of 0.3% and, with probability
        3%, a spike of 2-25% (tail ratios p99/p50 of about 1.01-1.25, the
        range of Table A.3).
    """
    import torch
    g = torch.Generator(device="cpu").manual_seed(0x5EED0000 + seed)
    if shape_us is None:
        shape_us = [50.0 * (2 ** s) for s in range(n_shapes)]
    lat = torch.tensor(shape_us, dtype=torch.float64)
    spread = torch.exp(torch.rand(n_cands, generator=g, dtype=torch.float64) * math.log(30.0))
    spread[0] = 5.0
    mean = spread[:, None, None] * lat[None, :, None]
    jitter = torch.randn(n_cands, n_shapes, n_iter, generator=g, dtype=torch.float64).abs() * 0.003
    spike = (torch.rand(n_cands, n_shapes, n_iter, generator=g, dtype=torch.float64) < 0.03)
    spike_amt = 0.02 + 0.23 * torch.rand(n_cands, n_shapes, n_iter, generator=g, dtype=torch.float64)
    t = mean * (1.0 + jitter + spike.double() * spike_amt)
    return t.to(device)
