"""Seeded synthetic screening workloads (shared input generator).

This module only synthesizes inputs: a reference output and K candidate
outputs per workload, built with torch's own seeded generator on the device
they will be screened on.  It holds none of the screening arithmetic and none
of the library's generator; the parity tests hand the same bytes to the HIP
library (on the GPU) and to the CPU oracle (after a copy to the host).

Workloads (the five screening configurations):

  c1  K=4,    N=65,536 fp32,        atol=rtol=1e-5: reference N(0,1); a copy,
      a copy with U(+-1e-6) noise, one with 5 NaNs at drawn indices, one with
      1% of its elements scaled by 1.01;
  c2  K=16,   4096x4096 bf16,       atol=rtol=1e-2: reference bf16(64 z);
      candidate k is bf16(r + r eps), eps ~ U(-s_k, s_k), s_k = 2^(-8 + 2k/15),
      and candidates 0 and 1 also get a drawn 64x64 tile set to 0;
  c3  K=1024, 256x1024 fp32,        atol=1e-6, rtol=1e-5: softmax rows of
      2 z (binary64, rounded); candidate k adds s_k z, s_k log-spaced 1e-9..1e-3;
  c4  K=64,   8x2048x4096 fp16,     atol=rtol=1e-3: reference fp16(z); by k mod
      4: a copy, last-bit flips on 0.1% of elements, 64 infinities with the
      sign of r, both;
  c5  K=8,    2^30 fp32,            atol=1e-8, rtol=1e-6: Student-t (3) with
      subnormals, signed zeros and infinities; per element with probability
      1/2 a zero-sign flip, a subnormal flush or a 1e-7 relative change.

Every workload also has a scaled form (`scale` < 1 shrinks N, keeping the
recipe) for the oracle-sized parity cases.
"""
import math
from dataclasses import dataclass, field
from typing import List

import torch

SPECS = {
    "c1": dict(K=4, shape=(65536,), dtype=torch.float32, atol=1e-5, rtol=1e-5),
    "c2": dict(K=16, shape=(4096, 4096), dtype=torch.bfloat16, atol=1e-2, rtol=1e-2),
    "c3": dict(K=1024, shape=(256, 1024), dtype=torch.float32, atol=1e-6, rtol=1e-5),
    "c4": dict(K=64, shape=(8, 2048, 4096), dtype=torch.float16, atol=1e-3, rtol=1e-3),
    "c5": dict(K=8, shape=(1 << 30,), dtype=torch.float32, atol=1e-8, rtol=1e-6),
}

# purposes of the independent seeded draws
REF, NOISE, MASK, INDEX, AUX = 0, 1, 2, 3, 4
CHUNK = 1 << 26  # elements per construction chunk (bounds temporaries)


@dataclass
class Workload:
    name: str
    ref: torch.Tensor
    cands: List[torch.Tensor]
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


def _gen(device, seed, cfg, purpose, k=0, chunk=0):
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + (cfg << 40) + (purpose << 32) + (k << 12) + chunk)
    return g


def scaled_shape(shape, scale):
    if scale >= 1.0:
        return tuple(shape)
    n = max(1, int(round(math.prod(shape) * scale)))
    return (n,)


def _distinct(g, n, m, device):
    """m distinct indices in [0, n)."""
    m = min(m, n)
    if n <= (1 << 24):
        return torch.randperm(n, generator=g, device=device)[:m]
    picked = torch.unique(torch.randint(0, n, (2 * m + 16,), generator=g, device=device))
    return picked[torch.randperm(picked.numel(), generator=g, device=device)[:m]]


# ------------------------------------------------------------------- c1 ---

def _c1(device, seed, shape):
    n = math.prod(shape)
    ref = torch.randn(shape, generator=_gen(device, seed, 1, REF), device=device)
    c0 = ref.clone()
    noise = torch.rand(shape, generator=_gen(device, seed, 1, NOISE, 1), device=device)
    c1 = ref + (noise * 2e-6 - 1e-6)
    c2 = ref.clone()
    idx = _distinct(_gen(device, seed, 1, INDEX, 2), n, 5, device)
    c2.view(-1)[idx] = float("nan")
    mask = torch.rand(shape, generator=_gen(device, seed, 1, MASK, 3), device=device) < 0.01
    c3 = torch.where(mask, ref * 1.01, ref)
    return ref, [c0, c1, c2, c3], {"nan_index": idx.cpu().tolist()}


# ------------------------------------------------------------------- c2 ---

def _c2(device, seed, shape, K=16):
    z = torch.randn(shape, generator=_gen(device, seed, 2, REF), device=device)
    ref = (z * 64.0).to(torch.bfloat16)
    r32 = ref.float()
    cands, tiles = [], []
    for k in range(K):
        sigma = 2.0 ** (-8.0 + 2.0 * k / 15.0)
        u = torch.rand(shape, generator=_gen(device, seed, 2, NOISE, k), device=device)
        eps = (u * 2.0 - 1.0) * sigma
        c = (r32 + r32 * eps).to(torch.bfloat16)
        if k < 2 and len(shape) == 2 and shape[0] >= 64 and shape[1] >= 64:
            g = _gen(device, seed, 2, INDEX, k)
            tr = int(torch.randint(0, shape[0] // 64, (1,), generator=g, device=device))
            tc = int(torch.randint(0, shape[1] // 64, (1,), generator=g, device=device))
            c[64 * tr:64 * tr + 64, 64 * tc:64 * tc + 64] = 0
            tiles.append((tr, tc))
        cands.append(c)
    return ref, cands, {"tiles": tiles}


# ------------------------------------------------------------------- c3 ---

def _c3(device, seed, shape, K=1024):
    logits = torch.randn(shape, generator=_gen(device, seed, 3, REF), device=device) * 2.0
    ref = torch.softmax(logits.double(), dim=-1).float()
    cands = []
    for k in range(K):
        sigma = 10.0 ** (-9.0 + 6.0 * k / max(1, K - 1))
        z = torch.randn(shape, generator=_gen(device, seed, 3, NOISE, k), device=device)
        cands.append(ref + z * sigma)
    return ref, cands, {}


# ------------------------------------------------------------------- c4 ---

def _c4(device, seed, shape, K=64):
    n = math.prod(shape)
    ref = torch.randn(shape, generator=_gen(device, seed, 4, REF), device=device).half()
    bits = ref.view(torch.int16)
    n_inf = min(64, n)
    cands = []
    for k in range(K):
        kind = k % 4
        c = ref.clone()
        if kind in (1, 3):
            flip = torch.rand(shape, generator=_gen(device, seed, 4, MASK, k), device=device) < 0.001
            cb = c.view(torch.int16)
            cb.copy_(torch.where(flip, bits ^ 1, bits))
        if kind in (2, 3):
            idx = _distinct(_gen(device, seed, 4, INDEX, k), n, n_inf, device)
            flat = c.view(-1)
            flat[idx] = torch.copysign(torch.full_like(flat[idx], float("inf")), ref.view(-1)[idx])
        cands.append(c)
    return ref, cands, {}


# ------------------------------------------------------------------- c5 ---

SUBNORMAL_P = 2.0 ** -10
ZERO_P = 2.0 ** -9
INF_P = 2.0 ** -9 + 2.0 ** -20


def _c5_ref_chunk(device, seed, lo, hi, ci):
    n = hi - lo
    g = _gen(device, seed, 5, REF, 0, ci)
    z = torch.randn((4, n), generator=g, device=device)
    t = z[0] / torch.sqrt((z[1] * z[1] + z[2] * z[2] + z[3] * z[3]) / 3.0)
    gm = _gen(device, seed, 5, MASK, 0, ci)
    u = torch.rand(n, generator=gm, device=device)
    sign = torch.where(torch.rand(n, generator=gm, device=device) < 0.5, -1.0, 1.0)
    mant = torch.randint(0, 1 << 23, (n,), generator=gm, device=device, dtype=torch.int32) | 1
    sub = mant.view(torch.float32) * sign  # bit pattern mant with exponent 0: a subnormal
    t = torch.where(u < SUBNORMAL_P, sub, t)
    t = torch.where((u >= SUBNORMAL_P) & (u < ZERO_P), sign * 0.0, t)
    t = torch.where((u >= ZERO_P) & (u < INF_P), sign * float("inf"), t)
    return t


def _c5_cand_chunk(device, seed, r, k, ci):
    g = _gen(device, seed, 5, NOISE, k, ci)
    v = torch.rand(r.numel(), generator=g, device=device)
    delta = torch.rand(r.numel(), generator=g, device=device) * 2e-7 - 1e-7
    hit = v < 0.5
    a = r.abs()
    is_zero = a == 0
    is_sub = (a > 0) & (a < 2.0 ** -126)
    is_inf = torch.isinf(r)
    normal = ~(is_zero | is_sub | is_inf)
    c = r.clone()
    c = torch.where(hit & is_zero, -r, c)                      # sign-of-zero flip
    c = torch.where(hit & is_sub, r * 0.0, c)                   # flush, keeps the sign
    c = torch.where(hit & normal, r + r * delta, c)             # 1e-7-relative perturbation
    return c


def _c5(device, seed, shape, K=8):
    n = math.prod(shape)
    ref = torch.empty(n, dtype=torch.float32, device=device)
    cands = [torch.empty(n, dtype=torch.float32, device=device) for _ in range(K)]
    for ci, lo in enumerate(range(0, n, CHUNK)):
        hi = min(n, lo + CHUNK)
        r = _c5_ref_chunk(device, seed, lo, hi, ci)
        ref[lo:hi] = r
        for k in range(K):
            cands[k][lo:hi] = _c5_cand_chunk(device, seed, r, k, ci)
    return ref.view(shape), [c.view(shape) for c in cands], {}


BUILDERS = {"c1": _c1, "c2": _c2, "c3": _c3, "c4": _c4, "c5": _c5}


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


def build(name, device="cpu", seed=0, scale=1.0, K=None):
    """Workload `name` on `device`; scale < 1 shrinks N (and K=None keeps K)."""
    spec = SPECS[name]
    shape = spec["shape"] if scale >= 1.0 else scaled_shape(spec["shape"], scale)
    if name == "c2" and scale < 1.0:
        side = max(64, int(round(math.sqrt(math.prod(spec["shape"]) * scale))) // 64 * 64)
        shape = (side, side)
    kwargs = {}
    if K is not None and name != "c1":
        kwargs["K"] = K
    with torch.no_grad():
        ref, cands, meta = BUILDERS[name](torch.device(device), seed, shape, **kwargs)
    return Workload(name, ref, cands, spec["atol"], spec["rtol"], meta)
