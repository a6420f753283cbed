#!/usr/bin/env python3
"""Screening throughput on one MI355X: candidate GB/s screened.

One step is one pass of the screening hot path over one batch of candidate
outputs already resident in HBM: the policy gate, the screening kernel (one
coalesced read of the reference and the K candidates, per-candidate
statistics) and the K records with their pass/fail verdicts, which the kernel
writes into pinned host memory and the library's kb_summarize turns into
verdicts.  Steps run back to back on ONE stream, so a step's kernel never
overlaps another's: the host enqueues step i and takes the verdicts of the
steps whose completion event has passed (one event per BATCH steps over a
ring of 2 * BATCH record slots), so host work hides behind the device.
value = K * numel * element bytes / step time (GB/s), on the headline
workload (default c5: 8 candidates of 2^30 fp32, the largest that fits one
GPU).  A few fully synchronous steps (launch, copy back, wait) are timed too
(sync_step_ms).  With --two-streams the same steps also run alternating over
two streams (pipelined_two_streams), which lets one step's first work-groups
start while the previous step's last ones finish (off by default: its
overlapping kernels would stretch the kernel's durations in a trace of the
default command).

Inputs are built on the device by the library's own seeded generator (the
synth recipes: kb_gen_inputs, kb_gen_softmax_rows, kb_gen_indices,
kb_gen_perturb, kb_gen_scatter) before the timed region.

roofline: the screening kernel of the headline workload.  Its duration is
the interval between two HIP events recorded on the screening stream around
the timed steps, divided by the steps (the kernels run back to back there,
so this is the kernel time per launch including the dispatch gap, and agrees
with a kernel trace of the run); achieved = (K + 1) * numel * element bytes
(a compulsory read of every candidate and of the reference) / that time.
roofline.traffic is the kernel's HBM bytes per launch from hardware counters
(FETCH_SIZE and WRITE_SIZE, each scaled by the reading of the same counter for
a plain device copy of known size, from two rocprofv3 --pmc runs of
`bench.py --config <w> --only-config --copy-calibration`), kept in
profiles/screen_traffic_<workload>.txt with a digest of the kernel sources;
null when the sources changed since.

configs: the same measurement (kernel time between events over back-to-back
launches on one stream) for the other four workloads, with their verdicts.

cpu_baseline: the CPU oracle (oracle/, the plain per-element loop) screening
a bounded sample of the headline workload -- the first S elements of the
reference and of every candidate, S sized for about --cpu-seconds of
single-core work -- built on the host by the oracle itself from the same
recipe; timed on one core, and on all the host cores the process may use
(threads over (candidate, 2^22-element chunk), merged in chunk order).  The
host's core count, CPU model and memory are reported beside it.

Other legs (skipped with --only-config): the position search -- found in the
screening pass (kb_screen_ex with positions) and as a separate pass
(kb_screen_locate) -- and the fail-fast screen (KB_FAIL_FAST) on the
16-candidate bf16 workload (which has failing candidates), a multi-output
screen, the rung
statistics and promotion decision, the generator's throughput, and plain
copy/reduction rates of the box for context.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# Steps between completion events of the pipelined loop: an event recorded
# between two launches was measured to add about 3.3 us to that step (the
# device's signal between kernels), so the host takes the verdicts in
# batches of BATCH steps over a ring of 2 * BATCH pinned record slots.
BATCH_DEFAULT = 4
METRIC = "candidate GB/s screened (K×N×dtype bytes/s) and % of MI355X HBM peak"
KERNEL_SOURCES = ["paper_2608_02611_amd/csrc/kb_screen.hip", "paper_2608_02611_amd/csrc/kb_device.hpp",
                  "paper_2608_02611_amd/csrc/kb_internal.hpp"]
WORKLOADS = {
    "c1": "K=4 candidates, N=65,536 fp32, atol=rtol=1e-5",
    "c2": "K=16 candidates, 4096x4096 bf16 (GEMM-output shape), atol=rtol=1e-2",
    "c3": "K=1024 candidates, 256x1024 fp32 softmax rows, atol=1e-6 rtol=1e-5",
    "c4": "K=64 candidates, 8x2048x4096 fp16 (attention-output shape), atol=rtol=1e-3",
    "c5": "K=8 candidates, 2^30 fp32 Student-t(3) with planted specials (4 GiB each), atol=1e-8 rtol=1e-6",
}
MAX_CPU_THREADS = 16  # the host share of one GPU


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_digest():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counted_traffic(config):
    """HBM bytes per launch from the committed counter summary, or None when
    there is none or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "screen_traffic_%s.txt" % config)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_digest") != kernel_digest():
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def copy_calibration(dev, nbytes=1 << 30, reps=3):
    """A plain device copy of known size (nbytes read, nbytes written per
    launch), run so that a counter pass can scale its readings."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def stream_context(dev, nbytes=1 << 30):
    """What plain library kernels reach on this machine (context for the
    roofline, not a bound of the screening kernel): a device-to-device copy
    (nbytes read + nbytes written) and torch's sum over nbytes of fp32
    (nbytes read)."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    x = src.view(torch.float32)
    res = {}
    for name, fn, moved in (("copy", lambda: dst.copy_(src), 2 * nbytes), ("sum_f32", lambda: x.sum(), nbytes)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(10):
            fn()
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / 10
        res[name] = {"bytes": moved, "ms": round(ms, 4), "GB_per_s": round(moved / ms / 1e6, 1)}
    del src, dst, x
    return res


def warm_device(launch, seconds=0.2):
    """Back-to-back launches until the device runs at its sustained clock (a
    timed loop right after a short warmup was measured about 6% slower while
    the clocks ramp)."""
    import torch
    t = time.perf_counter() + seconds
    while time.perf_counter() < t:
        for _ in range(8):
            launch()
        torch.cuda.synchronize()


def event_time(launch, reps, stream):
    """Device time per launch: reps launches back to back on `stream` between
    two HIP events recorded on that stream (ms)."""
    import torch
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        launch()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


class Pipeline:
    """Steps over one or more streams, each with its own Screener and a ring
    of 2 * batch pinned record slots; one completion event per stream after
    every `batch` steps of it, and the verdicts of the batch before taken
    once its events have passed."""

    def __init__(self, kb, w, streams, batch):
        self.batch, self.streams = batch, streams
        self.scrs = [kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st, host_slots=2 * batch) for st in streams]

    def slot_of(self, i):
        S = len(self.scrs)
        return self.scrs[i % S], (i // S) % (2 * self.batch)

    def run(self, n):
        import torch
        per_batch = self.batch * len(self.scrs)
        evs, summary = [], None

        def take(bi):
            nonlocal summary
            for e in evs[bi]:
                e.synchronize()
            for i in range(bi * per_batch, min(n, (bi + 1) * per_batch)):
                sc, sl = self.slot_of(i)
                summary = sc.summarize(sl)

        for i in range(n):
            sc, sl = self.slot_of(i)
            sc.launch(sl)
            if (i + 1) % per_batch == 0 or i == n - 1:
                evb = []
                for st in self.streams:
                    e = torch.cuda.Event()
                    e.record(st)
                    evb.append(e)
                evs.append(evb)
                if len(evs) >= 2:
                    take(len(evs) - 2)
        take(len(evs) - 1)
        return summary


def verdict_counts(summary):
    d = summary.as_dict() if hasattr(summary, "as_dict") else summary
    return {k: d[k] for k in ("n_passed", "n_failed", "n_rejected")}


def config_record(kb, name, w, reps):
    """Kernel time over back-to-back launches on one stream, between events,
    and the verdicts, for one workload."""
    import torch
    st = torch.cuda.Stream()
    scr = kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st)
    warm_device(scr.launch, 0.1)
    ms = event_time(scr.launch, reps, st)
    summ = scr.read()
    K, n, b = len(w.cands), w.numel, w.dtype_bytes
    alg = (K + 1) * n * b
    return {"workload": "%s: %s" % (name, WORKLOADS[name]), "K": K, "numel": n,
            "storage_dtype": str(w.ref.dtype).replace("torch.", ""), "launch": scr.launch_plan(),
            "kernel_ms": round(ms, 5), "screened_GB_per_s": round(K * n * b / ms / 1e6, 1),
            "achieved_GB_per_s": round(alg / ms / 1e6, 1), "frac": round(alg / ms / 1e6 / HBM_PEAK_GBPS, 4),
            "traffic": counted_traffic(name), "verdicts": verdict_counts(summ)}


def host_description():
    model, mem = None, None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal"):
                    mem = round(int(line.split()[1]) / (1 << 20), 1)
                    break
    except OSError:
        pass
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"nproc": os.cpu_count(), "usable_cpus": usable, "cpu_model": model, "mem_GiB": mem}


def cpu_baseline(name, seconds, threads):
    """The oracle screening the first S elements of every candidate of the
    workload (built by the oracle on the host), on one core, then on
    `threads` cores over (candidate, chunk) tasks merged in chunk order."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    from oracle import workloads
    probe = workloads.build(name, prefix=1 << 20)
    dt, K = probe.dtype, len(probe.cands)
    t = time.perf_counter()
    oracle.screen(probe.ref, probe.cands[0], dt, probe.atol, probe.rtol)
    per_elem = max(1e-10, (time.perf_counter() - t) / probe.ref.size)
    n_full = synthetic_numel(name)
    S = int(min(n_full, max(1 << 20, seconds / per_elem / K)))
    S = max(1 << 20, S >> 20 << 20) if S < n_full else n_full
    w = workloads.build(name, prefix=S)
    S = w.ref.size
    nbytes = K * S * (4 if dt == "f32" else 2)
    t = time.perf_counter()
    one = [oracle.screen(w.ref, c, dt, w.atol, w.rtol) for c in w.cands]
    t1 = time.perf_counter() - t
    chunk = 1 << 22
    bounds = [(lo, min(S, lo + chunk)) for lo in range(0, S, chunk)]

    def part(task):
        k, (lo, hi) = task
        return oracle.screen_partial(w.ref, w.cands[k], dt, w.atol, w.rtol, 0, lo, hi)

    tasks = [(k, b) for k in range(K) for b in bounds]
    t = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(part, tasks))
    many = [oracle.finalize(oracle.merge(parts[k * len(bounds):(k + 1) * len(bounds)])) for k in range(K)]
    tn = time.perf_counter() - t
    exact = ("numel", "mismatches", "nan_count", "pos_inf_count", "neg_inf_count", "max_abs_err", "max_rel_err",
             "bitwise_equal", "passed")
    same = all(a[f] == b[f] for a, b in zip(one, many) for f in exact)
    sample = ("the first %d elements of the reference and of each of the %d candidates (%.1f MB screened), "
              "built on the host by the oracle from the workload's recipe" % (S, K, nbytes / 1e6))
    return {"value": round(nbytes / t1 / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle", "sample": sample,
            "seconds": round(t1, 2),
            "all_cores": {"value": round(nbytes / tn / 1e9, 4), "unit": "GB/s", "cores": threads,
                          "seconds": round(tn, 2), "counts_flags_maxima_equal_to_one_core": bool(same)},
            "host": host_description()}


def synthetic_numel(name):
    import math

    import synth
    return math.prod(synth.SPECS[name]["shape"])


def gen_throughput(dev, kb, n):
    """Generator kernels on n elements: binary32 normal, uniform and
    Student-t, and one planted change (ms and Gsamples/s)."""
    import torch
    out = torch.empty(n, dtype=torch.float32, device=dev)
    res = {}
    for name, fn in (("normal", lambda i: kb.kb_gen_inputs(out, kb.KB_DIST_NORMAL, 0.0, 1.0, 0, 0x7701, i)),
                     ("uniform", lambda i: kb.kb_gen_inputs(out, kb.KB_DIST_UNIFORM, 0.0, 1.0, 0, 0x7701, i)),
                     ("student_t3", lambda i: kb.kb_gen_inputs(out, kb.KB_DIST_STUDENT_T3, 0.0, 1.0, 0, 0x7701, i)),
                     ("perturb_rel", lambda i: kb.kb_gen_perturb(out, out, kb.KB_PERTURB_ZERO_SUBNORMAL_REL,
                                                                  -1e-7, 1e-7, 0.5, 0, 0x7702, i))):
        fn(0)
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for i in range(3):
            fn(i)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / 3
        res[name] = {"n": n, "ms": round(ms, 4), "Gsamples_per_s": round(n / ms / 1e6, 2)}
    del out
    return res


def multi_output_leg(dev, kb, K=16):
    """kb_screen_multi on an attention-style output pair: out fp16
    [4, 32, 2048, 128] and lse fp32 [4, 32, 2048], K candidates (in-tolerance
    noise on both outputs, planted by the library); kernel time over both
    outputs and the algorithmic GB/s ((K + 1) x the bytes of one output
    tuple), calls back to back with the arguments marshalled once."""
    import torch
    out = torch.empty(4, 32, 2048, 128, dtype=torch.float16, device=dev)
    lse = torch.empty(4, 32, 2048, dtype=torch.float32, device=dev)
    kb.kb_gen_inputs(out, kb.KB_DIST_NORMAL, 0.0, 1.0, seed=0, stream_id=0x0600)
    kb.kb_gen_inputs(lse, kb.KB_DIST_NORMAL, 8.0, 1.0, seed=0, stream_id=0x0601)
    cands = []
    for k in range(K):
        co, cl = torch.empty_like(out), torch.empty_like(lse)
        kb.kb_gen_perturb(co, out, kb.KB_PERTURB_REL_UNIFORM, -2e-3, 2e-3, 0.0, seed=0, stream_id=0x0610, sub=k)
        kb.kb_gen_perturb(cl, lse, kb.KB_PERTURB_ADD_NORMAL, 1e-6, 0.0, 0.0, seed=0, stream_id=0x0611, sub=k)
        cands.append([co, cl])
    ms_ = kb.MultiScreener([out, lse], cands, [1e-2, 1e-4], [1e-2, 1e-4])
    for _ in range(3):
        ms_.launch()
    torch.cuda.synchronize()
    m = event_time(ms_.launch, 10, torch.cuda.current_stream())
    tup = out.numel() * 2 + lse.numel() * 4
    recs = ms_.records()
    return {"outputs": ["f16 [4,32,2048,128]", "f32 [4,32,2048]"], "K": K, "ms": round(m, 4),
            "algorithmic_GB_per_s": round((K + 1) * tup / (m * 1e-3) / 1e9, 1),
            "n_passed": sum(1 for k in range(K) if recs[k]["passed"] and recs[K + k]["passed"])}


def rung_stats_leg(dev, kb, synth, C=1024, S=3, N=60):
    """kb_rung_stats on 1024 candidates x 3 shapes x 60 iterations (the
    last rung of the paper's schedule) and the promotion decision."""
    import torch
    t = synth.timing_samples(C, S, N, seed=7)
    d = t.to(dev)
    rows, scores = kb.kb_rung_stats(d, 0, 2, 60.0)
    torch.cuda.synchronize()
    us = []
    for _ in range(20):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        kb.kb_rung_stats(d, 0, 2, 60.0, rows=rows, scores=scores)
        e1.record()
        torch.cuda.synchronize()
        us.append(e0.elapsed_time(e1) * 1e3)
    pus = []
    for _ in range(20):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rank, order, prom = kb.kb_rung_promote(scores, C, 0, 2, 5)
        e1.record()
        torch.cuda.synchronize()
        pus.append(e0.elapsed_time(e1) * 1e3)
    return {"candidates": C, "shapes": S, "iterations": N, "us": round(sorted(us)[len(us) // 2], 1),
            "sample_bytes": C * S * N * 8, "promote_us": round(sorted(pus)[len(pus) // 2], 1),
            "promoted": int(prom.sum().item())}


def positions_leg(kb, w, reps=20, rounds=3):
    """The screen with positions found in the same pass (kb_screen_ex with
    opts.d_loc) against the plain screen, back to back on one stream: kernel
    time per launch of each (the best of `rounds` alternating measurements),
    and the positions, which must equal those of the separate pass
    (kb_screen_locate).  The separate pass is timed too: device time per call
    (its fill of the positions and its kernel), calls back to back."""
    import torch
    st = torch.cuda.Stream()
    plain = kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st)
    withpos = kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st, positions=True)
    warm_device(plain.launch, 0.1)
    plain_ms = pos_ms = float("inf")
    for _ in range(rounds):
        plain_ms = min(plain_ms, event_time(plain.launch, reps, st))
        pos_ms = min(pos_ms, event_time(withpos.launch, reps, st))
    plain.read()
    withpos.read()
    precs, wrecs = plain.records(), withpos.records()
    assert [r["passed"] for r in precs] == [r["passed"] for r in wrecs], "verdicts differ with positions"
    got = withpos.positions()
    loc = kb.Locator(w.ref, w.cands, w.atol, w.rtol, plain.d_stats, stream=st)
    loc.launch()
    want = loc.read()
    assert got == want, "positions of the screening pass differ from the separate pass"
    sep_ms = min(event_time(loc.launch, reps, st) for _ in range(rounds))
    assert loc.read() == want, "repeated separate passes differ"
    K, n, b = len(w.cands), w.numel, w.dtype_bytes
    alg = (K + 1) * n * b
    return {"plain_kernel_ms": round(plain_ms, 5), "with_positions_kernel_ms": round(pos_ms, 5),
            "ratio": round(pos_ms / plain_ms, 3), "with_positions_frac": round(alg / pos_ms / 1e6 / HBM_PEAK_GBPS, 4),
            "separate_pass_ms": round(sep_ms, 5), "separate_pass_vs_plain": round(sep_ms / plain_ms, 3),
            "launch": withpos.launch_plan(), "positions_equal_separate_pass": True,
            "failed_candidates_first_mismatch": [l["first_mismatch"] for l in got if l["first_mismatch"] >= 0][:4]}


def failing_workload_legs(kb, w):
    """The position search (in the screening pass, and as a separate pass)
    and the fail-fast screen on a workload with failing candidates (the
    16-candidate bf16 one)."""
    import torch
    K, n = len(w.cands), w.numel
    st = torch.cuda.current_stream()
    fused = positions_leg(kb, w)
    full = kb.Screener(w.ref, w.cands, w.atol, w.rtol)
    full.launch()
    full.read()
    full_ms = event_time(full.launch, 10, st)
    frec = full.records()
    loc = kb.Locator(w.ref, w.cands, w.atol, w.rtol, full.d_stats)
    for _ in range(3):
        loc.launch()
    torch.cuda.synchronize()
    loc_ms = event_time(loc.launch, 10, st)
    locs = loc.read()
    ff = kb.Screener(w.ref, w.cands, w.atol, w.rtol, flags=kb.KB_FAIL_FAST)
    ff.launch()
    ff.read()
    ff_ms = event_time(ff.launch, 10, st)
    ff.read()
    ffrec = ff.records()
    assert [r["passed"] for r in ffrec] == [r["passed"] for r in frec], "fail-fast verdicts differ"
    return {
        "workload": "c2: " + WORKLOADS["c2"], "screen_kernel_ms": round(full_ms, 5),
        "screen_with_positions": fused,
        "locate": {"device_ms": round(loc_ms, 5), "vs_screen": round(loc_ms / full_ms, 3),
                   "failed_candidates_first_mismatch": [l["first_mismatch"] for l in locs
                                                        if l["first_mismatch"] >= 0][:4]},
        "fail_fast": {"kernel_ms": round(ff_ms, 5), "speedup_vs_full": round(full_ms / ff_ms, 2),
                      "candidate_elements_read_frac": round(sum(r["numel"] for r in ffrec) / (K * n), 4),
                      "n_failed": sum(1 for r in ffrec if not r["passed"])}}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c5", choices=sorted(WORKLOADS))
    ap.add_argument("--batch", type=int, default=BATCH_DEFAULT,
                    help="steps between completion events (verdicts taken per batch)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only-config", action="store_true",
                    help="measure the named workload only (no other workloads, no side legs): for counter runs")
    ap.add_argument("--two-streams", action="store_true",
                    help="also time the steps alternating over two streams (pipelined_two_streams)")
    ap.add_argument("--positions", action="store_true",
                    help="with --only-config: also time the screen with positions on the named workload")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run 3 plain 1 GiB device copies (for counter calibration)")
    args = ap.parse_args()
    batch = max(1, args.batch)
    if args.gpus != 1:
        print("bench.py measures one GPU: the screening library runs on a single MI355X "
              "(sharding over several GPUs is described, not implemented); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import __graft_entry__
    __graft_entry__._ensure_built()
    import torch

    import paper_2608_02611_amd as kb
    import synth

    dev = torch.device("cuda:0")
    log("building workload", args.config)
    w = synth.build(args.config, dev, seed=0)
    torch.cuda.synchronize()
    K, n, b = len(w.cands), w.numel, w.dtype_bytes
    stream = torch.cuda.Stream()
    pipe = Pipeline(kb, w, [stream], batch)
    scr = pipe.scrs[0]
    plan = scr.launch_plan()

    log("device warm-up")
    warm_device(lambda: scr.launch(0))
    log("warmup", args.warmup)
    if args.warmup > 0:
        pipe.run(args.warmup)
    torch.cuda.synchronize()
    log("timing", args.steps, "steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    t0 = time.perf_counter()
    summary = pipe.run(args.steps)
    e1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    kern_ms = e0.elapsed_time(e1) / args.steps
    summ = verdict_counts(summary)
    log("summary", summ)

    # synchronous steps: launch, copy the records back, wait
    sync = kb.Screener(w.ref, w.cands, w.atol, w.rtol)
    sync.launch()
    sync.read()
    ts = time.perf_counter()
    for _ in range(5):
        sync.launch()
        sync.read()
    sync_ms = (time.perf_counter() - ts) * 1e3 / 5
    sc, sl = pipe.slot_of(args.steps - 1)
    assert sync.records() == sc.records(sl), "pipelined and synchronous records differ"
    del sync

    screened = K * n * b
    algorithmic = (K + 1) * n * b
    value = screened / (ms_per_step * 1e-3) / 1e9
    achieved = algorithmic / (kern_ms * 1e-3) / 1e9
    traffic = counted_traffic(args.config)
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "sync_step_ms": round(sync_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "f16": "f16", "bf16": "bf16"}[synth.SPECS[args.config]["dtype"]],
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (args.config, WORKLOADS[args.config]), "K": K, "numel": n,
                   "storage_dtype": str(w.ref.dtype).replace("torch.", ""), "atol": w.atol, "rtol": w.rtol,
                   "seed": 0, "launch": plan,
                   "pipeline": {"streams": 1, "steps_per_completion_event": batch}, "verdicts": summ},
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBPS, 2),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "kernel_ms": round(kern_ms, 5), "algorithmic_bytes_per_launch": algorithmic,
                     "kernel_digest": kernel_digest(),
                     "traffic_GB_per_s": round(traffic / (kern_ms * 1e-3) / 1e9, 1) if traffic else None},
    }
    if args.copy_calibration:
        log("copy calibration")
        copy_calibration(dev)
    if args.positions and args.only_config:
        log("screen with positions")
        out["screen_with_positions"] = positions_leg(kb, w)
    if args.two_streams:
        log("two-stream pipeline")
        two = Pipeline(kb, w, [stream, torch.cuda.Stream()], batch)
        two.run(2 * batch * 2)
        torch.cuda.synchronize()
        t = time.perf_counter()
        two.run(args.steps)
        torch.cuda.synchronize()
        ms2 = (time.perf_counter() - t) * 1e3 / args.steps
        out["pipelined_two_streams"] = {"ms_per_step": round(ms2, 5),
                                        "screened_GB_per_s": round(screened / ms2 / 1e6, 1)}
        del two
    if not args.only_config:
        del pipe, scr
        # the other workloads: kernel time, roofline fraction, verdicts
        del w
        torch.cuda.empty_cache()
        out["configs"] = {}
        c2 = None
        for name in sorted(WORKLOADS):
            if name == args.config:
                continue
            log("workload", name)
            wk = synth.build(name, dev, seed=0)
            out["configs"][name] = config_record(kb, name, wk, 20 if name != "c5" else 5)
            if name == "c2":
                c2 = wk
            else:
                del wk
            torch.cuda.empty_cache()
        if c2 is not None:
            log("position search and fail-fast on c2")
            out["failing_workload_legs"] = failing_workload_legs(kb, c2)
            del c2
            torch.cuda.empty_cache()
        log("multi-output")
        out["multi_output"] = multi_output_leg(dev, kb)
        log("rung statistics")
        out["rung_stats"] = rung_stats_leg(dev, kb, synth)
        log("generator throughput")
        out["gen"] = gen_throughput(dev, kb, 1 << 28)
        log("stream context")
        out["stream_context"] = stream_context(dev)
    if not args.no_cpu_baseline:
        log("cpu baseline")
        threads = max(1, min(MAX_CPU_THREADS, host_description()["usable_cpus"] or 1))
        out["cpu_baseline"] = cpu_baseline(args.config, args.cpu_seconds, threads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
