#!/usr/bin/env python3
"""Screening throughput on one MI355X: candidate GB/s screened.

One step is one pass of the screening hot path over one batch of candidate
outputs already resident in HBM: the policy gate, the screening kernel (one
coalesced read of the reference and the K candidates, per-candidate
statistics) and the readback of the K records with the pass/fail verdict.
Steps are pipelined the way a screening service runs independent batches:
they alternate over two streams, each with its own workspace, so that a
pass starts on the work-group slots the previous pass frees while its last
work-groups finish; the kernel of each step writes its records straight
into one of 2 * BATCH pinned host buffers (a ring per stream), one
completion event per stream follows every BATCH steps of that stream, and
while the device works on the current batch the host takes the verdicts of
the batch before it (after that batch's events).  value = K * numel *
element bytes / step time (GB/s).  A few fully synchronous steps (launch,
copy back, wait) are timed too and reported as sync_step_ms.

Before the timed region the device runs about 0.2 s of back-to-back
launches (untimed), so that the timed steps run at the sustained clock, and
the W warmup steps run the same pipelined loop as the timed ones.

The JSON line also carries the roofline of the screening kernel.  Its
duration is measured right after the timed steps: the same number of
launches back to back on one stream between a pair of HIP events on that
stream, with nothing else in between, so the interval divided by the
launches is the kernel's time per launch, including the dispatch gap
between kernels (and agreeing with a kernel trace of the run).  The
algorithmic bytes are (K+1) * numel * element bytes per launch, a compulsory
read of every candidate and the reference once.  Also: single launches
timed warm and cold (after a 512 MiB read that evicts the caches), the CPU
oracle timed on a bounded sample of the same workload, the generator's
throughput, two
optional passes over the same candidates (the position search,
kb_screen_locate, and the fail-fast screen, KB_FAIL_FAST, whose kernel time
and share of candidate elements read are reported beside the full
screen's), a multi-output screen (kb_screen_multi) of attention-style
output pairs, and the rung statistics and promotion decision
(kb_rung_stats, kb_rung_promote) over synthetic timing samples.

roofline.traffic is the kernel's HBM traffic per launch from hardware
counters (FETCH_SIZE and WRITE_SIZE, each scaled by the reading of the same
counter for a plain device copy of known size, collected by two rocprofv3
--pmc runs of `bench.py --copy-calibration`).  The collected numbers are
kept in profiles/screen_traffic_<workload>.txt together with a digest of the
kernel sources they were taken from; when the sources have changed since,
traffic is null.
"""
import hashlib
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# Steps per stream between completion events of the pipelined loop: an
# event recorded between two launches was measured to add about 3.3 us to
# that step (the device's signal between kernels), so the host takes the
# verdicts in batches of BATCH steps per stream, over a ring of 2 * BATCH
# pinned record slots per stream (--batch).
BATCH_DEFAULT = 4
METRIC = "candidate GB/s screened (K\u00d7N\u00d7dtype bytes/s) and % of MI355X HBM peak"
KERNEL_SOURCES = ["paper_2608_02611_amd/csrc/kb_screen.hip", "paper_2608_02611_amd/csrc/kb_device.hpp",
                  "paper_2608_02611_amd/csrc/kb_internal.hpp"]
WORKLOADS = {
    "c1": "K=4 candidates, N=65,536 fp32, atol=rtol=1e-5",
    "c2": "K=16 candidates, 4096x4096 bf16 (GEMM-output shape), atol=rtol=1e-2",
    "c3": "K=1024 candidates, 256x1024 fp32 softmax rows, atol=1e-6 rtol=1e-5",
    "c4": "K=64 candidates, 8x2048x4096 fp16 (attention-output shape), atol=rtol=1e-3",
    "c5": "K=8 candidates, 2^30 fp32 (4 GiB each), atol=1e-8 rtol=1e-6",
}


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
            if ":" in line and not line.startswith(" "):
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
    for name, fn, moved in (("copy", lambda: dst.copy_(src), 2 * nbytes),
                            ("sum_f32", lambda: x.sum(), nbytes)):
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


def single_launch(scr, stream, dev, reps=10, flush_bytes=512 << 20):
    """One launch at a time, each between its own pair of events: warm (the
    previous launch's data may still sit in L2 and the 256 MB last-level
    cache) and cold (a 512 MiB buffer read just before, outside the event
    pair, evicts them; read rather than written, so that no dirty lines are
    left to be written back during the launch).  Medians in ms; each
    includes one launch's dispatch and the events' own signal."""
    import torch
    buf = torch.ones(flush_bytes // 4, dtype=torch.float32, device=dev)
    res = {}
    for name, flush in (("warm_ms", False), ("cold_ms", True)):
        ms = []
        for _ in range(reps):
            if flush:
                buf.sum()
                torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            scr.launch(0)
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        res[name] = round(sorted(ms)[len(ms) // 2], 5)
    del buf
    return res


def cpu_baseline(w, seconds):
    """The oracle, single-threaded, on the first S elements of every candidate,
    S chosen from a probe so that the sample takes about `seconds`; when the
    whole workload takes less, whole passes over it are repeated until about
    `seconds` have passed (the rate is over all of them)."""
    import oracle
    from tests.helpers import dtype_name, storage

    dt = dtype_name(w.ref)
    n = w.numel
    probe = min(n, 1 << 18)
    r = storage(w.ref.reshape(-1)[:probe])
    c = storage(w.cands[0].reshape(-1)[:probe])
    t = time.perf_counter()
    oracle.screen(r, c, dt, w.atol, w.rtol)
    per_elem = max(1e-10, (time.perf_counter() - t) / probe)
    per_cand = max(1, min(n, int(seconds / per_elem / len(w.cands))))
    r = storage(w.ref.reshape(-1)[:per_cand])
    cs = [storage(x.reshape(-1)[:per_cand]) for x in w.cands]
    passes = 0
    t = time.perf_counter()
    while True:
        for x in cs:
            oracle.screen(r, x, dt, w.atol, w.rtol)
        passes += 1
        el = time.perf_counter() - t
        if per_cand < n or el >= 0.9 * seconds:
            break
    nbytes = passes * len(cs) * per_cand * w.dtype_bytes
    what = ("first %d elements of each of the %d candidates" % (per_cand, len(cs)) if per_cand < n
            else "%d pass%s over all %d candidates of %d elements" % (passes, "" if passes == 1 else "es",
                                                                      len(cs), n))
    return {"value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "%s (%.1f MB screened, %.1f s)" % (what, nbytes / 1e6, el)}


def gen_throughput(dev, kb, n, dtype):
    import torch
    out = torch.empty(n, dtype=dtype, device=dev)
    res = {}
    for name, dist in (("normal", kb.KB_DIST_NORMAL), ("uniform", kb.KB_DIST_UNIFORM)):
        kb.kb_gen_inputs(out, dist, 0.0, 1.0, seed=0, stream_id=0x7701)
        torch.cuda.synchronize()
        reps = 5
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for i in range(reps):
            kb.kb_gen_inputs(out, dist, 0.0, 1.0, seed=0, stream_id=0x7701, sub=i)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / reps
        res[name] = {"n": n, "ms": round(ms, 4), "Gsamples_per_s": round(n / ms / 1e6, 2),
                     "GB_per_s_written": round(n * out.element_size() / ms / 1e6, 1)}
    del out
    return res


def multi_output_leg(dev, kb, K=16):
    """kb_screen_multi on an attention-style output pair: out fp16
    [4, 32, 2048, 128] and lse fp32 [4, 32, 2048], K candidates (in-tolerance
    noise on both outputs).  Kernel time over both outputs and the
    algorithmic GB/s ((K + 1) x the bytes of one output tuple), calls back
    to back with the arguments marshalled once.  (fp16, so
    that its launches are not the same kernel instantiation as the headline
    workload's, whose profile they would otherwise mix into.)"""
    import torch
    g = torch.Generator(device=dev).manual_seed(3)
    out = torch.randn(4, 32, 2048, 128, generator=g, device=dev).to(torch.float16)
    lse = torch.randn(4, 32, 2048, generator=g, device=dev) + 8.0
    refs = [out, lse]
    cands = []
    for k in range(K):
        gk = torch.Generator(device=dev).manual_seed(100 + k)
        cands.append([(out.float() * (1 + 1e-3 * torch.randn(out.shape, generator=gk, device=dev)))
                      .to(torch.float16),
                      lse + 1e-6 * torch.randn(lse.shape, generator=gk, device=dev)])
    ms_ = kb.MultiScreener(refs, cands, [1e-2, 1e-4], [1e-2, 1e-4])
    for _ in range(3):
        ms_.launch()
    torch.cuda.synchronize()
    # calls back to back (arguments marshalled once), timed as one region
    ms = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            ms_.launch()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1) / 10)
    m = sorted(ms)[len(ms) // 2]
    tup = out.numel() * 2 + lse.numel() * 4
    recs = ms_.records()
    return {"outputs": ["f16 [4,32,2048,128]", "f32 [4,32,2048]"], "K": K, "ms": round(m, 4),
            "algorithmic_GB_per_s": round((K + 1) * tup / (m * 1e-3) / 1e9, 1),
            "n_passed": sum(1 for k in range(K) if recs[k]["passed"] and recs[K + k]["passed"])}


def rung_stats_leg(dev, kb, synth, C=1024, S=3, N=60):
    """kb_rung_stats on 1024 candidates x 3 shapes x 60 iterations (the
    last rung of the paper's schedule): kernel time, plus the samples and
    scores for the CPU-baseline leg's comparison."""
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
    grows, gscores = kb.rung_records(rows, scores, C, S)
    # the promotion decision over those scores (2/5 of the candidates, the
    # baseline carried)
    pus = []
    for _ in range(20):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rank, order, prom = kb.kb_rung_promote(scores, C, 0, 2, 5)
        e1.record()
        torch.cuda.synchronize()
        pus.append(e0.elapsed_time(e1) * 1e3)
    leg = {"candidates": C, "shapes": S, "iterations": N, "us": round(sorted(us)[len(us) // 2], 1),
           "sample_bytes": C * S * N * 8, "promote_us": round(sorted(pus)[len(pus) // 2], 1),
           "promoted": int(prom.sum().item())}
    return leg, (t.numpy(), grows, gscores)


def rung_cpu_baseline(samples, grows, gscores):
    """The oracle on the same timing samples, single-threaded (CPU-baseline
    leg): its time, and whether every score and row field is the same bits."""
    import oracle
    t0 = time.perf_counter()
    orows, oscores = oracle.rung_stats(samples, 0, 2, 60.0)
    ms = (time.perf_counter() - t0) * 1e3
    same = all(g["score"] == o["score"] and g["latency_us"] == o["latency"]
               for g, o in zip(gscores, oscores)) and \
        all(g["p99_over_p50"] == o["tail99"] and g["mean_us"] == o["mean"]
            for gr, orr in zip(grows, orows) for g, o in zip(gr, orr))
    return {"ms": round(ms, 2), "cores": 1, "kind": "oracle", "bit_identical_to_gpu": bool(same)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c2", choices=sorted(WORKLOADS))
    ap.add_argument("--batch", type=int, default=BATCH_DEFAULT,
                    help="steps per stream between completion events (verdicts taken per batch)")
    ap.add_argument("--streams", type=int, default=2,
                    help="streams the pipelined steps alternate over (each with its own workspace)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gen", action="store_true")
    ap.add_argument("--no-stream-context", action="store_true")
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
    # One screener (workspace, ring of record slots) per stream; steps
    # alternate over the streams.
    streams = [torch.cuda.Stream() for _ in range(args.streams)]
    scrs = [kb.Screener(w.ref, w.cands, w.atol, w.rtol, stream=st, host_slots=2 * batch) for st in streams]
    scr = scrs[0]
    plan = scr.launch_plan()
    S = len(scrs)

    def slot_of(i):
        return scrs[i % S], (i // S) % (2 * batch)

    def pipelined(n):
        """n steps, step i on stream i mod S into that stream's ring of
        2 * batch pinned record slots; after every `batch` steps per stream
        one completion event per stream, and the verdicts of the batch
        before it (whose events have then been reached).  Returns the
        summary of the last step."""
        per_batch = batch * S
        evs = []
        summary = None

        def take(bi):
            nonlocal summary
            for e in evs[bi]:
                e.synchronize()
            for i in range(bi * per_batch, min(n, (bi + 1) * per_batch)):
                sc, sl = slot_of(i)
                summary = sc.summarize(sl)

        for i in range(n):
            sc, sl = slot_of(i)
            sc.launch(sl)
            if (i + 1) % per_batch == 0 or i == n - 1:
                evb = []
                for st in streams:
                    e = torch.cuda.Event()
                    e.record(st)
                    evb.append(e)
                evs.append(evb)
                if len(evs) >= 2:
                    take(len(evs) - 2)
        take(len(evs) - 1)
        return summary

    # Untimed: bring the device to its sustained clock (about 0.2 s of
    # back-to-back launches; a timed loop right after a short warmup was
    # measured about 6% slower while the clocks ramp), then the W warmup
    # steps, pipelined like the timed ones.
    log("device warm-up")
    t_warm = time.perf_counter() + 0.2
    while time.perf_counter() < t_warm:
        for i in range(20):
            scr.launch(i % (2 * batch))
        torch.cuda.synchronize()
    log("warmup", args.warmup)
    if args.warmup > 0:
        pipelined(args.warmup)
    torch.cuda.synchronize()
    log("timing", args.steps, "steps")
    t0 = time.perf_counter()
    summary = pipelined(args.steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    # The kernel alone, for the roofline: the same number of launches back to
    # back on one stream, between a pair of HIP events on that stream (no
    # completion events in between), so that the interval divided by the
    # launches is the kernel's time per launch including the dispatch gap.
    first = torch.cuda.Event(enable_timing=True)
    last = torch.cuda.Event(enable_timing=True)
    first.record(streams[0])
    for i in range(args.steps):
        scr.launch(i % (2 * batch))
    last.record(streams[0])
    torch.cuda.synchronize()
    kern_ms = first.elapsed_time(last) / args.steps
    # synchronous steps: launch, copy the records back, wait
    sync = kb.Screener(w.ref, w.cands, w.atol, w.rtol)
    sync.launch()
    sync.read()
    ts = time.perf_counter()
    for _ in range(10):
        sync.launch()
        sync.read()
    sync_ms = (time.perf_counter() - ts) * 1e3 / 10
    for i in range(max(0, args.steps - S), args.steps):
        sc, sl = slot_of(i)
        assert sync.records() == sc.records(sl), "pipelined and synchronous records differ"
    screened = K * n * b
    algorithmic = (K + 1) * n * b
    value = screened / (ms_per_step * 1e-3) / 1e9
    achieved = algorithmic / (kern_ms * 1e-3) / 1e9
    summ = {k: summary.as_dict()[k] for k in ("n_passed", "n_failed", "n_rejected")}
    log("summary", summ)

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
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (args.config, WORKLOADS[args.config]), "K": K,
                   "numel": n, "storage_dtype": str(w.ref.dtype).replace("torch.", ""),
                   "atol": w.atol, "rtol": w.rtol, "launch": plan,
                   "pipeline": {"streams": S, "steps_per_completion_event": batch},
                   "verdicts": summ},
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBPS, 2),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": counted_traffic(args.config), "kernel_ms": round(kern_ms, 5),
                     "algorithmic_bytes_per_launch": algorithmic, "kernel_digest": kernel_digest()},
    }
    tr = out["roofline"]["traffic"]
    # counted HBM bytes per launch over the same kernel time
    out["roofline"]["traffic_GB_per_s"] = round(tr / (kern_ms * 1e-3) / 1e9, 1) if tr else None
    # one launch at a time, warm and after a cache flush
    sl = single_launch(scr, streams[0], dev)
    sl["cold_algorithmic_GB_per_s"] = round(algorithmic / (sl["cold_ms"] * 1e-3) / 1e9, 1)
    out["single_launch"] = sl
    if args.copy_calibration:
        log("copy calibration")
        copy_calibration(dev)
    # the optional position pass (kb_screen_locate) over all candidates,
    # after the synchronous screen above (its records stay on the device)
    loc_ms = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        locs = kb.kb_screen_locate(w.ref, w.cands, w.atol, w.rtol, sync.d_stats)
        e1.record()
        torch.cuda.synchronize()
        loc_ms.append(e0.elapsed_time(e1))
    # the same pass with its arguments marshalled once, calls back to back:
    # the device time per call (the fill of the positions and the kernel)
    loc = kb.Locator(w.ref, w.cands, w.atol, w.rtol, sync.d_stats)
    for _ in range(3):
        loc.launch()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        loc.launch()
    e1.record()
    torch.cuda.synchronize()
    assert loc.read() == locs, "pre-marshalled positions differ"
    out["locate"] = {"ms": round(sorted(loc_ms)[len(loc_ms) // 2], 4),
                     "device_ms": round(e0.elapsed_time(e1) / 10, 4),
                     "failed_candidates_first_mismatch": [l["first_mismatch"] for l in locs
                                                          if l["first_mismatch"] >= 0][:4]}
    # the fail-fast mode (KB_FAIL_FAST) on the same candidates: the verdicts
    # must be the ones of the full screen; reported are its kernel time and
    # the share of candidate elements it read
    log("fail-fast")
    ff = kb.Screener(w.ref, w.cands, w.atol, w.rtol, flags=kb.KB_FAIL_FAST)
    ff.launch()
    ff.read()
    ff_ms = []
    for _ in range(10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ff.launch()
        e1.record()
        torch.cuda.synchronize()
        ff_ms.append(e0.elapsed_time(e1))
    ff.read()
    frec, full = ff.records(), sync.records()
    assert [r["mismatches"] > 0 for r in frec] == [r["mismatches"] > 0 for r in full], \
        "fail-fast verdicts differ from the full screen"
    ffm = sorted(ff_ms)[len(ff_ms) // 2]
    out["fail_fast"] = {"kernel_ms": round(ffm, 5),
                        "vs_full_kernel": round(kern_ms / ffm, 2),
                        "candidate_elements_read_frac": round(sum(r["numel"] for r in frec) / (K * n), 4),
                        "n_failed": sum(r["mismatches"] > 0 for r in frec)}
    # the rung benchmarker's statistics (kb_rung_stats) over synthetic timing
    # samples (the CPU-baseline leg compares them with the oracle)
    log("multi-output")
    out["multi_output"] = multi_output_leg(dev, kb)
    log("rung statistics")
    out["rung_stats"], rung_data = rung_stats_leg(dev, kb, synth)
    if not args.no_stream_context:
        log("stream context")
        out["stream_context"] = stream_context(dev)
    if not args.no_gen:
        log("generator throughput")
        out["gen"] = gen_throughput(dev, kb, n, w.ref.dtype)
    if not args.no_cpu_baseline:
        log("cpu baseline")
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
        out["cpu_baseline"]["rung_stats"] = rung_cpu_baseline(*rung_data)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
