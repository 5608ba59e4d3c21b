"""Benchmark of the RoI N:M mask sampler step (mask forward + backward) on one GPU.

A step is one forward (hard top-n sample, masked weights and selected
indices) and one backward (grad_logits from grad_W_masked) over the whole
synthetic stack, with every input already resident in HBM.  The default
workload is the 7B-class full stack at 2:4 (28 layers x 7 linears, 196
tensors, 6.53e9 masked weights) with tau annealed from 1.0 to 0.1 over 10
steps (§4.2.3 exponential schedule); the stack is one back-to-back slab, so
each direction is one kernel launch.

Prints one JSON line (rank 0).  Kernel durations come from HIP events
recorded on the stream the kernels are launched on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "masked weights/sec (mask fwd+bwd) and achieved HBM GB/s vs peak, 7B-class 2:4"
HBM_PEAK_GBPS = 8000.0
# MI355X fp32 vector peak: 256 CUs x 128 fp32 lanes x 2 flops (fused multiply-add)
# x 2.4 GHz.
FP32_VECTOR_PEAK_TFLOPS = 157.3
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "roi_mask_qwen7b_stack_2of4_traffic.json")
VALU_FILE = os.path.join(ROOT, "profiles", "roi_mask_valu_counters.json")


# The sources the benchmark's two kernels (fwd_lane_kernel, bwd_lane_kernel
# for m = 4 and 8) are compiled from.
KERNEL_SOURCES = ("roi.hip", "common.hpp", "noise.hpp", "relax.hpp", "host.hpp")
# ... and those of every straight-through forward and backward kernel (the
# counter record covers the lane and the wide kernels).
ALL_KERNEL_SOURCES = KERNEL_SOURCES + ("wide.hpp", "wide_fwd.hip", "wide_bwd.hip")


def code_only(text: str) -> str:
    """C/C++ source without its comments, whitespace collapsed (string and
    character literals kept as they are)."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash(sources=KERNEL_SOURCES) -> str:
    """Hash of the code of the measured kernels' sources (comments and
    whitespace aside): measured counters are reported only while it is
    unchanged."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_23048_amd", "csrc")
    for name in sources:
        h.update(name.encode())
        h.update(code_only(open(os.path.join(csrc, name)).read()).encode())
    return h.hexdigest()[:16]


def measured_traffic():
    """Per-launch HBM bytes of the dominant kernel from the committed rocprofv3
    counter summary, or None when it is missing or the kernels changed since."""
    import json as _json
    if not os.path.exists(TRAFFIC_FILE):
        return None
    rec = _json.load(open(TRAFFIC_FILE))
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec


# Hardware-counter passes of the traffic record (rocprofv3 --pmc, one pass
# each; a pass holds at most four TCC counters).  FETCH_SIZE and WRITE_SIZE
# are the derived memory-side kilobytes per dispatch.  The second estimates
# come from other counters: the read requests to memory counted by size
# (128, 64 and 32 bytes), and the 32-byte sectors of the write requests that
# reach the L2 from the compute units.
COUNTER_PASSES = {
    "fetch": ["FETCH_SIZE"],
    "write": ["WRITE_SIZE", "TCC_WRITE_SECTORS_sum"],
    "reads": ["TCC_EA0_RDREQ_128B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_32B_sum"],
}


def counter_calibration(nbytes: int) -> int:
    """Three kernels that move known bytes, for the counter passes: the
    library's streaming copy (reads and writes nbytes, with the access pattern
    of the sampler's kernels), a sum over nbytes (reads only) and a fill of
    nbytes (writes only)."""
    import torch

    import paper_2608_23048_amd as roi
    # The contents do not matter, only the bytes moved: the buffers are left
    # uninitialized, so that the fill below is the program's only fill, and the
    # sum runs over fp32 (an integer sum would first widen the data).
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    roi.stream_copy(a, b)
    torch.cuda.synchronize()
    a.view(torch.float32).sum()
    torch.cuda.synchronize()
    b.fill_(3)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_bytes": nbytes}), flush=True)
    return 0


def _dispatch_counters(path):
    """{dispatch id: (kernel name, {counter: value})} from a rocprofv3 --pmc CSV."""
    import csv
    out = {}
    for r in csv.DictReader(open(path)):
        d = out.setdefault(r["Dispatch_Id"], (r["Kernel_Name"], {}))
        d[1][r["Counter_Name"]] = d[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def _bytes_of(c):
    """Byte estimates of one dispatch from whatever counters it carries."""
    est = {}
    if "FETCH_SIZE" in c:
        est["fetch_size"] = c["FETCH_SIZE"] * 1024.0
    if "WRITE_SIZE" in c:
        est["write_size"] = c["WRITE_SIZE"] * 1024.0
    if "TCC_EA0_RDREQ_128B_sum" in c:
        est["read_requests"] = (128.0 * c["TCC_EA0_RDREQ_128B_sum"] +
                                64.0 * c["TCC_EA0_RDREQ_64B_sum"] +
                                32.0 * c["TCC_EA0_RDREQ_32B_sum"])
    if "TCC_WRITE_SECTORS_sum" in c:
        est["write_requests"] = 32.0 * c["TCC_WRITE_SECTORS_sum"]
    return est


def _largest(disp, key):
    """Mean byte estimates over the full-size dispatches (within a factor 2 of
    the largest) of the kernels whose name contains key."""
    rows = [_bytes_of(c) for name, c in disp.values() if key in name]
    rows = [r for r in rows if r]
    if not rows:
        return None
    out = {}
    for k in rows[0]:
        vals = [r[k] for r in rows if k in r]
        big = [v for v in vals if v >= 0.5 * max(vals)] or vals
        out[k] = sum(big) / len(big)
    return out


def _total(disp, key):
    """Byte estimates summed over every dispatch of the kernels whose name
    contains key (a library may split one operation into several launches)."""
    out = {}
    for name, c in disp.values():
        if key in name:
            for k, v in _bytes_of(c).items():
                out[k] = out.get(k, 0.0) + v
    return out


def traffic_summary(bench_csvs, calib_csvs, calib_bytes: int, numel: int, n: int, m: int) -> int:
    """The committed traffic record from the counter passes of the benchmark
    and of the calibration run (one CSV per pass, in COUNTER_PASSES order).
    FETCH_SIZE and WRITE_SIZE are scaled by what they read for the streaming
    copy of known size; the read-only and write-only kernels and the
    request-size counters check those scales."""
    import json as _json
    bench, calib = {}, {}
    for path in bench_csvs:
        for k, v in _dispatch_counters(path).items():
            bench.setdefault(k + "@" + path, v)
    for path in calib_csvs:
        for k, v in _dispatch_counters(path).items():
            calib.setdefault(k + "@" + path, v)

    def merged(disp, key, per_launch=True):
        est = {}
        for path in set(p.split("@", 1)[1] for p in disp):
            sub = {k: v for k, v in disp.items() if k.endswith("@" + path)}
            e = _largest(sub, key) if per_launch else _total(sub, key)
            if e:
                est.update(e)
        return est

    B = float(calib_bytes)
    known = {"stream_copy": (B, B), "reduce": (B, 0.0), "fill": (0.0, B)}
    cal = {}
    for key, (rd, wr) in known.items():
        pattern = {"stream_copy": "stream_copy_kernel", "reduce": "reduce_kernel",
                   "fill": "FillFunctor"}[key]
        e = merged(calib, pattern, per_launch=False)
        cal[key] = {"known_read_bytes": rd, "known_write_bytes": wr, **e}
    sc = cal["stream_copy"]
    fetch_scale = B / sc["fetch_size"] if sc.get("fetch_size") else None
    write_scale = B / sc["write_size"] if sc.get("write_size") else None
    for key, e in cal.items():
        rd, wr = known[key]
        if rd and e.get("fetch_size"):
            e["fetch_size_over_known"] = e["fetch_size"] / rd
        if rd and e.get("read_requests"):
            e["read_requests_over_known"] = e["read_requests"] / rd
        if wr and e.get("write_size"):
            e["write_size_over_known"] = e["write_size"] / wr
        if wr and e.get("write_requests"):
            e["write_requests_over_known"] = e["write_requests"] / wr
    bf, bb = algorithmic_bytes(n, m)
    out = {"kernel_source_hash": kernel_source_hash(), "calibration_bytes": calib_bytes,
           "fetch_scale": fetch_scale, "write_scale": write_scale, "calibration": cal,
           "kernels": {}}
    for key, alg in (("fwd_lane_kernel", bf), ("bwd_lane_kernel", bb)):
        e = merged(bench, key)
        if not e or "fetch_size" not in e or "write_size" not in e:
            continue
        rd = e["fetch_size"] * fetch_scale
        wr = e["write_size"] * write_scale
        rec = {"fetch_kib": e["fetch_size"] / 1024.0, "write_kib": e["write_size"] / 1024.0,
               "read_bytes": rd, "write_bytes": wr, "traffic_bytes": rd + wr,
               "algorithmic_bytes": alg * numel,
               "traffic_over_algorithmic": (rd + wr) / (alg * numel)}
        if "read_requests" in e and "write_requests" in e:
            rec["request_counters_bytes"] = e["read_requests"] + e["write_requests"]
            rec["request_counters_over_algorithmic"] = rec["request_counters_bytes"] / (alg * numel)
        out["kernels"][key] = rec
    _json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
    print(_json.dumps(out), flush=True)
    return 0


def algorithmic_bytes(n: int, m: int) -> tuple[float, float]:
    """Bytes per weight the method must move: forward reads W (bf16) and the
    logits (fp32) and writes W_masked (bf16) and n/m index bytes; backward
    reads grad_W_masked and W (bf16) and the logits, and writes grad_logits."""
    return 2 + 4 + 2 + n / m, 2 + 2 + 4 + 4


def backward_flops(n: int) -> int:
    """Floating-point operations per weight of the backward, counted from the
    algorithm (Gumbel keys, §3.2's relaxation recursion with the stable
    log(1 - mu), and its reverse sweep), whatever the kernel does to get
    there.  Each add, multiply, divide, comparison, exp and log counts 1; a
    fused multiply-add counts 2.
      keys          g = -log(-log u): 2 logs + 2 negations; kappa = phi/lambda
                    + g as one fused multiply-add                          6
      upstream      sbar = grad * W                                        1
      each of the n steps of the recursion, per entry: the group maximum
                    (1), (alpha - max) / tau (2), exp (1), its share of the
                    total (1), mu = e / T (1), omega = (sum of the others) / T
                    (2)                                                    8
                    before the last step: max(omega, FLT_MIN), log, add    3
      each of the n steps of the sweep, per entry: its share of <mu, mubar>
                    (2), mubar - <mu, mubar> (1), times mu (1), times 1/tau
                    (1), accumulate (1)                                    6
                    before the last step: mubar = sbar - abar / omega      2
      output        grad_logits = abar / lambda                            1
    The Philox noise is integer work and not counted.  Total 19 n + 3."""
    return 6 + 1 + 8 * n + 3 * (n - 1) + 6 * n + 2 * (n - 1) + 1


def step_rooflines(workload: str, n: int, m: int, numel: int, fwd_ms: float, bwd_ms: float,
                   traffic, fwd_bytes: float | None = None) -> dict:
    """The step's two rooflines.  HBM: algorithmic bytes of the slower kernel
    over its event time, against 8 TB/s.  ALU: the backward's algorithmic
    flops (backward_flops) over its event time, against the fp32 vector peak,
    with the measured VALU instruction counts beside it when the committed
    record matches the kernels.  `roofline` is the one that bounds the path:
    HBM for m = 4 and 8, whose relaxation is at most 4 steps per weight; ALU
    for m = 16 and 32 (8 and 16 steps per weight, 155 and 307 flops).  fwd_bytes
    overrides the straight-through forward's bytes per weight (the soft
    forward moves 8)."""
    bf, bb = algorithmic_bytes(n, m)
    if fwd_bytes is not None:
        bf = fwd_bytes
    slow = ("roi_mask_bwd", bb, bwd_ms) if bwd_ms >= fwd_ms else ("roi_mask_fwd", bf, fwd_ms)
    hbm_gbps = slow[1] * numel / (slow[2] * 1e-3) / 1e9
    hbm = {"kernel": slow[0], "bound": "hbm", "achieved": hbm_gbps, "peak": HBM_PEAK_GBPS,
           "unit": "GB/s", "frac": hbm_gbps / HBM_PEAK_GBPS, "traffic": traffic}
    flops = backward_flops(n)
    tflops = flops * numel / (bwd_ms * 1e-3) / 1e12
    alu = {"kernel": "roi_mask_bwd", "bound": "alu", "achieved": tflops,
           "peak": FP32_VECTOR_PEAK_TFLOPS, "unit": "TFLOP/s",
           "frac": tflops / FP32_VECTOR_PEAK_TFLOPS, "traffic": None,
           "flops_per_weight": flops, "valu": None}
    rec = measured_valu(workload)
    key = "bwd_wide_kernel" if m >= 8 else "bwd_lane_kernel"
    if rec and key in rec:
        per_w = rec[key]["valu_lane_insts_per_weight"]
        rate = per_w * numel / (bwd_ms * 1e-3) / 1e12
        alu["valu"] = {"lane_insts_per_weight": per_w,
                       "trans_lane_insts_per_weight": rec[key]["trans_lane_insts_per_weight"],
                       "lane_insts_per_s_T": rate,
                       "issue_peak_T": FP32_VECTOR_PEAK_TFLOPS / 2,
                       "issue_frac": rate / (FP32_VECTOR_PEAK_TFLOPS / 2)}
    if m >= 16:
        return {"roofline": alu, "hbm_roofline": hbm}
    return {"roofline": hbm, "alu_roofline": alu}


def measured_valu(workload: str):
    """The VALU counters of a workload's kernels from the committed rocprofv3
    summary, or None when missing or the kernels changed since."""
    if not os.path.exists(VALU_FILE):
        return None
    rec = json.load(open(VALU_FILE))
    if rec.get("kernel_source_hash") != kernel_source_hash(ALL_KERNEL_SOURCES):
        return None
    return rec.get("workloads", {}).get(workload)


def valu_summary(insts_csv, workload: str) -> int:
    """Add one workload's VALU counters to the committed record, from a
    rocprofv3 --pmc CSV of SQ_INSTS_VALU, SQ_INSTS_VALU_TRANS_F32 and SQ_WAVES
    (wave instructions, summed over the chip).  Per kernel: the mean over its
    full-size dispatches, and the lane instructions per weight."""
    import csv
    from paper_2608_23048_amd import workloads as wl
    numel = wl.WORKLOADS[workload].numel
    kernels = {}
    rows = list(csv.DictReader(open(insts_csv)))
    for key in ("fwd_lane_kernel", "bwd_lane_kernel", "fwd_wide_kernel", "bwd_wide_kernel"):
        per = {}  # counter -> dispatch -> value
        for r in rows:
            if key in r["Kernel_Name"]:
                d = per.setdefault(r["Counter_Name"], {})
                d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
        insts = per.get("SQ_INSTS_VALU")
        if not insts:
            continue
        big = [d for d, v in insts.items() if v >= 0.5 * max(insts.values())]

        def mean(counter):
            vals = [per.get(counter, {}).get(d) for d in big]
            vals = [v for v in vals if v is not None]
            return sum(vals) / len(vals) if vals else None

        valu, trans, waves = mean("SQ_INSTS_VALU"), mean("SQ_INSTS_VALU_TRANS_F32"), mean("SQ_WAVES")
        kernels[key] = {
            "dispatches": len(big), "valu_insts": valu, "trans_insts": trans, "waves": waves,
            "valu_insts_per_wave": valu / waves if waves else None,
            "valu_lane_insts_per_weight": valu * 64 / numel,
            "trans_lane_insts_per_weight": trans * 64 / numel if trans is not None else None,
        }
    rec = json.load(open(VALU_FILE)) if os.path.exists(VALU_FILE) else {}
    h = kernel_source_hash(ALL_KERNEL_SOURCES)
    if rec.get("kernel_source_hash") != h:
        rec = {"kernel_source_hash": h, "workloads": {}}
    rec["workloads"][workload] = kernels
    json.dump(rec, open(VALU_FILE, "w"), indent=1, sort_keys=True)
    print(json.dumps({workload: kernels}), flush=True)
    return 0


def copy_reference(nbytes: int = 1 << 32, reps: int = 3) -> dict:
    """The same GPU's streaming bandwidth for the sampler's access pattern:
    roi_stream_copy of nbytes (nbytes read + nbytes written; 16 bytes per lane,
    non-temporal, one-shot grid), timed with HIP events, best of reps."""
    import torch

    import paper_2608_23048_amd as roi
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    a.fill_(1)
    b = torch.empty_like(a)
    best = None
    for _ in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        roi.stream_copy(a, b)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    ok = bool(torch.equal(a[:: 1 << 20], b[:: 1 << 20]))
    del a, b
    torch.cuda.empty_cache()
    return {"kernel": "roi_stream_copy", "bytes_moved": 2 * nbytes, "ms": best,
            "GBps": 2 * nbytes / (best * 1e-3) / 1e9, "checked": ok}


def cpu_baseline(W, L, G, work, n, m, tau):
    """The CPU oracle, as it is, on a bounded sample of the same workload: the
    seven tensors of layer 0 (one mask forward + backward) on the host's
    cores -- the oracle's threaded entry points split the groups over POSIX
    threads, at most the 16 cores that are one GPU's share of the host --
    plus the single-threaded oracle on the 896x896 layer (2:4, tau = 1)."""
    import numpy as np
    import torch

    import oracle
    from paper_2608_23048_amd import workloads as wl

    threads = oracle.host_threads()
    layer = [t for t in work.tensors if t.name.startswith("layers.0.")] or list(work.tensors[:1])
    end = layer[-1].offset + layer[-1].numel
    bits = lambda t: t[:end].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    Wb, Gb, Lf = bits(W), bits(G), L[:end].cpu().numpy()
    t0 = time.perf_counter()
    oracle.mask_fwd(Wb, Lf, n, m, tau, 1.0, 0, 0, 0, want_soft=False, threads=threads)
    oracle.mask_bwd(Gb, Wb, Lf, n, m, tau, 1.0, 0, 0, 0, threads=threads)
    dt = time.perf_counter() - t0
    del Wb, Gb, Lf
    # the single-threaded figure on the one-layer workload
    single = wl.WORKLOADS["single-896x896-2:4"]
    W1, L1, G1 = wl.fill_slab(single, "cpu")
    b1 = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
    t1 = time.perf_counter()
    oracle.mask_fwd(b1(W1), L1.numpy(), single.n, single.m, single.tau, 1.0, 0, 0, 0,
                    want_soft=False)
    oracle.mask_bwd(b1(G1), b1(W1), L1.numpy(), single.n, single.m, single.tau, 1.0, 0, 0, 0)
    dt1 = time.perf_counter() - t1
    names = "+".join(t.name.split(".")[-1] for t in layer)
    return {"value": end / dt, "unit": "masked weights/s", "cores": threads, "kind": "oracle",
            "host_cpus": os.cpu_count(),
            "sample": f"layer 0 ({names}, {end} weights), one mask fwd+bwd, {dt:.2f} s on "
                      f"{threads} threads",
            "single_thread": {"value": single.numel / dt1, "unit": "masked weights/s",
                              "cores": 1, "sample": f"{single.name} ({single.numel} weights), "
                                                    f"one mask fwd+bwd, {dt1:.2f} s"}}


def forward_soft_flops(n: int) -> int:
    """Floating-point operations per weight of the pure soft forward, counted
    from the algorithm as in backward_flops: keys 6; each of the n steps of the
    recursion 8, plus 1 for accumulating S; before the last step 3 (floor, log,
    add); the product W S 1.  Total 12 n + 4."""
    return 6 + 9 * n + 3 * (n - 1) + 1


def run_soft(args) -> int:
    """--mode soft: the step of the paper's default setting, without the
    straight-through estimator: the pure soft forward W_soft = bf16(W (.) S)
    (roi_mask_fwd_soft; no indices, S not stored) and the same backward."""
    import torch

    import paper_2608_23048_amd as roi
    from paper_2608_23048_amd import workloads as wl

    roi.lib()
    work = wl.WORKLOADS[args.workload]
    n, m = work.n, work.m
    dev = torch.device("cuda:0")
    numel = work.numel
    print(f"# soft mode, workload {work.name}: {numel} weights, {n}:{m}", file=sys.stderr,
          flush=True)
    W, L, G = wl.fill_slab(work, dev, step=0)
    Ws = torch.empty_like(W)
    dphi = torch.empty_like(L)
    sched = work.tau_schedule or (work.tau, work.tau, 1)

    def step(t, ev=None):
        tau = roi.anneal(sched[0], sched[1], t, sched[2])
        if ev is not None:
            ev[0].record()
        roi.mask_fwd(W, L, n, m, tau, 1.0, 0, t, 0, want_soft=False, want_idx=False,
                     out={"W_masked": Ws}, soft_forward=True)
        if ev is not None:
            ev[1].record()
        roi.mask_bwd(G, W, L, n, m, tau, 1.0, 0, t, 0, out=dphi)
        if ev is not None:
            ev[2].record()

    for i in range(args.warmup):
        step(1000 + i)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.steps):
        step(t, evs[t])
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    f_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    b_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    bf = 2 + 4 + 2  # W and logits read, W_soft written
    _, bb = algorithmic_bytes(n, m)
    ff = forward_soft_flops(n)
    f_gbps = bf * numel / (f_ms * 1e-3) / 1e9
    f_tflops = ff * numel / (f_ms * 1e-3) / 1e12
    print(f"# soft step: {el * 1e3 / args.steps:.3f} ms/step, soft fwd {f_ms:.3f} ms "
          f"({f_gbps:.0f} GB/s, {f_tflops:.1f} TFLOP/s), bwd {b_ms:.3f} ms", file=sys.stderr,
          flush=True)
    rooflines = step_rooflines(work.name, n, m, numel, f_ms, b_ms, None, fwd_bytes=bf)
    out = {"metric": "masked weights/sec (pure soft forward + backward)",
           "value": numel * args.steps / el, "unit": "masked weights/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": el * 1e3 / args.steps,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (as the default mode)",
           "config": {"workload": work.name, "masked_weights": numel, "pattern": f"{n}:{m}",
                      "forward": "pure soft, W_soft = bf16(W * S)"},
           "kernels": {
               "roi_mask_fwd_soft": {
                   "avg_ms": f_ms, "algorithmic_bytes_per_weight": bf, "GBps": f_gbps,
                   "hbm_frac": f_gbps / HBM_PEAK_GBPS, "flops_per_weight": ff,
                   "TFLOPs": f_tflops, "alu_frac": f_tflops / FP32_VECTOR_PEAK_TFLOPS},
               "roi_mask_bwd": {"avg_ms": b_ms, "algorithmic_bytes_per_weight": bb,
                                "GBps": bb * numel / (b_ms * 1e-3) / 1e9}},
           **rooflines}
    print(json.dumps(out), flush=True)
    return 0


def run_adamw(args) -> int:
    """--mode adamw: the training step with the optimizer, as the appendix
    trains the logits: forward (masked weights + indices) and the backward with
    one AdamW step fused in (beta 0.9 / 0.95, weight decay 0.05, the learning
    rate annealed 1e-3 -> 1e-4 like the temperatures).  For comparison, the
    same step unfused: roi_mask_bwd, then PyTorch's fused AdamW kernel over the
    per-tensor views of the logits."""
    import torch

    import paper_2608_23048_amd as roi
    from paper_2608_23048_amd import workloads as wl

    roi.lib()
    work = wl.WORKLOADS[args.workload]
    n, m = work.n, work.m
    dev = torch.device("cuda:0")
    numel = work.numel
    print(f"# adamw mode, workload {work.name}: {numel} weights, {n}:{m}", file=sys.stderr,
          flush=True)
    W, L, G = wl.fill_slab(work, dev, step=0)
    Wm = torch.empty_like(W)
    idx = torch.empty((numel // m, n), dtype=torch.uint8, device=dev)
    mom = torch.zeros_like(L)
    sec = torch.zeros_like(L)
    sched = work.tau_schedule or (work.tau, work.tau, 1)
    T = sched[2]

    def tau_at(t):
        return roi.anneal(sched[0], sched[1], t, T)

    def lr_at(t):
        return roi.anneal(1e-3, 1e-4, t, T)

    def fused_step(t, ev=None):
        tau = tau_at(t)
        if ev is not None:
            ev[0].record()
        roi.mask_fwd(W, L, n, m, tau, 1.0, 0, t, 0, out={"W_masked": Wm, "sel_idx": idx})
        if ev is not None:
            ev[1].record()
        roi.mask_bwd_adamw(G, W, L, mom, sec, n, m, tau, 1.0, 0, t, 0,
                           opt=roi.adamw_params(lr_at(t), t=t + 1))
        if ev is not None:
            ev[2].record()

    def timed(fn, steps):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(steps):
            fn(t, evs[t])
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        f = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
        b = sum(e[1].elapsed_time(e[2]) for e in evs) / steps
        return el, f, b

    for i in range(args.warmup):
        fused_step(i)
    el, f_ms, b_ms = timed(fused_step, args.steps)
    bf, _ = algorithmic_bytes(n, m)
    bb = 2 + 2 + 4 + 4 + 4 + 4 + 4 + 4  # G, W, logits, m, v read; logits, m, v written
    b_gbps = bb * numel / (b_ms * 1e-3) / 1e9
    print(f"# fused: {el * 1e3 / args.steps:.3f} ms/step, fwd {f_ms:.3f} ms, bwd+AdamW "
          f"{b_ms:.3f} ms ({b_gbps:.0f} GB/s)", file=sys.stderr, flush=True)

    # unfused: roi_mask_bwd, then PyTorch's fused AdamW over the per-tensor views
    dphi = torch.empty_like(L)
    views = lambda x: [x[t.offset:t.offset + t.numel].view(t.rows, t.cols) for t in work.tensors]
    Lv, Dv, Mv, Sv = views(L), views(dphi), views(mom), views(sec)

    # PyTorch's fused AdamW reads the (already incremented) step count per tensor
    step_tensors = [[torch.full((), float(t + 1), device=dev) for _ in Lv]
                    for t in range(max(args.steps, 1))]

    def unfused_step(t, ev=None):
        tau = tau_at(t)
        if ev is not None:
            ev[0].record()
        roi.mask_fwd(W, L, n, m, tau, 1.0, 0, t, 0, out={"W_masked": Wm, "sel_idx": idx})
        if ev is not None:
            ev[1].record()
        roi.mask_bwd(G, W, L, n, m, tau, 1.0, 0, t, 0, out=dphi)
        torch._fused_adamw_(Lv, Dv, Mv, Sv, [], step_tensors[t], lr=lr_at(t), beta1=0.9,
                            beta2=0.95,
                            weight_decay=0.05, eps=1e-8, amsgrad=False, maximize=False)
        if ev is not None:
            ev[2].record()

    unfused_step(0)
    uel, uf_ms, ub_ms = timed(unfused_step, args.steps)
    print(f"# unfused: {uel * 1e3 / args.steps:.3f} ms/step, fwd {uf_ms:.3f} ms, bwd + torch "
          f"AdamW {ub_ms:.3f} ms", file=sys.stderr, flush=True)
    value = numel * args.steps / el
    out = {
        "metric": "masked weights/sec (mask fwd + bwd with fused AdamW on the logits), "
                  "7B-class 2:4",
        "value": value, "unit": "masked weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": el * 1e3 / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (as the default mode); AdamW moments start at zero",
        "config": {"workload": work.name, "masked_weights": numel, "pattern": f"{n}:{m}",
                   "optimizer": "AdamW beta=(0.9, 0.95) wd=0.05 eps=1e-8, "
                                "lr 1e-3->1e-4 exponential", "launches_per_step": 2},
        "kernels": {"roi_mask_fwd": {"avg_ms": f_ms, "algorithmic_bytes_per_weight": bf},
                    "roi_mask_bwd_adamw": {"avg_ms": b_ms, "algorithmic_bytes_per_weight": bb,
                                           "GBps": b_gbps}},
        "roofline": {"kernel": "roi_mask_bwd_adamw", "bound": "hbm", "achieved": b_gbps,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": b_gbps / HBM_PEAK_GBPS,
                     "traffic": None},
        "unfused": {"ms_per_step": uel * 1e3 / args.steps, "fwd_ms": uf_ms,
                    "bwd_plus_torch_fused_adamw_ms": ub_ms,
                    "algorithmic_bytes_per_weight": 12 + 28},
    }
    print(json.dumps(out), flush=True)
    return 0


def run_export(args) -> int:
    """--mode export: the final-mask export after training over the whole stack
    (top-n of the logits; compressed bf16 values and, for 2:4, the 2-bit index
    metadata: what a 2:4 sparse deployment loads)."""
    import torch

    import paper_2608_23048_amd as roi
    from paper_2608_23048_amd import workloads as wl

    roi.lib()
    work = wl.WORKLOADS[args.workload]
    n, m = work.n, work.m
    numel = work.numel
    W, L, G = wl.fill_slab(work, torch.device("cuda:0"))
    del G
    meta = n == 2 and m == 4
    print(f"# export mode, workload {work.name}: {numel} weights, {n}:{m}", file=sys.stderr,
          flush=True)
    for _ in range(max(args.warmup, 1)):
        out = roi.mask_export(L, W, n, m, want_dense=False, want_idx=False, want_meta=meta)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    keep = []
    for e0, e1 in evs:
        e0.record()
        keep.append(roi.mask_export(L, W, n, m, want_dense=False, want_idx=False,
                                    want_meta=meta))
        e1.record()
        keep = keep[-1:]
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
    bpw = 4 + 2 + 2 * n / m + (1.0 / 8 if meta else 0.0)
    gbps = bpw * numel / (ms * 1e-3) / 1e9
    print(f"# export: {ms:.3f} ms ({gbps:.0f} GB/s)", file=sys.stderr, flush=True)
    out = {"metric": "masked weights/sec (final-mask export: compressed values + metadata)",
           "value": numel / (ms * 1e-3), "unit": "masked weights/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (as the default mode)",
           "config": {"workload": work.name, "masked_weights": numel, "pattern": f"{n}:{m}",
                      "outputs": "values bf16 [G, n]" + (" + meta uint32" if meta else "")},
           "roofline": {"kernel": "roi_mask_export", "bound": "hbm", "achieved": gbps,
                        "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbps / HBM_PEAK_GBPS,
                        "traffic": None, "algorithmic_bytes_per_weight": bpw}}
    print(json.dumps(out), flush=True)
    return 0


def run_cat(args) -> int:
    """--mode cat: the categorical sampler (one logit per candidate mask, the
    parameterization the paper compares with) against the item sampler on the
    same stack and pattern (--pattern n:m), one forward + one backward each."""
    import torch

    import paper_2608_23048_amd as roi
    from paper_2608_23048_amd import workloads as wl

    roi.lib()
    work = wl.WORKLOADS[args.workload]
    n, m = (int(x) for x in (args.pattern or f"{work.n}:{work.m}").split(":"))
    C = roi.cat_num_candidates(n, m)
    numel = work.numel
    dev = torch.device("cuda:0")
    print(f"# cat mode, workload {work.name}: {numel} weights, {n}:{m}, {C} logits per group",
          file=sys.stderr, flush=True)
    W, L, G = wl.fill_slab(work, dev)
    Wm = torch.empty_like(W)

    def timed(fwd, bwd):
        for t in range(max(args.warmup, 1)):
            fwd(t), bwd(t)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(args.steps):
            ev[t][0].record()
            fwd(t)
            ev[t][1].record()
            bwd(t)
            ev[t][2].record()
        torch.cuda.synchronize()
        el = (time.perf_counter() - t0) * 1e3 / args.steps
        return (el, sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps,
                sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps)

    tau = work.tau
    idx = torch.empty((numel // m, n), dtype=torch.uint8, device=dev)
    dphi = torch.empty_like(L)
    roi_ms = timed(lambda t: roi.mask_fwd(W, L, n, m, tau, 1.0, 0, t, 0,
                                          out={"W_masked": Wm, "sel_idx": idx}),
                   lambda t: roi.mask_bwd(G, W, L, n, m, tau, 1.0, 0, t, 0, out=dphi))
    del L, dphi, idx
    torch.cuda.empty_cache()
    print(f"# item sampler: {roi_ms[0]:.3f} ms/step (fwd {roi_ms[1]:.3f}, bwd {roi_ms[2]:.3f})",
          file=sys.stderr, flush=True)
    ngroups = numel // m
    A = torch.empty((ngroups, C), dtype=torch.float32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(4_000_000)
    A.normal_(0.0, 1.0, generator=gen)
    dA = torch.empty_like(A)
    ch = torch.empty(ngroups, dtype=torch.uint8, device=dev)
    cat_ms = timed(lambda t: roi.cat_mask_fwd(W, A, n, m, tau, 1.0, 0, t, 0,
                                              out={"W_masked": Wm, "choice": ch}),
                   lambda t: roi.cat_mask_bwd(G, W, A, n, m, tau, 1.0, 0, t, 0, out=dA))
    print(f"# categorical sampler: {cat_ms[0]:.3f} ms/step (fwd {cat_ms[1]:.3f}, bwd "
          f"{cat_ms[2]:.3f})", file=sys.stderr, flush=True)
    cb_f = 2 + 4 * C / m + 2 + 1 / m
    cb_b = 2 + 2 + 8 * C / m
    bf, bb = algorithmic_bytes(n, m)
    out = {"metric": f"masked weights/sec (categorical sampler fwd+bwd), {work.name} {n}:{m}",
           "value": numel / (cat_ms[0] * 1e-3), "unit": "masked weights/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": cat_ms[0],
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (as the default mode; categorical logits ~N(0,1))",
           "config": {"workload": work.name, "masked_weights": numel, "pattern": f"{n}:{m}",
                      "logits_per_weight": {"categorical": C / m, "item": 1.0}},
           "categorical": {"fwd_ms": cat_ms[1], "bwd_ms": cat_ms[2],
                           "bytes_per_weight": {"fwd": cb_f, "bwd": cb_b},
                           "GBps": {"fwd": cb_f * numel / cat_ms[1] / 1e6,
                                    "bwd": cb_b * numel / cat_ms[2] / 1e6}},
           "item": {"ms_per_step": roi_ms[0], "fwd_ms": roi_ms[1], "bwd_ms": roi_ms[2],
                    "bytes_per_weight": {"fwd": bf, "bwd": bb}}}
    print(json.dumps(out), flush=True)
    return 0


def grouped_timing(grouped_step, steps, work):
    """Times `steps` steps through the grouped calls (after one warm-up)."""
    import torch
    grouped_step(1000)
    gev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    g0 = time.perf_counter()
    for t in range(steps):
        grouped_step(t, gev[t])
    torch.cuda.synchronize()
    g_elapsed = time.perf_counter() - g0
    g_fwd = sum(e[0].elapsed_time(e[1]) for e in gev) / len(gev)
    g_bwd = sum(e[1].elapsed_time(e[2]) for e in gev) / len(gev)
    per_launch = 32  # pieces per grid (common.hpp kMaxPieces)
    grouped = {"ms_per_step": g_elapsed * 1e3 / steps, "fwd_ms": g_fwd, "bwd_ms": g_bwd,
               "descriptors": len(work.tensors),
               "launches_per_step": 2 * -(-len(work.tensors) // per_launch)}
    print(f"# grouped calls over {len(work.tensors)} tensors: {grouped['ms_per_step']:.3f} "
          f"ms/step, fwd {g_fwd:.3f} ms, bwd {g_bwd:.3f} ms", file=sys.stderr, flush=True)
    return grouped


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="qwen2.5-7b-stack-2:4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-grouped", action="store_true",
                    help="skip the secondary timing through the grouped calls")
    ap.add_argument("--pattern", default=None, help="n:m for --mode cat (default: the workload's)")
    ap.add_argument("--mode", choices=("st", "soft", "adamw", "export", "cat"), default="st",
                    help="st: forward + backward (the headline); soft: the pure soft forward "
                         "(no straight-through) + backward; adamw: forward + backward "
                         "with the AdamW step on the logits fused in; export: the final-mask "
                         "export after training; cat: the categorical sampler against the item "
                         "sampler")
    ap.add_argument("--counter-calibration", type=int, metavar="BYTES",
                    help="only run three kernels that move BYTES (copy, read, write): the "
                         "known-size references of the traffic counters")
    ap.add_argument("--valu-summary", metavar="INSTS_CSV",
                    help="add the workload's VALU counters (rocprofv3 --pmc SQ_INSTS_VALU "
                         "SQ_INSTS_VALU_TRANS_F32 SQ_WAVES) to the committed record")
    ap.add_argument("--traffic-summary", nargs=7,
                    metavar=("B_FETCH", "B_WRITE", "B_READS", "C_FETCH", "C_WRITE", "C_READS",
                             "BYTES"),
                    help="write the traffic record from the rocprofv3 --pmc CSVs of the "
                         "counter passes (benchmark, then calibration) and the calibration size")
    args = ap.parse_args()
    if args.counter_calibration:
        return counter_calibration(args.counter_calibration)
    if args.valu_summary:
        return valu_summary(args.valu_summary, args.workload)
    if args.traffic_summary:
        from paper_2608_23048_amd import workloads as wl
        work = wl.WORKLOADS[args.workload]
        t = args.traffic_summary
        return traffic_summary(t[0:3], t[3:6], int(t[6]), work.numel, work.n, work.m)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the sampler needs no collectives, and the "
              "benchmark runs and reports a single MI355X (pass --gpus 1).", file=sys.stderr)
        return 2

    if args.mode == "soft":
        return run_soft(args)
    if args.mode == "adamw":
        return run_adamw(args)
    if args.mode == "export":
        return run_export(args)
    if args.mode == "cat":
        return run_cat(args)

    import torch

    import paper_2608_23048_amd as roi
    from paper_2608_23048_amd import workloads as wl

    roi.lib()  # raises if the HIP library is not built
    work = wl.WORKLOADS[args.workload]
    n, m = work.n, work.m
    dev = torch.device("cuda:0")
    numel = work.numel
    print(f"# workload {work.name}: {len(work.tensors)} tensors, {numel} weights, {n}:{m}",
          file=sys.stderr, flush=True)
    W, L, G = wl.fill_slab(work, dev, step=0)
    Wm = torch.empty_like(W)
    idx = torch.empty((numel // m, n), dtype=torch.uint8, device=dev)
    dphi = torch.empty_like(L)
    torch.cuda.synchronize()

    def tau_at(t: int) -> float:
        if work.tau_schedule is None:
            return work.tau
        a, b, T = work.tau_schedule
        return roi.anneal(a, b, t, T)

    def step(t: int, ev=None):
        tau = tau_at(t)
        if ev is not None:
            ev[0].record()
        roi.mask_fwd(W, L, n, m, tau, 1.0, 0, t, 0, want_soft=False, want_idx=True,
                     out={"W_masked": Wm, "sel_idx": idx})
        if ev is not None:
            ev[1].record()
        roi.mask_bwd(G, W, L, n, m, tau, 1.0, 0, t, 0, out=dphi)
        if ev is not None:
            ev[2].record()

    for i in range(args.warmup):
        step(1000 + i)
    torch.cuda.synchronize()
    print(f"# warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.steps):
        step(t, events[t])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    fwd_ms = [e[0].elapsed_time(e[1]) for e in events]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in events]
    fwd_avg = sum(fwd_ms) / len(fwd_ms)
    bwd_avg = sum(bwd_ms) / len(bwd_ms)
    bf, bb = algorithmic_bytes(n, m)
    fwd_gbps = bf * numel / (fwd_avg * 1e-3) / 1e9
    bwd_gbps = bb * numel / (bwd_avg * 1e-3) / 1e9
    traffic = None
    rec = measured_traffic() if work.name == "qwen2.5-7b-stack-2:4" else None
    if rec is not None:
        key = "bwd_lane_kernel" if bwd_avg >= fwd_avg else "fwd_lane_kernel"
        if key in rec["kernels"]:
            traffic = rec["kernels"][key]["traffic_bytes"]
    rooflines = step_rooflines(work.name, n, m, numel, fwd_avg, bwd_avg, traffic)
    value = numel * args.steps / elapsed
    ms_per_step = elapsed * 1e3 / args.steps
    print(f"# timed {args.steps} steps: {ms_per_step:.3f} ms/step, fwd {fwd_avg:.3f} ms "
          f"({fwd_gbps:.0f} GB/s), bwd {bwd_avg:.3f} ms ({bwd_gbps:.0f} GB/s)", file=sys.stderr,
          flush=True)

    # The same step through the grouped entry points, one descriptor per tensor
    # (the layout of a model whose linear layers are separate tensors): a
    # secondary figure, timed after the headline steps.
    views = []
    for t in work.tensors:
        sl = slice(t.offset, t.offset + t.numel)
        views.append((W[sl].view(t.rows, t.cols), L[sl].view(t.rows, t.cols),
                      G[sl].view(t.rows, t.cols), Wm[sl].view(t.rows, t.cols),
                      idx[t.offset // m:(t.offset + t.numel) // m],
                      dphi[sl].view(t.rows, t.cols)))
    fwd_in = [(v[0], v[1]) for v in views]
    fwd_out = [(v[3], None, v[4]) for v in views]
    bwd_in = [(v[2], v[0], v[1]) for v in views]
    bwd_out = [v[5] for v in views]
    offs = [t.offset for t in work.tensors]

    def grouped_step(t: int, ev=None):
        tau = tau_at(t)
        if ev is not None:
            ev[0].record()
        roi.mask_fwd_grouped(fwd_in, n, m, tau, 1.0, 0, t, offsets=offs, outs=fwd_out)
        if ev is not None:
            ev[1].record()
        roi.mask_bwd_grouped(bwd_in, n, m, tau, 1.0, 0, t, offsets=offs, outs=bwd_out)
        if ev is not None:
            ev[2].record()

    grouped = None
    if not args.no_grouped:
        grouped = grouped_timing(grouped_step, args.steps, work)

    copy = copy_reference()
    rooflines["roofline"]["copy_reference"] = copy
    if rooflines["roofline"]["bound"] == "hbm":
        rooflines["roofline"]["frac_of_copy"] = rooflines["roofline"]["achieved"] / copy["GBps"]
    print(f"# device copy: {copy['GBps']:.0f} GB/s", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(W, L, G, work, n, m, tau_at(0))

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "masked weights/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded W~N(0,0.02^2) bf16, logits~N(0,1) fp32, "
                "grad~N(0,1e-6) bf16; Qwen2.5 shapes only)",
        "config": {
            "workload": work.name,
            "tensors": len(work.tensors),
            "masked_weights": numel,
            "pattern": f"{n}:{m}",
            "tau": (f"{work.tau_schedule[0]}->{work.tau_schedule[1]} exponential over "
                    f"{work.tau_schedule[2] + 1} steps" if work.tau_schedule else work.tau),
            "lambda": 1.0,
            "launches_per_step": 2,
        },
        "step_algorithmic_GBps": (bf + bb) * value / 1e9,
        "kernels": {
            "roi_mask_fwd": {"avg_ms": fwd_avg, "algorithmic_bytes_per_weight": bf,
                             "GBps": fwd_gbps},
            "roi_mask_bwd": {"avg_ms": bwd_avg, "algorithmic_bytes_per_weight": bb,
                             "GBps": bwd_gbps},
        },
        **rooflines,
        "cpu_baseline": cpu,
        "grouped_calls": grouped,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
