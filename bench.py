"""Benchmark: Horovod-style fused ring-allreduce of N simulated ranks on one MI355X.

One step = one allreduce (AVERAGE) of every rank's gradient tensors: the Tensor
Fusion plan's copy-in, the ring's N-1 reduce-scatter and N-1 all-gather steps,
and the copy-out, for every fusion buffer, with inputs already in GPU memory.
The metric is algorithm bandwidth: one rank's fp32 gradient bytes / step time.

    python bench.py [--steps K] [--warmup W] [--workload vgg16] [--no-per-config]

Prints one JSON line.  The headline workload is VGG-16 (32 ranks, 138M parameters,
553 MB of gradients per rank), the largest binary32 one, whose per-step working
sets are several times the 256 MB Infinity Cache.  Besides the headline workload it
reports, per workload, the step time and the per-kernel time split measured with
HIP events; the roofline object is for the kernel with the largest share of the
step (HBM-bound: achieved algorithmic bytes / time against the 8 TB/s peak), and
`ring_roofline` the same for the ring's adding and replacing step kernels together.
`cpu_baseline` times the C oracle on the same whole workload on this host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
TILED_REPLACE_IN_TENSORS, TILED_ADD_FROM_TENSORS = 1, 2  # the HVDX_TILED_* bits of FusedAllreduce.tiled_flags
# FusedAllreduce arguments of each way of running the fusion buffers
BUFFER_MODES = {"ring_on_tensors": {}, "copy_in": {"add_from_tensors": False},
                "paper_copies": {"replace_in_tensors": False}}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="vgg16")
    p.add_argument("--broadcast-workload", default="resnet50",
                   help="workload whose parameters the broadcast measurement sends (161 tensors for ResNet-50)")
    p.add_argument("--no-per-config", action="store_true", help="time only the headline workload")
    p.add_argument("--fusion-buffer-mode", default="ring_on_tensors", choices=sorted(BUFFER_MODES),
                   help="how the headline workload's fusion buffers run: the ring on the tensors (default), the "
                        "copy-in kept, or the paper's copies around a ring in the buffers (same bits)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-ablation", action="store_true", help="skip the fusion-threshold sweep")
    p.add_argument("--no-broadcast", action="store_true", help="skip the broadcast measurement")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target oracle time for the CPU baseline")
    p.add_argument("--calibration-copy-mib", type=int, default=0,
                   help="first run 3 plain device copies of this many MiB (a known-traffic kernel for counters)")
    p.add_argument("--oracle-configs", metavar="NAMES",
                   help="time only the C oracle on these workloads (comma-separated, whole, host cores) and exit")
    p.add_argument("--summarize-profiles", metavar="DIR",
                   help="no GPU: summarize rocprofv3 output under DIR (prof_*/ kernel stats, pmc_fetch/, pmc_write/) "
                        "into profiles/")
    return p.parse_args()


def kernel_bytes(ar, kind, bi, step):
    """Algorithmic HBM bytes one launch must move (reads + writes); a launch that serves
    two buckets' rings (bi a pair of indices) moves the sum of both."""
    if isinstance(bi, tuple):
        return sum(kernel_bytes(ar, kind, x, step) for x in bi)
    b = ar.buckets[bi]
    n = ar.nranks
    es_t = 4 if ar.dtype == 0 else 2  # tensor element size
    es_b = 4 if ar.buf_dtype == 0 else 2  # buffer element size
    data = sum(ar.numel[t] for t in b.tensors)
    if kind == "pack":
        return n * (es_t * data + es_b * b.count)
    if kind == "pack_rs":  # the adding step reuses the values it packs; no rank stores its own sent chunk
        return n * es_t * data + (n - 1) * es_b * b.count
    if kind in ("cycle_small", "ring_small"):  # every step's messages, as the per-step kernels count them
        es = es_t if b.direct else es_b
        ring = (n - 1) * 5 * es * b.count
        return ring if b.direct else ring + n * (es_t * data + es_b * b.count) + n * (es_b + es_t) * data
    if kind in ("unpack", "ag_unpack"):  # the fused replacing step only changes which buffer is read
        return n * (es_b + es_t) * data
    compressed = b.direct and ar.compress
    flags = 0 if b.direct else ar.tiled_flags
    if flags & TILED_ADD_FROM_TENSORS and kind == "rs":  # the receiver's own elements from its tensors
        if step == 0:  # the sender's too: two tensors in, the receiver's buffer out
            return (2 * es_t + es_b) * data
        return (es_t + 2 * es_b) * data  # the sender's buffer in; tensors' elements only, no padding
    if flags & TILED_REPLACE_IN_TENSORS and kind in ("rs_ag", "ag"):
        # replacing steps into the tensors: the tensors' elements only
        if kind == "rs_ag":  # owner's values and sender's buffer in, owner's and the next rank's tensors out
            own = es_t if flags & TILED_ADD_FROM_TENSORS else es_b
            return (own + es_b + 2 * es_t) * data
        return 2 * es_t * data  # sender's tensors in, receiver's out
    if kind == "rs_ag":  # read owner and sender, write owner and the next rank
        if compressed:  # binary32 owner, binary16 sender (binary32 when N = 2: its first touch)
            return (16 if n == 2 else 14) * b.count
        return 4 * (es_t if b.direct else es_b) * b.count
    if kind == "rs":
        if compressed:
            return (10 if step == 0 else 8) * b.count
        return 3 * es_b * b.count if not b.direct else 3 * es_t * b.count
    if kind == "ag":
        if compressed:  # step 0 widens the owner's binary16 into two buffers; later steps copy binary32
            return (10 if step == 0 else 8) * b.count
        return 2 * es_b * b.count if not b.direct else 2 * es_t * b.count
    if kind == "fold":  # every rank's value read once and the result written to every rank
        return 2 * n * (es_t if b.direct else es_b) * b.count
    return 0


KIND_CODE = {"pack": 0, "rs": 1, "ag": 2, "unpack": 3, "ring": 4, "rs_ag": 6, "fold": 7, "pack_rs": 8,
             "ag_unpack": 9, "ring_small": 10, "cycle_small": 11}


def kernel_name(ar, kind, bi):
    b = ar.buckets[bi[0] if isinstance(bi, tuple) else bi]
    if kind in ("cycle_small", "ring_small"):
        return kind
    if kind in ("rs", "ag", "rs_ag"):
        flags = 0 if b.direct else ar.tiled_flags
        # a compressed bucket's steps that read or write binary32 tensors are the compressed ring's
        tensor_side = flags & TILED_ADD_FROM_TENSORS if kind == "rs" else flags & TILED_REPLACE_IN_TENSORS
        if ar.compress and (b.direct or tensor_side):
            return f"{kind}_step_c16"
        return f"{kind}_step_{'f16' if (ar.buf_dtype == 1 and not b.direct) else 'f32'}"
    return kind


def time_graph(ar, steps, stream):
    """ms per allreduce replaying one HIP graph of the whole cycle `steps` times."""
    import torch

    graph = ar.capture()
    for _ in range(2):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    del graph
    return e0.elapsed_time(e1) / steps


MALL_FLUSH_BYTES = 1 << 30  # written between allreduces: 4x the 256 MB Infinity Cache


def measure(name, steps, warmup, threshold=64 << 20, per_kernel_pass=True, schedule="ring", graph_pass=True,
            flush_bytes=0, **modes):
    """Time `steps` allreduces of workload `name`.  With flush_bytes, a buffer that
    large is overwritten before every allreduce (outside its timing), so each one
    starts with none of its data in the Infinity Cache; each allreduce then has its
    own event pair and the median is reported."""
    import torch

    import paper_1802_05799_amd as hv
    from workloads import configs
    from workloads import gpu as wgpu

    w = configs.get(name)
    per_rank, storage, starts = wgpu.make_rank_tensors(w)
    ar = hv.FusedAllreduce(per_rank, op=w.op, compress=w.compress, threshold_bytes=threshold, schedule=schedule,
                           **modes)
    stream = torch.cuda.current_stream()
    sid = stream.cuda_stream
    scratch = torch.empty(flush_bytes // 4, dtype=torch.float32, device="cuda") if flush_bytes else None

    def flush(i):
        if scratch is not None:
            scratch.fill_(float(i))

    for i in range(warmup):
        flush(i)
        ar(sid)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    if scratch is None:
        # timed region: exactly `steps` whole allreduces, one event pair around them
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            ar(sid)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
    else:
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for i, (a, b) in enumerate(ev):
            flush(i)
            a.record(stream)
            ar(sid)
            b.record(stream)
        torch.cuda.synchronize()
        ms = sorted(a.elapsed_time(b) for a, b in ev)[steps // 2]
    wall = time.perf_counter() - t0
    # the same cycle submitted as one HIP graph per step (launch overhead removed)
    graph_ms = time_graph(ar, steps, stream) if graph_pass and scratch is None else None
    if not per_kernel_pass:
        res = {"ms_per_step": ms, "algbw_GBps": w.rank_bytes / (ms * 1e-3) / 1e9, "buckets": len(ar.buckets),
               "launches_per_step": len(ar.kernel_sequence()), "graph_ms_per_step": graph_ms}
        del ar, per_rank, storage
        torch.cuda.empty_cache()
        return res

    # the same steps once more with every launch timed by its own dispatch (the
    # library hands timeline events to hipExtLaunchKernel, which stamps them with the
    # kernel's start and end, as a kernel trace does).  Each launch position's median
    # over the timed steps is kept: a sample the host stalled is an outlier.
    seq = ar.kernel_sequence()
    with hv.Timeline(capacity=len(seq) * (steps + 1) + 16) as tl:
        for i in range(steps + 1):
            flush(i)  # not a library launch: no timeline record
            ar(sid)
    recs = tl.records
    if tl.dropped or len(recs) != len(seq) * (steps + 1):
        raise RuntimeError(f"timeline recorded {len(recs)} launches for {steps + 1} steps of {len(seq)}")
    if [KIND_CODE[k] for k, _bi, _st in seq] != [r["kind"] for r in recs[:len(seq)]]:
        raise RuntimeError("timeline records do not follow the expected launch order")
    per_kernel = {}
    outliers = 0
    for j, (kind, bi, st) in enumerate(seq):
        samples = sorted(recs[i * len(seq) + j]["duration_us"] / 1000.0 for i in range(1, steps + 1))
        med = samples[len(samples) // 2]
        outliers += sum(1 for x in samples if x > 1.5 * med)
        d = per_kernel.setdefault(kernel_name(ar, kind, bi), {"launches": 0, "ms": 0.0, "bytes": 0})
        d["launches"] += steps
        d["ms"] += med * steps
        d["bytes"] += kernel_bytes(ar, kind, bi, st) * steps
    traced_ms = sum(d["ms"] for d in per_kernel.values()) / steps
    for d in per_kernel.values():
        d["avg_us"] = 1000.0 * d["ms"] / d["launches"]
        d["GBps"] = d["bytes"] / (d["ms"] * 1e-3) / 1e9 if d["ms"] > 0 else None
        d["hbm_frac"] = d["GBps"] / HBM_PEAK_GBS if d["GBps"] else None
        d["share"] = d["ms"] / (traced_ms * steps)
        d["ms_per_step"] = d["ms"] / steps
        del d["ms"]
    res = {
        "workload": name,
        "nranks": w.nranks,
        "steps": steps,
        "ms_per_step": ms,
        "algbw_GBps": w.rank_bytes / (ms * 1e-3) / 1e9,
        "busbw_GBps": w.rank_bytes / (ms * 1e-3) / 1e9 * 2 * (w.nranks - 1) / w.nranks,
        "wall_ms_per_step": 1000.0 * wall / steps,
        "graph_ms_per_step": graph_ms,
        "kernels": per_kernel,
        "timing_outliers": outliers,
        "buckets": [(b.count, len(b.tensors), b.direct) for b in ar.buckets],
    }
    del ar, per_rank, storage, scratch
    torch.cuda.empty_cache()
    return res


def hbm_fracs(r):
    """HBM fraction (algorithmic bytes over time) of the ring's kernels alone and of
    the whole step."""
    ring = [v for k, v in r["kernels"].items() if k.startswith(("rs_step", "ag_step", "rs_ag_step"))]
    ring_bytes = sum(v["bytes"] for v in ring) / r["steps"]  # per step
    ring_ms = sum(v["ms_per_step"] for v in ring)
    path_bytes = sum(v["bytes"] for v in r["kernels"].values()) / r["steps"]
    return (round(ring_bytes / (ring_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if ring_ms else None,
            round(path_bytes / (r["ms_per_step"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))


def measure_broadcast(name, steps, warmup=2):
    """Rank 0's parameters to every rank (paper sections 4 and 5): broadcast_ (every
    tensor in one chain, descriptor tables built and uploaded per call), the same with
    the tables prepared once (TensorBroadcast), one hvdx_broadcast chain per tensor, and
    one chain over each rank's whole contiguous parameter storage."""
    import torch

    import paper_1802_05799_amd as hv
    from workloads import configs
    from workloads import gpu as wgpu

    w = configs.get(name)
    per_rank, storage, starts = wgpu.make_rank_tensors(w)
    stream = torch.cuda.current_stream()
    sid = stream.cuda_stream
    flat_ptrs = [x.data_ptr() for x in storage]
    flat_bytes = storage[0].numel() * 4

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    def per_tensor_chains():
        for ts in zip(*per_rank):
            hv.hvdx_broadcast([x.data_ptr() for x in ts], w.nranks, ts[0].numel() * ts[0].element_size(), 0, sid)

    prepared = hv.TensorBroadcast(per_rank)
    ms_call = timed(lambda: hv.broadcast_(per_rank, 0))
    ms_prepared = timed(lambda: prepared(0, sid))
    ms_tensors = timed(per_tensor_chains)
    ms_flat = timed(lambda: hv.hvdx_broadcast(flat_ptrs, w.nranks, flat_bytes, 0, sid))
    moved = 2 * (w.nranks - 1) * w.rank_bytes  # every non-root rank reads and writes each byte once
    res = {
        "workload": name,
        "tensors": len(w.numel()),
        "call_ms": round(ms_call, 4),
        "call_algbw_GBps": round(w.rank_bytes / (ms_call * 1e-3) / 1e9, 2),
        "prepared_ms": round(ms_prepared, 4),
        "prepared_hbm_GBps": round(moved / (ms_prepared * 1e-3) / 1e9, 1),
        "per_tensor_chains_ms": round(ms_tensors, 4),
        "flat_ms": round(ms_flat, 4),
        "flat_hbm_GBps": round(2 * (w.nranks - 1) * flat_bytes / (ms_flat * 1e-3) / 1e9, 1),
        "launches_per_call": 2 * w.nranks - 2,
    }
    del per_rank, storage, prepared
    torch.cuda.empty_cache()
    return res


def kernel_source_hash():
    """Hash of the kernel sources' code, with // comments and blank lines dropped, so
    the counter traffic recorded in profiles/traffic.json is tied to the code it was
    measured on and not to the wording of its comments."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_1802_05799_amd", "csrc")
    for f in sorted(os.listdir(d)):
        h.update(f.encode() + b"\n")
        with open(os.path.join(d, f)) as fh:
            for line in fh:
                code = line.split("//")[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def traffic_for(kernel, workload):
    """Counter-measured HBM bytes per launch, if recorded for the current kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("per_launch_bytes", {}).get(f"{workload}/{kernel}")


def short_kernel_name(full):
    """rocprofv3 kernel name (demangled, or mangled where it holds binary16 template
    arguments) -> the names bench.py reports."""
    import re

    base = full.replace("(anonymous namespace)", "anon").split("(")[0]
    for key, short in (("rs_ag_step_c16_kernel", "rs_ag_step_c16"), ("rs_step_c16_kernel", "rs_step_c16"),
                       ("ag_first_c16_kernel", "ag_first_c16"), ("roundtrip_c16_kernel", "ring"),
                       ("fold_kernel", "fold")):
        if key in base:
            return short
    half = "<_Float16" in base or "IDF16_" in base
    if "small_cycle_kernel" in base:
        return "cycle_small"
    if "chain_kernel" in base:
        return "ring_small"
    # the tile-driven ring steps report as the ring step they are; binary32 tensors with
    # binary16 buffers are the compressed ring's (its replacing steps copy binary32)
    mixed = re.search(r"tiles_kernel<float, _Float16", base) or re.search(r"tiles_kernelIfDF16_", base)
    for key, step in (("rs_ag_tiles_kernel", "rs_ag_step"), ("add_tiles_kernel", "rs_step"),
                      ("ag_tiles_kernel", "ag_step")):
        if key in base:
            return step + ("_c16" if mixed else "_f16" if half else "_f32")
    # a launch serving two fusion buffers' rings reports as the one-ring kernel of its step
    for key in ("rs_ag_step_pair_kernel", "rs_step_pair_kernel", "ag_step_pair_kernel", "rs_ag_step_kernel",
                "rs_step_kernel", "ag_step_kernel"):
        if key in base:
            return key.replace("_pair", "").replace("_kernel", "") + ("_f16" if half else "_f32")
    if "unpack_tiles_kernel" in base:  # tile-driven copies, always fused with a ring step
        return "ag_unpack"
    if "pack_tiles_kernel" in base:
        return "pack_rs"
    if "unpack_pair_kernel" in base:  # two fusion buffers per launch, always fused with a ring step
        return "ag_unpack"
    if "pack_pair_kernel" in base:
        return "pack_rs"
    # the copy kernels' last template argument: fused with a ring step
    ring = base.rstrip().endswith(", true>") or re.search(r"Lb1EEEv", base) is not None
    if "unpack_kernel" in base:
        return "ag_unpack" if ring else "unpack"
    if "pack_kernel" in base:
        return "pack_rs" if ring else "pack"
    return None


def shape_of(full):
    """The launch-shape part of a kernel name (Policy<...> or CopyCfg<...>), for tables;
    " x2" marks a launch that serves two fusion buffers' rings."""
    import re

    two = " x2" if "pair_kernel" in full else ""
    if "tiles_kernel" in full:  # the vectors per lane: the last template argument
        m = re.search(r"tiles_kernel<[^>]*,\s*(\d+)>", full) or re.search(r"tiles_kernelI.*Li(\d+)EEEv", full)
        return f"tiles<{m.group(1)}>" if m else "tiles"
    m = re.search(r"(Policy|CopyCfg)<[^>]*>", full)
    if m:
        return m.group(0).replace(" ", "") + two
    m = re.search(r"(Policy|CopyCfg)I((?:L[ib]\d+E)+)E", full)  # mangled: PolicyILi1ELi64ELb1E...E
    if m:
        return m.group(1) + "<" + ",".join(x[2:] for x in re.findall(r"L[ib]\d+", m.group(2))) + ">" + two
    return ""


def summarize_profiles(d):
    """Per-kernel durations (kernel trace, prof_<workload>/) and HBM bytes per dispatch
    (FETCH_SIZE and WRITE_SIZE runs, pmc_fetch_<workload>/ and pmc_write_<workload>/),
    each counter scaled by what it reads for a plain 1 GiB device copy in the same run.
    Rows are per instantiation (launch shape); the counted bytes over the traced
    average duration give the HBM rate each achieved.  Writes profiles/traffic.json
    (per workload and reported kernel: counted bytes per launch, weighted by launches)."""
    import csv
    import glob

    out_lines, traffic, cal_used = [], {}, {}
    trace = {}  # (workload, full name) -> (calls, total ns)
    for f in sorted(glob.glob(os.path.join(d, "prof_*", "*_kernel_stats.csv"))):
        workload = os.path.basename(os.path.dirname(f))[len("prof_"):]
        for r in csv.DictReader(open(f)):
            if short_kernel_name(r["Name"]):
                trace[(workload, r["Name"])] = (int(r["Calls"]), float(r["TotalDurationNs"]))
    workloads = sorted({w for w, _ in trace} | {os.path.basename(x)[len("pmc_fetch_"):]
                                               for x in glob.glob(os.path.join(d, "pmc_fetch_*")) if os.path.isdir(x)})
    for workload in workloads:
        pmc = {}
        for counter, sub in (("FETCH_SIZE", "pmc_fetch_"), ("WRITE_SIZE", "pmc_write_")):
            files = glob.glob(os.path.join(d, sub + workload, "*_counter_collection.csv"))
            if not files:
                continue
            rows = [r for r in csv.DictReader(open(files[0])) if r["Counter_Name"] == counter]
            cal = [float(r["Counter_Value"]) for r in rows
                   if "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) >= (1 << 17)]
            if not cal:
                continue
            factor = (1 << 20) / (sum(cal) / len(cal))  # a 1 GiB copy reads and writes 2^20 KiB
            per = {}
            for r in rows:
                if short_kernel_name(r["Kernel_Name"]):
                    per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * factor * 1024)
            pmc[counter] = (factor, {k: sum(v) / len(v) for k, v in per.items()})
        names = sorted((n for w, n in trace if w == workload), key=lambda n: -trace[(workload, n)][1])
        # with fp16 compression the binary32 replacing-step kernel runs only as the
        # compressed ring's later replacing steps, which bench.py reports as ag_step_c16
        compressed = any(short_kernel_name(n) == "rs_step_c16" for n in names)

        def short(n):
            k = short_kernel_name(n)
            return "ag_step_c16" if compressed and k == "ag_step_f32" else k

        counted = len(pmc) == 2
        if counted:
            cal_used[workload] = {"FETCH_SIZE": pmc["FETCH_SIZE"][0], "WRITE_SIZE": pmc["WRITE_SIZE"][0]}
        out_lines.append(f"## {workload}\n")
        if counted:
            out_lines.append(f"HBM bytes per dispatch from FETCH_SIZE x {pmc['FETCH_SIZE'][0]:.3f} and WRITE_SIZE x "
                             f"{pmc['WRITE_SIZE'][0]:.3f} (the factors that make a plain 1 GiB device copy read "
                             f"and write 1 GiB); counted rate = those bytes / the traced average duration.\n")
        out_lines.append("| kernel | shape | calls | average us | total ms | fetch MB | write MB | counted GB/s "
                         "| % of 8 TB/s |\n|---|---|---|---|---|---|---|---|---|")
        per_short = {}
        for n in names:
            calls, tot_ns = trace[(workload, n)]
            k, avg_us = short(n), tot_ns / calls / 1e3
            cells = ["-", "-", "-", "-"]
            if counted and n in pmc["FETCH_SIZE"][1]:
                fb, wb = pmc["FETCH_SIZE"][1][n], pmc["WRITE_SIZE"][1].get(n, 0.0)
                rate = (fb + wb) / (avg_us * 1e-6) / 1e9
                cells = [f"{fb / 1e6:.1f}", f"{wb / 1e6:.1f}", f"{rate:.0f}", f"{rate / HBM_PEAK_GBS * 100:.1f}"]
                acc = per_short.setdefault(k, [0.0, 0])
                acc[0] += (fb + wb) * calls
                acc[1] += calls
            out_lines.append(f"| {k} | `{shape_of(n)}` | {calls} | {avg_us:.2f} | {tot_ns / 1e6:.2f} | "
                             + " | ".join(cells) + " |")
        out_lines.append("")
        # the same rows gathered under the names bench.py reports (all launch shapes of a
        # kernel together, weighted by calls), as its per-kernel figures are
        out_lines.append("Per reported kernel (all its launch shapes, weighted by calls):\n")
        out_lines.append("| kernel | calls | average us | total ms | counted MB per launch |\n|---|---|---|---|---|")
        agg = {}
        for n in names:
            calls, tot_ns = trace[(workload, n)]
            a = agg.setdefault(short(n), [0, 0.0])
            a[0] += calls
            a[1] += tot_ns
        for k, (calls, tot_ns) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            mb = f"{per_short[k][0] / per_short[k][1] / 1e6:.1f}" if k in per_short else "-"
            out_lines.append(f"| {k} | {calls} | {tot_ns / calls / 1e3:.2f} | {tot_ns / 1e6:.2f} | {mb} |")
        out_lines.append("")
        for k, (b, c) in per_short.items():
            traffic[f"{workload}/{k}"] = round(b / c)
    if traffic:
        with open(TRAFFIC_FILE, "w") as f:
            json.dump({"source_hash": kernel_source_hash(), "per_launch_bytes": traffic, "calibration": cal_used},
                      f, indent=1)
    return "\n".join(out_lines)


def _oracle_inputs(name):
    """Every rank's tensors of workload `name` in host memory, from the workload's seeded
    generator (run on the GPU, then copied), with preallocated, touched outputs and a
    fusion-buffer workspace for the C oracle."""
    import numpy as np
    import torch

    from oracle import native
    from workloads import configs
    from workloads import gpu as wgpu

    w = configs.get(name)
    numel = w.numel()
    per_rank_dev, storage, starts = wgpu.make_rank_tensors(w, device="cuda:0")
    torch.cuda.synchronize()
    flats = [f.cpu().numpy() for f in storage]
    del per_rank_dev, storage
    torch.cuda.empty_cache()
    inputs = [[flat[s : s + n] for s, n in zip(starts, numel)] for flat in flats]
    out = [[np.ones(n, dtype=np.float32) for n in numel] for _ in range(w.nranks)]  # touched before timing
    ws = np.ones(native.workspace_bytes(numel, w.nranks, compress=w.compress), dtype=np.uint8)
    return w, inputs, out, ws


def _time_oracle(w, inputs, out, ws, threads, target_s):
    """(allreduces, seconds): the C oracle repeated until about target_s seconds."""
    from oracle import native

    reps, spent = 0, 0.0
    while reps == 0 or spent < target_s:
        t0 = time.perf_counter()
        native.allreduce(inputs, w.op, compress=w.compress, threads=threads, out=out, workspace=ws)
        spent += time.perf_counter() - t0
        reps += 1
    return reps, spent


def cpu_baseline(name, target_s):
    """The C oracle (oracle/csrc/oracle.c: plan, copy-in, ring, copy-out) on the whole
    workload: every rank's tensors from the workload's seeded generator, copied to host
    memory; the fusion buffers allocated once, as the paper's step 2 allocates the
    fusion buffer once.  Timed with every thread OpenMP is given (OMP_NUM_THREADS),
    repeated until about target_s seconds, and once with a single thread."""
    from oracle import native

    w, inputs, out, ws = _oracle_inputs(name)
    numel = w.numel()
    threads = native.max_threads()
    _time_oracle(w, inputs, out, ws, threads, 0.0)  # warm-up
    reps, t_threads = _time_oracle(w, inputs, out, ws, threads, target_s)
    _, t_one = _time_oracle(w, inputs, out, ws, 1, 0.0)
    rank_bytes = 4 * sum(numel)
    return {
        "value": rank_bytes * reps / t_threads / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{name} whole: {len(numel)} tensors, {sum(numel)} elements per rank, {w.nranks} ranks; "
        f"C oracle, {threads} OpenMP threads, {reps} allreduces in {t_threads:.1f} s",
        "ms_per_allreduce": 1e3 * t_threads / reps,
        "single_thread": {"value": rank_bytes / t_one / 1e9, "ms_per_allreduce": 1e3 * t_one},
        "host_cpus": os.cpu_count(),
        "host_cpu_model": host_cpu_model(),
    }


def oracle_per_config(names, target_s):
    """The C oracle on every named workload, whole: one warm-up allreduce, then all
    OpenMP threads until about target_s seconds, then one allreduce on one thread."""
    import gc

    from oracle import native

    res = {}
    threads = native.max_threads()
    for name in names:
        print(f"oracle {name}: inputs", file=sys.stderr, flush=True)
        w, inputs, out, ws = _oracle_inputs(name)
        print(f"oracle {name}: warm-up", file=sys.stderr, flush=True)
        _time_oracle(w, inputs, out, ws, threads, 0.0)
        print(f"oracle {name}: {threads} threads", file=sys.stderr, flush=True)
        reps, t_threads = _time_oracle(w, inputs, out, ws, threads, target_s)
        rank_bytes = 4 * sum(w.numel())
        res[name] = {
            "nranks": w.nranks,
            "threads": threads,
            "ms_threads": round(1e3 * t_threads / reps, 3),
            "algbw_threads_GBps": round(rank_bytes * reps / t_threads / 1e9, 4),
            "allreduces": reps,
        }
        # one thread takes up to `threads` times as long; left out where that could pass two minutes
        if t_threads / reps * threads <= 120.0:
            print(f"oracle {name}: one thread", file=sys.stderr, flush=True)
            _, t_one = _time_oracle(w, inputs, out, ws, 1, 0.0)
            res[name]["ms_one_thread"] = round(1e3 * t_one, 3)
            res[name]["algbw_one_thread_GBps"] = round(rank_bytes / t_one / 1e9, 4)
        print(f"oracle {name}: {res[name]}", file=sys.stderr, flush=True)
        del inputs, out, ws
        gc.collect()
    return {"oracle_per_config": res, "host_cpus": os.cpu_count(), "host_cpu_model": host_cpu_model()}


def host_cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    args = parse()
    if args.summarize_profiles:
        print(summarize_profiles(args.summarize_profiles))
        return
    if args.oracle_configs:
        print(json.dumps(oracle_per_config(args.oracle_configs.split(","), args.cpu_seconds)), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(
            "bench.py runs on one GPU: the N simulated ranks live side by side in that GPU's memory, "
            "so there is no multi-GPU mode (run with --gpus 1).",
            file=sys.stderr,
        )
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    if args.calibration_copy_mib:
        n = args.calibration_copy_mib << 18  # float32 elements
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()

    head = measure(args.workload, args.steps, args.warmup, **BUFFER_MODES[args.fusion_buffer_mode])
    print(f"# {args.workload}: {head['ms_per_step']:.3f} ms/step, {head['algbw_GBps']:.1f} GB/s, "
          f"graph {head['graph_ms_per_step']:.3f} ms/step", file=sys.stderr,
          flush=True)
    per_config = {}
    if not args.no_per_config:
        from workloads import configs

        for name in configs.WORKLOADS:
            if name == args.workload and args.fusion_buffer_mode == "ring_on_tensors":
                r = head
            else:
                r = measure(name, max(3, args.steps // 2), 2)
                print(f"# {name}: {r['ms_per_step']:.3f} ms/step, {r['algbw_GBps']:.1f} GB/s, "
                      f"graph {r['graph_ms_per_step']:.3f} ms/step", file=sys.stderr,
                      flush=True)
            ring_frac, path_frac = hbm_fracs(r)
            # the same allreduce started with the Infinity Cache flushed
            f = measure(name, max(3, args.steps // 2), 1, graph_pass=False, flush_bytes=MALL_FLUSH_BYTES)
            f_ring, f_path = hbm_fracs(f)
            print(f"# {name} (cache flushed): {f['ms_per_step']:.3f} ms/step, ring {f_ring}", file=sys.stderr,
                  flush=True)
            per_config[name] = {
                "nranks": r["nranks"],
                "ms_per_step": round(r["ms_per_step"], 4),
                "graph_ms_per_step": r["graph_ms_per_step"] and round(r["graph_ms_per_step"], 4),
                # algorithmic bytes over time: the ring's kernels alone, and the whole step
                "ring_hbm_frac": ring_frac,
                "path_hbm_frac": path_frac,
                "mall_flushed": {"ms_per_step": round(f["ms_per_step"], 4),
                                 "algbw_GBps": round(f["algbw_GBps"], 2),
                                 "ring_hbm_frac": f_ring, "path_hbm_frac": f_path,
                                 "kernels_hbm_frac": {k: v["hbm_frac"] and round(v["hbm_frac"], 4)
                                                      for k, v in f["kernels"].items()}},
                "algbw_GBps": round(r["algbw_GBps"], 2),
                "busbw_GBps": round(r["busbw_GBps"], 2),
                "kernels": {k: {"avg_us": round(v["avg_us"], 2), "GBps": v["GBps"] and round(v["GBps"], 1),
                                "hbm_frac": v["hbm_frac"] and round(v["hbm_frac"], 4),
                                "share": round(v["share"], 4)} for k, v in r["kernels"].items()},
            }

    # the fusion buffers' ring on the tensors (the default) against the paper's copies: the
    # copy-in kept (fused with adding step 0), and the whole ring in the buffers between
    # the copy-in and the copy-out (fused with the first and last steps); same bits
    buffer_modes = {}
    if not args.no_per_config:
        for name in ("resnet50", "inceptionv3", "vgg16", "vgg16fp16"):
            row = {"ring_on_tensors_ms": per_config[name]["ms_per_step"]}
            for key, kw in (("copy_in_ms", BUFFER_MODES["copy_in"]), ("paper_copies_ms", BUFFER_MODES["paper_copies"])):
                r = measure(name, max(3, args.steps // 2), 2, per_kernel_pass=False, graph_pass=False, **kw)
                row[key] = round(r["ms_per_step"], 4)
            buffer_modes[name] = row
            print(f"# {name} fusion buffer modes: {row}", file=sys.stderr, flush=True)

    # fusion ablation (paper section 7): ResNet-50 and Inception-V3 with other buffer
    # sizes; threshold 0 reduces every tensor with its own ring (no fusion)
    ablation = {}
    if not args.no_ablation:
        # the workloads with many small tensors; the headline alone when only it is timed
        for name in ([args.workload] if args.no_per_config else ["resnet50", "inceptionv3"]):
            ablation[name] = {}
            for thr in (0, 1 << 20, 4 << 20, 16 << 20, 64 << 20, 256 << 20):
                r = measure(name, max(3, args.steps // 4), 2, threshold=thr, per_kernel_pass=False)
                ablation[name][str(thr)] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()}
                print(f"# {name} fusion threshold {thr}: {r['ms_per_step']:.3f} ms/step, "
                      f"graph {r['graph_ms_per_step']:.3f}", file=sys.stderr, flush=True)

    # the ring's fold computed directly (same bits, no per-step messages): a bound for
    # one GPU, reported beside the ring, never as the headline value
    fold = {}
    if not args.no_per_config:
        from workloads import configs

        for name in configs.WORKLOADS:
            r = measure(name, max(3, args.steps // 2), 2, per_kernel_pass=False, schedule="fold", graph_pass=False)
            fold[name] = {"ms_per_step": round(r["ms_per_step"], 4), "algbw_GBps": round(r["algbw_GBps"], 2)}
            print(f"# fold schedule {name}: {r['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)

    bcast = None
    if not args.no_broadcast:
        bcast = measure_broadcast(args.broadcast_workload, max(3, args.steps // 2))
        print(f"# broadcast: {bcast['call_ms']:.3f} ms per call, {bcast['prepared_ms']:.3f} ms prepared, "
              f"{bcast['flat_ms']:.3f} ms flat, {bcast['per_tensor_chains_ms']:.3f} ms one chain per tensor",
              file=sys.stderr, flush=True)

    dom_name, dom = max(head["kernels"].items(), key=lambda kv: kv[1]["share"])
    roofline = {
        "bound": "hbm",
        "kernel": dom_name,
        "achieved": round(dom["GBps"], 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(dom["GBps"] / HBM_PEAK_GBS, 4),
        "traffic": traffic_for(dom_name, args.workload),
        "avg_launch_us": round(dom["avg_us"], 2),
        "launches_per_step": dom["launches"] // args.steps,
        "timing": "median over the timed steps of each launch's kernel time, stamped by its own dispatch "
                  "(hipExtLaunchKernel events), averaged over the kernel's launches",
        "timing_outlier_samples": head["timing_outliers"],
        "algorithmic_bytes_per_step": dom["bytes"] // args.steps,
    }
    # the ring's own step kernels (adding, replacing, and the fused boundary step), all
    # launches together: their algorithmic bytes over their summed kernel time
    ring_k = {k: v for k, v in head["kernels"].items() if k.startswith(("rs_step", "ag_step", "rs_ag_step"))}
    ring_bytes = sum(v["bytes"] for v in ring_k.values()) // args.steps
    ring_ms = sum(v["ms_per_step"] for v in ring_k.values())
    ring_roofline = {
        "bound": "hbm",
        "kernels": sorted(ring_k),
        "achieved": round(ring_bytes / (ring_ms * 1e-3) / 1e9, 1) if ring_ms else None,
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(ring_bytes / (ring_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if ring_ms else None,
        "launches_per_step": sum(v["launches"] for v in ring_k.values()) // args.steps,
        "kernel_ms_per_step": round(ring_ms, 4),
        "algorithmic_bytes_per_step": ring_bytes,
    }
    out = {
        "metric": "allreduce algorithm bandwidth GB/s and % of MI355X HBM peak, per config",
        "value": round(head["algbw_GBps"], 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if head["workload"] == "vgg16fp16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": args.workload,
            "simulated_ranks": head["nranks"],
            "op": "average",
            "fusion_threshold_bytes": 64 << 20,
            # adding steps read each rank's own elements from its tensors, partial sums in the
            # fusion buffers, replacing steps write the tensors (fusion_buffer_modes: the others)
            "fusion_buffer_mode": args.fusion_buffer_mode,
            "buckets": head["buckets"],
        },
        "busbw_GBps": round(head["busbw_GBps"], 2),
        "roofline": roofline,
        "ring_roofline": ring_roofline,
        "per_config": per_config,
        "fusion_buffer_modes": buffer_modes,
        "fusion_ablation": {"by_workload_and_threshold_bytes": ablation},
        "broadcast": bcast,
        "fold_schedule": fold,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
