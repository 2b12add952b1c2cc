#!/usr/bin/env python3
"""Throughput of the exact EDT on one MI355X.

Default workload: 3-D EDT of 8 x 1 x 128^3 uint8 masks whose foreground is the
union of 30 random solid balls (radius 4-30 voxels) per volume, unit
sampling, float32 distances.  One step = one tm_edt_ws call over the whole
batch with the mask already resident in HBM and the output (and the
workspace, used by 2-D column passes only) preallocated.  On this
shape the call runs two kernels: the axis-0 nearest-background scan straight
from the mask, writing one byte per voxel ("col_scan.o8"), and one workgroup
per 128 x 128 plane doing both remaining axes and the square root
("plane_final.i8").

Prints one JSON line: voxels/s, per-step time, the dominant kernel's
algorithmic bytes per launch over its HIP-event-timed average duration
against the MI355X HBM peak, the counter-measured traffic and VALU-issue
share of that kernel when a rocprofv3 summary taken on the current kernel
sources is committed under profiles/, and the CPU oracle's throughput on a
bounded sample on this host (median of three runs).
"""
import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
SOURCES = sorted(os.path.relpath(p, ROOT) for p in
                 glob.glob(os.path.join(ROOT, "paper_2608_24738_amd", "csrc", "*.h")) +
                 glob.glob(os.path.join(ROOT, "paper_2608_24738_amd", "csrc", "*.hip")))


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def source_digest():
    """Digest of the kernel sources with comments and whitespace removed, so
    that a profile stays matched to the code it measured across edits of
    comments only."""
    h = hashlib.sha256()
    for s in SOURCES:
        with open(os.path.join(ROOT, s), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(name, total, ndim, want_idx, out_bytes=4):
    """Bytes one launch of kernel `name` must move (separable-pass model):
    the last-axis scan reads the 1-byte mask and writes the 4-byte field,
    every strided pass reads and writes the field, and the final pass reads
    the field and writes the outputs.  A ".i16" / ".o16" suffix marks a
    field read / written as 16-bit values (2 bytes per voxel), ".i8" / ".o8"
    as 8-bit values (1 byte per voxel)."""
    base, *tags = name.split(".")
    fin = 2 if "i16" in tags else 1 if "i8" in tags else 4     # field bytes read
    fout = 2 if "o16" in tags else 1 if "o8" in tags else 4    # field bytes written
    if base.startswith("scan"):
        return total * (1 + fout)
    if base in ("plane_pair", "cdt_plane", "col_scan"):  # reads the mask, writes the field
        return total * (1 + fout)
    if base in ("plane_pair_final", "cdt_plane_final"):
        return total * (1 + out_bytes)
    if base == "scan_signed":                # mask in, signed field out
        return total * (1 + 4)
    if base == "col_scan_signed":            # mask in, class and axis-0 distance as one byte out
        return total * (1 + 1)
    if base == "plane_signed_final":         # those bytes in, signed distances out
        return total * (1 + out_bytes)
    if base in ("fh_field", "tile_pair", "cdt_pair", "cdt_line", "cdt_none",
                "line_search", "line_search_signed", "line_pair", "cdt_l1_scan"):
        return total * (fin + fout)
    if base in ("fh_field_final", "tile_pair_final", "cdt_pair_final", "cdt_line_final",
                "line_search_final", "plane_final", "line_search_signed_final", "line_pair_final",
                "cdt_l1_scan_final"):
        return total * (fin + out_bytes)
    if base == "small2d":                    # mask in; distances (and indices) out
        return total * (1 + out_bytes + (4 * ndim if want_idx else 0))
    if base in ("fh_index", "tile_idx", "fh_long"):     # flat-index carrier in and out
        return total * (4 + 4)
    if base in ("fh_index_final", "tile_idx_final", "fh_long_final"):
        # carrier in; coordinates (with indices) and distances out
        return total * (4 + (4 * ndim if want_idx else 0) + out_bytes)
    if base == "order":                      # 8 bytes per group of 16 lines: not counted
        return 0
    if base in ("cdt_l1_long", "cdt_l1_long_final"):
        return total * (4 + 4) * 2                       # two sweeps, each reads and writes
    raise KeyError(name)


def read_profile(kernel, workload_name):
    """The JSON block of a committed rocprofv3 summary of `kernel` on
    `workload_name`, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "%s__%s.md" % (kernel, workload_name))
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    try:
        data = json.loads(text[start + 7:end])
    except ValueError:
        return None
    if data.get("source_digest") != source_digest():
        return None
    return data


def cpu_model():
    """The host CPU's model name (lscpu), or None."""
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, ValueError):
        pass
    return None


def cpu_baseline(mask_np, ndim, sampling, want_idx, run_s=3.5):
    """The oracle on this host's cores: three runs, each repeating the whole
    batch for about `run_s` seconds, reported as the median rate; beside it
    the median of three single-thread runs on one volume."""
    import statistics

    from oracle import edt_oracle
    nthreads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or min(16, os.cpu_count() or 1)
    used = edt_oracle.threads_used(nthreads)
    batch = mask_np.shape[0]
    vox_per = int(mask_np[0].size)
    rates, reps = [], []
    for _ in range(3):
        done, n = 0, 0
        t0 = time.perf_counter()
        while True:
            edt_oracle.edt(mask_np, ndim, sampling, want_sq=False, want_dist=True, want_idx=want_idx,
                           nthreads=nthreads)
            n += 1
            done += batch * vox_per
            if time.perf_counter() - t0 >= run_s:
                break
        rates.append(done / (time.perf_counter() - t0))
        reps.append(n)
    singles = []
    for _ in range(3):
        t1 = time.perf_counter()
        edt_oracle.edt(mask_np[:1], ndim, sampling, want_sq=False, want_dist=True, want_idx=want_idx,
                       nthreads=1)
        singles.append(vox_per / (time.perf_counter() - t1))
    return {"value": statistics.median(rates), "unit": "voxels/s", "cores": used, "kind": "oracle",
            "sample": "median of 3 runs, each %s x the whole %d-volume batch (about %.1f s), %d OpenMP "
                      "threads" % ("/".join(map(str, reps)), batch, run_s, used),
            "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "runs": [round(r) for r in rates],
            "single_thread_value": statistics.median(singles)}


SETTLE_S = 0.2     # seconds of untimed steps before the warmup steps


def time_op(step, args, stream):
    """Settle the clocks, warm up, time args.steps steps between two events on
    `stream`, then time every kernel of the same number of steps with the
    library's own per-launch events.  Returns (ms per step, {kernel:
    {avg_ms, launches}}).

    The GPU's clocks rise over the first milliseconds of sustained work, so
    the step first runs untimed for about SETTLE_S seconds: without that, a
    20-step window right after 5 warmup steps reads 5-6 % slower than the
    steady rate (8 x 128^3: 42.2-42.4 against 40.6-40.8 us per step).  The
    timed region is unchanged: exactly args.steps whole steps."""
    import torch

    from paper_2608_24738_amd import binding
    log("settling clocks (%.1f s of untimed steps)" % SETTLE_S)
    t0, n = time.perf_counter(), 0
    while True:
        step()
        n += 1
        if n % 25 == 0:
            torch.cuda.synchronize()
            if time.perf_counter() - t0 >= SETTLE_S:
                break
    log("warmup %d" % args.warmup)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("timing %d steps" % args.steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log("timing kernels over %d steps" % args.steps)
    binding.prof_enable(8 * args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    per = {}
    for name, t in binding.prof_read():
        per.setdefault(name, []).append(t)
    shapes = dict(binding.prof_launches())
    binding.prof_enable(0)
    kernels = {k: {"avg_ms": sum(v) / len(v), "launches": len(v), "launch": shapes.get(k)}
               for k, v in per.items()}
    return ms, kernels


def roofline_of(kernels, steps, total, ndim, want_idx, workload_name, out_bytes=4):
    """Roofline entry of the kernel with the largest share of the step, and
    per-kernel algorithmic rates (kernels is updated in place)."""
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    dom_launches_per_step = kernels[dom]["launches"] / steps
    algo = algorithmic_bytes(dom, total, ndim, want_idx, out_bytes)
    achieved = algo / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    for k, v in kernels.items():
        b = algorithmic_bytes(k, total, ndim, want_idx, out_bytes)
        v["algorithmic_bytes"] = b
        v["achieved_GBs"] = round(b / (v["avg_ms"] * 1e-3) / 1e9, 1)
        v["avg_ms"] = round(v["avg_ms"], 5)
        v["launches"] = int(v["launches"] / steps)
    prof = read_profile(dom, workload_name) or {}
    out = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
           "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
           "traffic": prof.get("traffic_bytes_per_launch"),
           "kernel": dom, "launches_per_step": dom_launches_per_step}
    # What the counters say limits the kernel: its HBM traffic over its
    # traced duration against the peak, and its VALU issue time (wave
    # instructions x waves per SIMD x 4 cycles at 2.4 GHz) over the same
    # duration.  The byte roofline above stays the bound the method is
    # judged against; these say how far from it the kernel is and why.
    if prof.get("traced_us"):
        t = prof["traced_us"] * 1e-6
        if prof.get("traffic_bytes_per_launch"):
            out["traffic_frac"] = round(prof["traffic_bytes_per_launch"] / t / 1e9 / HBM_PEAK_GBS, 4)
        if prof.get("valu_issue_us"):
            out["valu_issue_frac"] = round(prof["valu_issue_us"] / prof["traced_us"], 3)
            out["limiter"] = ("valu-issue" if out["valu_issue_frac"] > out.get("traffic_frac", 0.0)
                              else "hbm")
    return out


def bench_cdt(args, dev, stream):
    """Chamfer transform (taxicab or chessboard from --metric, default
    chessboard) of workload 7 (8 x 1024^2) or 8 (8 x 256^2), the two sizes the
    paper's throughput table times it on; int32 distances."""
    import torch

    from paper_2608_24738_amd import binding, workloads
    key = args.workload if args.workload in (7, 8) else 7
    metric = args.metric if args.metric != "euclidean" else "chessboard"
    w = workloads.WORKLOADS[key]
    log("generating %s" % w.name)
    mask = workloads.make_mask(key)
    x = torch.from_numpy(mask).to(dev)
    out = torch.empty(mask.shape, dtype=torch.int32, device=dev)
    code = binding.METRICS[metric]
    ws_bytes = binding.tm_cdt_workspace_size(w.ndim, w.spatial, w.batch, code)
    ws = torch.zeros(max(1, ws_bytes // 4), dtype=torch.int32, device=dev) if ws_bytes else None

    def step():
        binding.tm_cdt_ws(x, w.ndim, code, out, ws, stream=stream)

    ms, kernels = time_op(step, args, stream)
    total = int(mask.size)
    roofline = roofline_of(kernels, args.steps, total, w.ndim, False, "%s_%s" % (w.name, metric))
    print(json.dumps({
        "metric": "chamfer DT inputs/ms (%s), batch %dx1x%s" % (metric, w.batch,
                                                                "x".join(map(str, w.spatial))),
        "value": w.batch / ms, "unit": "inputs/ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int32", "data": "synthetic",
        "config": {"workload": w.name, "metric": metric, "outputs": "int32 distances",
                   "workspace_bytes": ws_bytes,
                   "mask_sha256": workloads.mask_digest(mask)[:16]},
        "voxels_per_s": total / (ms * 1e-3),
        "roofline": roofline,
        "kernels": kernels,
        "source_digest": source_digest()}), flush=True)


def bench_signed(args, dev, stream):
    """Signed transform EDT(M) - EDT(not M) (the boundary-loss field) of an
    EDT workload (default: the 8 x 1 x 128^3 balls); float32 output."""
    import torch

    from paper_2608_24738_amd import binding, workloads
    key = args.workload
    w = workloads.WORKLOADS[key]
    log("generating %s" % w.name)
    mask = workloads.make_mask(key)
    x = torch.from_numpy(mask).to(dev)
    out = torch.empty(mask.shape, dtype=torch.float32, device=dev)

    def step():
        binding.tm_edt_signed(x, w.ndim, out, stream=stream)

    ms, kernels = time_op(step, args, stream)
    total = int(mask.size)
    roofline = roofline_of(kernels, args.steps, total, w.ndim, False, "%s_signed" % w.name)
    print(json.dumps({
        "metric": "signed EDT voxels/sec, %s" % w.name,
        "value": total / (ms * 1e-3), "unit": "voxels/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int32", "data": "synthetic",
        "config": {"workload": w.name, "outputs": "float32 signed distances",
                   "mask_sha256": workloads.mask_digest(mask)[:16]},
        "roofline": roofline,
        "kernels": kernels,
        "source_digest": source_digest()}), flush=True)


def bench_bf(args, dev, stream):
    """Brute-force transform: 8 x 256^2 images whose background is a seeded
    1 % Bernoulli sample (the paper times its brute-force transform on 256^2
    inputs); metric from --metric, float32 distances and int32 indices."""
    import torch

    from paper_2608_24738_amd import binding
    from paper_2608_24738_amd import workloads
    w = workloads.WORKLOADS[6]
    batch, n = w.batch, w.spatial[0]
    mask = workloads.make_mask(6)
    x = torch.from_numpy(mask).to(dev)
    dist = torch.empty(mask.shape, dtype=torch.float32, device=dev)
    idx = torch.empty((batch, 1, 2, n, n), dtype=torch.int32, device=dev)
    code = binding.METRICS[args.metric]

    def step():
        binding.tm_dt_bf(x, 2, code, None, dist, idx, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    zeros = int((mask == 0).sum())
    pairs = zeros * n * n                       # (element, background element) pairs per step
    print(json.dumps({
        "metric": "brute-force DT inputs/ms (%s), batch 8x1x256^2" % args.metric,
        "value": batch / ms, "unit": "inputs/ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int32", "data": "synthetic",
        "config": {"workload": w.name, "metric": args.metric,
                   "outputs": "float32 distances + int32 indices"},
        "pair_evaluations_per_s": pairs / (ms * 1e-3)}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=3,
                    help="workload key (paper_2608_24738_amd/workloads.py): 1-5, 9-15 edt "
                         "(3 = headline), 7-8 cdt")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--copy-calib", action="store_true",
                    help="run only a plain 256 MiB device copy (counter calibration)")
    ap.add_argument("--op", default="edt", choices=["edt", "bf", "cdt", "signed"],
                    help="edt: the exact transform (headline); bf: the brute-force transform; "
                         "cdt: the chamfer transform (workload 7 or 8); signed: EDT(M) - EDT(not M)")
    ap.add_argument("--metric", default="euclidean", choices=["euclidean", "taxicab", "chessboard"],
                    help="metric of --op bf / cdt (cdt: euclidean means chessboard)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only; --gpus %d is not supported (the EDT shards "
              "by batch with no exchange between GPUs)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_24738_amd import binding, build as hip_build, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    if args.copy_calib:
        n = 64 * 1024 * 1024                       # 256 MiB of float32 each way
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calib": True, "read_bytes": 4 * n, "write_bytes": 4 * n}))
        return

    if not os.path.exists(binding.LIB_PATH):
        hip_build.build()
    binding.load()
    if args.op == "bf":
        return bench_bf(args, dev, stream)
    if args.op == "cdt":
        return bench_cdt(args, dev, stream)
    if args.op == "signed":
        return bench_signed(args, dev, stream)

    w = workloads.WORKLOADS[args.workload]
    log("generating %s" % w.name)
    mask_np = workloads.make_mask(args.workload)
    ndim = w.ndim
    total = int(mask_np.size)
    x = torch.from_numpy(mask_np).to(dev)
    dist = torch.empty(mask_np.shape, dtype=torch.float32, device=dev)
    idx = None
    if w.want_idx:
        idx = torch.empty((w.batch, 1, ndim) + tuple(w.spatial), dtype=torch.int32, device=dev)
    samp = list(w.sampling) if w.sampling else None
    # the workspace in which tm_edt_ws keeps a dispatch order (2-D column
    # passes; none for the other workloads), allocated before timing
    ws_bytes = binding.tm_edt_workspace_size(ndim, w.spatial, w.batch, samp, w.want_idx)
    ws = torch.zeros(max(1, ws_bytes // 4), dtype=torch.int32, device=dev) if ws_bytes else None

    def step():
        binding.tm_edt_ws(x, ndim, samp, dist, idx, ws, stream=stream)

    # per-kernel durations: HIP events recorded by the library around each of
    # its launches, on the launch stream, over the same number of steps
    ms, kernels = time_op(step, args, stream)
    roofline = roofline_of(kernels, args.steps, total, ndim, w.want_idx, w.name)

    cpu = None
    if not args.no_cpu:
        log("timing the CPU oracle")
        cpu = cpu_baseline(mask_np.reshape((w.batch,) + tuple(w.spatial)), ndim, w.sampling, w.want_idx)

    vox_s = total / (ms * 1e-3)
    out = {
        "metric": ("EDT voxels/sec and achieved HBM GB/s (% of peak), batch 8x1x128^3"
                   if args.workload == 3 else "EDT voxels/sec, %s" % w.name),
        "value": vox_s,
        "unit": "voxels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_s": SETTLE_S,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32" if samp is None else "f64",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "channels": 1,
                   "spatial": list(w.spatial), "sampling": samp or "unit",
                   "workspace_bytes": ws_bytes,
                   "outputs": "float32 distances" + (" + int32 indices" if w.want_idx else ""),
                   "mask_sha256": workloads.mask_digest(mask_np)[:16]},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "inputs_per_ms": w.batch / ms,
        "model_GBs_per_step": round(sum(v["algorithmic_bytes"] * v["launches"]
                                        for v in kernels.values()) / (ms * 1e-3) / 1e9, 1),
        "source_digest": source_digest(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
