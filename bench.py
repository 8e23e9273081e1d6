#!/usr/bin/env python3
"""Flash Swin attention benchmark on one MI355X.

One step = one ``fla_swin_attn_fwd`` call: a whole shifted-window attention layer over
every batch entry and head of the workload (window partition, shift, border handling,
masking, Q.K^T, online softmax, P.V and the scatter back to token order, all inside the
kernel).  Inputs are synthetic (seeded N(0,1), see paper_2407_02109_amd/synth.py) and
resident in HBM before timing starts.

Prints one JSON line: microseconds per layer (the headline), TFLOP/s and the fraction of
the bf16 matrix-core peak, the HBM roofline of the kernel, the fp64 CPU oracle timed on
this host as a baseline, a "backward" object: the same layer's training forward and
backward pass (dq, dk, dv) with their own roofline, and a "cycle_scan" object: HRSAM's
Cycle-scan (Sec. 3.5) over the token sequence of a 4096^2 image (65536 tokens, 768 channels,
32 states, three copies), with its vector-ALU roofline and the oracle timed on a sample.

Headline mode.  A layer whose bytes exceed the 256 MB last-level cache (MALL) is timed
cold: before each timed call a read-only pass over a 1 GiB buffer evicts the inputs from
L2 and the MALL (reads only, so no dirty lines are left to compete with the call's own
traffic), and each call sits between its own pair of events.  Smaller layers fit the MALL
and are timed warm, back to back.  Both figures are always reported.
"""
from __future__ import annotations

import argparse
import collections
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
# transcendental rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, exponentials at a quarter of
# the plain fp32 rate
PEAK_EXP_TPS = 256 * 4 * 16 * 2.4e9 / 4 / 1e12
SIMDS = 256 * 4               # MI355X: 256 compute units of 4 SIMDs
XCDS = 8                      # accelerator complex dies; rocprofv3 sums GRBM_GUI_ACTIVE over them
MALL_BYTES = 256 << 20        # MI355X last-level (Infinity) cache
FLUSH_BYTES = 1 << 30         # read before each cold call: 4x the MALL
# the kernel each leg's roofline is about, and the sources its hash covers
KERNELS = {
    "fwd": ("swin_fwd_bf16", ["paper_2407_02109_amd/csrc/fla_swin_bf16.hip",
                              "paper_2407_02109_amd/csrc/fla_swin_internal.h",
                              "paper_2407_02109_amd/csrc/fla_swin_device.h"]),
    "bwd": ("swin_bwd_bf16", ["paper_2407_02109_amd/csrc/fla_swin_bwd_bf16_window.hip",
                              "paper_2407_02109_amd/csrc/fla_swin_bwd_bf16_blocks.hip",
                              "paper_2407_02109_amd/csrc/fla_swin_internal.h",
                              "paper_2407_02109_amd/csrc/fla_swin_device.h"]),
    "cycle": ("cycle_scan", ["paper_2407_02109_amd/csrc/fla_cycle_scan.hip",
                             "paper_2407_02109_amd/csrc/fla_cycle_scan.h",
                             "paper_2407_02109_amd/csrc/fla_swin_internal.h",
                             "paper_2407_02109_amd/csrc/fla_swin_device.h"]),
}


def kernel_hash(leg: str = "fwd") -> str:
    h = hashlib.sha256()
    for p in KERNELS[leg][1]:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_path(leg: str, workload: str, out_dir: str = "") -> str:
    return os.path.join(out_dir or os.path.join(ROOT, "profiles"),
                        "traffic_%s%s.json" % ({"fwd": "", "bwd": "bwd_"}.get(leg, leg + "_"), workload))


def roofline(flops: float, nbytes: float, us: float, traffic):
    """The roofline that bounds a launch of the given algorithmic work: HBM when its
    arithmetic intensity is below the ridge (peak FLOP/s / peak B/s = 312.5 FLOP/B), the
    bf16 matrix cores above it (windows of 1024 tokens and more)."""
    if flops / nbytes > PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        tf = flops / (us * 1e-6) / 1e12
        return {"bound": "mfma", "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": traffic}
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic}


def measured_traffic(workload: str, leg: str = "fwd"):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary,
    or None when it is missing or was taken on another version of the kernel source."""
    path = traffic_path(leg, workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_hash") != kernel_hash(leg):
        return None
    return rec.get("bytes_per_launch")


def copy_calibration(nbytes: int = 512 << 20, reps: int = 3):
    """Plain device-to-device copies of a known size, run inside the profiled process so
    that FETCH_SIZE / WRITE_SIZE can be scaled by what they read for a known byte count."""
    import torch
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()


def summarize(prof_dir: str, workload: str, command: str, leg: str = "fwd", out_dir: str = ""):
    """Turn rocprofv3 CSV output (kernel trace + FETCH_SIZE + WRITE_SIZE passes) into the
    committed summaries under profiles/ (or out_dir): a markdown table and the traffic JSON
    of the leg's kernel (swin_fwd_bf16 or swin_bwd_bf16)."""
    out_dir = out_dir or os.path.join(ROOT, "profiles")
    kname = KERNELS[leg][0]
    import csv
    import glob
    import statistics as st

    def rows(pattern):
        out = []
        for path in glob.glob(os.path.join(prof_dir, pattern), recursive=True):
            with open(path) as f:
                out.extend(csv.DictReader(f))
        return out

    all_rows = sorted(rows("trace/**/*kernel_trace.csv"), key=lambda r: int(r["Start_Timestamp"]))
    trace = [r for r in all_rows if kname in r["Kernel_Name"]]
    # the workload's own launches: the most common grid (the bench also times a one-token
    # launch of the same kernel, for the launch overhead)
    grids = collections.Counter(r["Grid_Size_X"] for r in trace)
    main_grid = grids.most_common(1)[0][0] if grids else None
    durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace if r["Grid_Size_X"] == main_grid]
    # cold launches: those that directly follow the read-only cache flush (a reduction kernel)
    cold_durs, warm_durs, prev = [], [], None
    for r in all_rows:
        if kname in r["Kernel_Name"] and r["Grid_Size_X"] == main_grid:
            # the flush is torch's reduction (at::native); the library's own pad-gradient
            # reduction kernel is not a flush
            cold = prev is not None and "reduce_kernel" in prev["Kernel_Name"] and "at::native" in prev["Kernel_Name"]
            (cold_durs if cold else warm_durs).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        prev = r
    # the kernel those launches ran (swin_bwd_bf16_block_kernel for windows of more than 256 tokens)
    found = sorted({m.group(1) for r in trace if r["Grid_Size_X"] == main_grid
                    for m in [re.search(r"(%s\w*_kernel)" % kname, r["Kernel_Name"])] if m})
    title = ", ".join(found) or kname + "_kernel"
    stats = rows("trace/**/*kernel_stats.csv")
    counters = {}
    copies = {}
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        per_dispatch, per_copy = {}, {}
        for r in rows("%s/**/*counter_collection.csv" % name.lower()):
            if r["Counter_Name"] != name:
                continue
            key = r["Dispatch_Id"]
            if kname in r["Kernel_Name"]:
                per_dispatch[key] = per_dispatch.get(key, 0.0) + float(r["Counter_Value"])
            elif "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) >= 65536:
                # the 512 MiB calibration copies (small copies elsewhere have tiny grids)
                per_copy[key] = per_copy.get(key, 0.0) + float(r["Counter_Value"])
        counters[name] = st.median(per_dispatch.values()) if per_dispatch else None
        copies[name] = st.median(per_copy.values()) if per_copy else None
    # optional matrix-core pass: SQ_INSTS_VALU_MFMA_MOPS_BF16 (units of 512 FLOP) and
    # SQ_VALU_MFMA_BUSY_CYCLES summed over the rows of a dispatch, GRBM_GUI_ACTIVE its max
    # (the reported value is the sum over the XCDs: divided by XCDS it is the kernel's cycles)
    mfma = {}
    mrows = [r for r in rows("mfma/**/*counter_collection.csv") if kname in r["Kernel_Name"]]
    mgrid = collections.Counter(r["Grid_Size"] for r in mrows).most_common(1)[0][0] if mrows else None
    for r in mrows:
        if r["Grid_Size"] != mgrid:   # the workload's own launches only
            continue
        d = mfma.setdefault(r["Dispatch_Id"], {})
        name, val = r["Counter_Name"], float(r["Counter_Value"])
        d[name] = max(d.get(name, 0.0), val) if name == "GRBM_GUI_ACTIVE" else d.get(name, 0.0) + val
    mfma_flop = mfma_busy = None
    full = [d for d in mfma.values()
            if {"SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"} <= set(d)]
    if full:
        mfma_flop = st.median(512.0 * d["SQ_INSTS_VALU_MFMA_MOPS_BF16"] for d in full)
        mfma_busy = st.median(d["SQ_VALU_MFMA_BUSY_CYCLES"] / (d["GRBM_GUI_ACTIVE"] / XCDS * SIMDS) for d in full)
    copy_bytes = 512 << 20
    fetch_scale = copy_bytes / (copies["FETCH_SIZE"] * 1024) if copies["FETCH_SIZE"] else None
    write_scale = copy_bytes / (copies["WRITE_SIZE"] * 1024) if copies["WRITE_SIZE"] else None
    traffic = None
    if counters["FETCH_SIZE"] and counters["WRITE_SIZE"] and fetch_scale and write_scale:
        traffic = (counters["FETCH_SIZE"] * 1024 * fetch_scale + counters["WRITE_SIZE"] * 1024 * write_scale)
    lines = ["# rocprofv3 summary: %s, workload %s" % (title, workload), "",
             "Command (run from the repository root on the GPU host):", "", "```", command, "```", ""]
    if durs:
        lines += ["Kernel trace: %d dispatches, duration avg %.2f us, median %.2f us, min %.2f us, max %.2f us"
                  % (len(durs), st.mean(durs) / 1e3, st.median(durs) / 1e3, min(durs) / 1e3, max(durs) / 1e3), ""]
    if cold_durs:
        lines += ["Cold launches (each right after the read-only 1 GiB flush): %d, duration avg %.2f us, "
                  "median %.2f us" % (len(cold_durs), st.mean(cold_durs) / 1e3, st.median(cold_durs) / 1e3),
                  "Warm launches (the others): %d, duration avg %.2f us, median %.2f us"
                  % (len(warm_durs), st.mean(warm_durs) / 1e3, st.median(warm_durs) / 1e3), ""]
    if stats:
        lines += ["| kernel | calls | total ns | average ns | percentage |", "|---|---|---|---|---|"]
        for r in stats:
            lines.append("| %s | %s | %s | %s | %s |" % (r["Name"][:70], r["Calls"], r["TotalDurationNs"],
                                                          r["AverageNs"], r["Percentage"]))
        lines.append("")
    lines += ["HBM counters (KiB per dispatch, median): FETCH_SIZE %s, WRITE_SIZE %s" % (counters["FETCH_SIZE"], counters["WRITE_SIZE"]),
              "Copy calibration (512 MiB device copy, KiB per dispatch): FETCH_SIZE %s, WRITE_SIZE %s" % (copies["FETCH_SIZE"], copies["WRITE_SIZE"]),
              "Scale factors (true bytes / counter bytes): fetch %s, write %s" % (fetch_scale, write_scale),
              "Traffic per launch (scaled): %s bytes" % (None if traffic is None else int(traffic)),
              "Kernel source hash: %s" % kernel_hash(leg), ""]
    if mfma_flop is not None:
        lines[-1:-1] = ["Matrix cores (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512, median per dispatch): %.4g FLOP per launch%s"
                        % (mfma_flop, ", %.1f TFLOP/s over the average duration" % (mfma_flop / st.mean(durs) / 1e3)
                           if durs else ""),
                        "MFMA busy (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / %d XCDs x %d SIMDs), median, "
                        "kernels serialised by the counter pass): %.3f" % (XCDS, SIMDS, mfma_busy)]
    os.makedirs(out_dir, exist_ok=True)
    with open(os.path.join(out_dir, "%s_%s.md" % (kname, workload)), "w") as f:
        f.write("\n".join(lines))
    if traffic is not None:
        with open(traffic_path(leg, workload, out_dir), "w") as f:
            json.dump({"workload": workload, "kernel": title, "kernel_hash": kernel_hash(leg),
                       "bytes_per_launch": int(traffic),
                       "fetch_kib": counters["FETCH_SIZE"], "write_kib": counters["WRITE_SIZE"],
                       "fetch_scale": fetch_scale, "write_scale": write_scale,
                       "mfma_flop_per_launch": mfma_flop, "mfma_busy": mfma_busy,
                       "avg_duration_us": st.mean(durs) / 1e3 if durs else None,
                       "avg_cold_us": st.mean(cold_durs) / 1e3 if cold_durs else None,
                       "avg_warm_us": st.mean(warm_durs) / 1e3 if warm_durs else None}, f, indent=1)
    print("\n".join(lines))


def summarize_cycle(prof_dir: str, command: str, out_dir: str = ""):
    """rocprofv3 CSV output of a bench run into profiles/cycle_scan_cyclescan_img4096.md: per
    Cycle-scan kernel (chunk scans, carries, output scans) the launches, their average
    duration cold (right after the read-only flush) and warm, and, when the FETCH_SIZE /
    WRITE_SIZE passes are there, HBM bytes per launch scaled by the 512 MiB copy."""
    out_dir = out_dir or os.path.join(ROOT, "profiles")
    import csv
    import glob
    import statistics as st

    def rows(pattern):
        out = []
        for path in glob.glob(os.path.join(prof_dir, pattern), recursive=True):
            with open(path) as f:
                out.extend(csv.DictReader(f))
        return out

    def short(name):
        m = re.search(r"(cycle_scan_\w+(?:<\d+>)?)", name)
        return m.group(1) if m else None

    all_rows = sorted(rows("trace/**/*kernel_trace.csv"), key=lambda r: int(r["Start_Timestamp"]))
    durs = collections.defaultdict(lambda: ([], []))   # kernel -> (cold, warm) durations in ns
    prev, cold_call = None, False
    for r in all_rows:
        k = short(r["Kernel_Name"])
        if k is None:
            prev = r
            continue
        if k.startswith("cycle_scan_chunks"):   # a call starts with its chunk scans
            cold_call = prev is not None and "reduce_kernel" in prev["Kernel_Name"] and "at::native" in prev["Kernel_Name"]
        durs[k][0 if cold_call else 1].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        prev = r
    counters = collections.defaultdict(dict)
    copies = {}
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        per, per_copy = collections.defaultdict(dict), {}
        for r in rows("%s/**/*counter_collection.csv" % name.lower()):
            if r["Counter_Name"] != name:
                continue
            k = short(r["Kernel_Name"])
            if k is not None:
                per[k][r["Dispatch_Id"]] = per[k].get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
            elif "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) >= 65536:
                per_copy[r["Dispatch_Id"]] = per_copy.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
        for k, d in per.items():
            counters[k][name] = st.median(d.values())
        copies[name] = st.median(per_copy.values()) if per_copy else None
    scale = {n: (512 << 20) / (copies[n] * 1024) if copies.get(n) else None for n in ("FETCH_SIZE", "WRITE_SIZE")}
    lines = ["# rocprofv3 summary: Cycle-scan kernels, workload cyclescan_img4096 "
             "(65536 tokens, 768 channels, 32 states, 3 copies)", "",
             "Command (run from the repository root on the GPU host):", "", "```", command, "```", "",
             "| kernel | cold launches | cold avg us | warm launches | warm avg us | HBM fetch MB | HBM write MB |",
             "|---|---|---|---|---|---|---|"]
    total = [0.0, 0.0]
    for k in sorted(durs, key=lambda k: ("chunks" not in k, "carries" not in k)):
        cold, warm = durs[k]
        c = st.mean(cold) / 1e3 if cold else None
        w = st.mean(warm) / 1e3 if warm else None
        total[0] += c or 0.0
        total[1] += w or 0.0
        mb = lambda n: ("%.1f" % (counters[k][n] * 1024 * scale[n] / 1e6)) if counters[k].get(n) and scale[n] else "-"
        lines.append("| %s | %d | %s | %d | %s | %s | %s |" % (k, len(cold), "%.2f" % c if c else "-", len(warm),
                                                               "%.2f" % w if w else "-", mb("FETCH_SIZE"), mb("WRITE_SIZE")))
    per_call = None
    if all(counters[k].get("FETCH_SIZE") and counters[k].get("WRITE_SIZE") for k in durs) and all(scale.values()):
        per_call = sum(counters[k]["FETCH_SIZE"] * 1024 * scale["FETCH_SIZE"]
                       + counters[k]["WRITE_SIZE"] * 1024 * scale["WRITE_SIZE"] for k in durs)
    lines += ["| sum (one call) | | %.2f | | %.2f | | |" % tuple(total), "",
              "HBM bytes per call (the three kernels, scaled): %s" % (None if per_call is None else int(per_call)),
              "Copy calibration (512 MiB device copy, KiB per dispatch): FETCH_SIZE %s, WRITE_SIZE %s"
              % (copies.get("FETCH_SIZE"), copies.get("WRITE_SIZE")),
              "Scale factors (true bytes / counter bytes): fetch %s, write %s" % (scale["FETCH_SIZE"], scale["WRITE_SIZE"]),
              "Kernel source hash: %s" % kernel_hash("cycle"), ""]
    os.makedirs(out_dir, exist_ok=True)
    with open(os.path.join(out_dir, "cycle_scan_cyclescan_img4096.md"), "w") as f:
        f.write("\n".join(lines))
    if per_call is not None:
        with open(traffic_path("cycle", "cyclescan_img4096", out_dir), "w") as f:
            json.dump({"workload": "cyclescan_img4096", "kernel": "cycle_scan_chunks, cycle_scan_carries, "
                       "cycle_scan_outputs", "kernel_hash": kernel_hash("cycle"), "bytes_per_launch": int(per_call),
                       "per_kernel_kib": {k: counters[k] for k in durs}, "fetch_scale": scale["FETCH_SIZE"],
                       "write_scale": scale["WRITE_SIZE"]}, f, indent=1)
    print("\n".join(lines))


def cpu_baseline(wl, q, k, v, budget_s: float, out=None):
    """Time the fp64 oracle (textbook Plain Swin form) on this host's cores; with the GPU's
    output `out` of the same inputs, also its error on the heads the oracle computed."""
    import oracle
    from paper_2407_02109_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    # bounded sample: whole layers of the workload when one fits the budget, else a
    # subset of heads (every head is the same amount of work), scaled to a layer
    heads = wl.heads
    q64, k64, v64 = (synth.to_f64_numpy(t) for t in (q, k, v))

    def layer(nh):
        if wl.rope:
            return oracle.swin_attention_rope(q64[:, :, :nh], k64[:, :, :nh], v64[:, :, :nh], wl.H, wl.W, wl.window,
                                              wl.shift, wl.pad_mode, wl.rope[0], wl.rope[1])
        if wl.grids:
            return oracle.swin_attention_ms(q64[:, :, :nh], k64[:, :, :nh], v64[:, :, :nh], list(wl.grid_list),
                                            wl.window, wl.shift, wl.pad_mode)
        return oracle.swin_attention_textbook(q64[:, :, :nh], k64[:, :, :nh], v64[:, :, :nh],
                                              wl.H, wl.W, wl.window, wl.shift, wl.pad_mode)

    t0 = time.perf_counter()
    layer(1)
    per_head = time.perf_counter() - t0
    use_heads = int(max(1, min(heads, budget_s / 3.0 / max(per_head, 1e-6))))
    times = []
    ref = None
    while len(times) < 3:
        t0 = time.perf_counter()
        ref = layer(use_heads)
        times.append((time.perf_counter() - t0) * heads / use_heads)
    check = None
    if out is not None:   # the GPU output of the timed entry point on the same inputs
        import numpy as np
        err = np.abs(synth.to_f64_numpy(out[:, :, :use_heads].cpu()) - ref)
        check = {"heads": use_heads, "max_abs_err": float(err.max()), "mean_abs_err": float(err.mean()),
                 "bound_max": 2e-2, "bound_mean": 2e-3,
                 "pass": bool(np.isfinite(err).all() and err.max() <= 2e-2 and err.mean() <= 2e-3)}
    return {"value": statistics.median(times) * 1e6, "unit": "us/layer", "cores": int(threads),
            "kind": "oracle",
            "sample": "fp64 textbook oracle on %d of %d heads of the %s layer, median of 3, "
                      "scaled to the whole layer; host %s with %d usable cores"
                      % (use_heads, heads, wl.name, cpu_model(), len(os.sched_getaffinity(0))),
            "cpu_model": cpu_model(), "usable_cores": len(os.sched_getaffinity(0)),
            "bruteforce_tiny_us": bruteforce_tiny(), "gpu_vs_oracle": check}


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return os.uname().machine


def bruteforce_tiny() -> dict:
    """The oracle's brute-force form (every query scans every key with the region test) on the
    two 32x32 fp32 workloads, shift 0 and 4: median of 3 runs, microseconds per layer."""
    import oracle
    from paper_2407_02109_amd import synth
    res = {}
    for name in ("tiny_s0", "tiny_s4"):
        wl = synth.WORKLOADS[name]
        q, k, v = (synth.to_f64_numpy(t) for t in synth.make_inputs(wl))
        times = []
        for _ in range(3):
            t0 = time.perf_counter()
            oracle.swin_attention_bruteforce(q, k, v, wl.H, wl.W, wl.window, wl.shift, wl.pad_mode)
            times.append(time.perf_counter() - t0)
        res[name] = round(statistics.median(times) * 1e6, 1)
    return res


def build_info(torch) -> dict:
    """What the numbers were measured with: ROCm and torch versions, and the source hash of each
    leg's kernels (the same hash the committed counter summaries carry)."""
    rocm = None
    try:
        with open("/opt/rocm/.info/version") as f:
            rocm = f.read().strip()
    except OSError:
        pass
    return {"rocm": rocm, "torch": torch.__version__, "hip": getattr(torch.version, "hip", None),
            "kernel_hash": {leg: kernel_hash(leg) for leg in KERNELS}}


def device_info(torch) -> dict:
    """Name, architecture and compute units as the runtime reports them, and the engine
    clock range from sysfs when it is readable."""
    p = torch.cuda.get_device_properties(0)
    info = {"name": p.name, "arch": getattr(p, "gcnArchName", ""), "cus": p.multi_processor_count}
    try:
        import glob
        for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
            with open(path) as f:
                mhz = [int(t.split(":")[1].strip().lower().split("mhz")[0]) for t in f.read().splitlines() if ":" in t]
            if mhz:
                info["sclk_mhz_max"] = max(mhz)
                break
    except (OSError, ValueError, IndexError):
        pass
    return info


def parse_sclk(text: str):
    """The current engine clock (MHz) from the text of pp_dpm_sclk: the line marked '*'."""
    for line in text.splitlines():
        if line.rstrip().endswith("*") and ":" in line:
            try:
                return int(line.split(":")[1].strip().lower().split("mhz")[0])
            except ValueError:
                return None
    return None


class ClockSampler:
    """Samples the engine clock from sysfs every `period` seconds in a thread while a block
    runs (`with sampler:`); `median()` of the samples, None when the clock is not readable
    (no sysfs file, or several GPUs whose files cannot be told apart)."""

    def __init__(self, period: float = 0.05):
        import glob
        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if len(paths) == 1 else None
        self.period = period
        self.samples = []

    def _run(self):
        while not self._stop.wait(self.period):
            try:
                with open(self.path) as f:
                    mhz = parse_sclk(f.read())
            except OSError:
                mhz = None
            if mhz is not None:
                self.samples.append(mhz)

    def __enter__(self):
        import threading
        self.samples = []
        if self.path is not None:
            self._stop = threading.Event()
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def __exit__(self, *exc):
        if self.path is not None:
            self._stop.set()
            self._thread.join()
        return False

    def median(self):
        xs = sorted(self.samples)
        return xs[len(xs) // 2] if xs else None


def percentiles(xs):
    xs = sorted(xs)
    pick = lambda f: xs[min(len(xs) - 1, int(f * len(xs)))]
    return round(pick(0.10), 3), round(pick(0.50), 3), round(pick(0.90), 3)


def per_call_us(step, stream, calls: int, before=None):
    """Duration of single calls, each bracketed by its own pair of events on the stream;
    `before` (e.g. a cache flush) runs ahead of each call, outside its events.  Without
    `before` each call is synchronised before the next is issued; with it the calls are
    issued without waiting (the flush ahead of each call keeps the queue ahead of the host)."""
    import torch
    evs = []
    for _ in range(calls):
        if before is not None:
            before()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step()
        e1.record(stream)
        if before is None:
            e1.synchronize()
        evs.append((e0, e1))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in evs]


class ReadFlush:
    """Evicts L2 and the MALL by reading FLUSH_BYTES of other data (a sum over a 1 GiB buffer
    on the stream): reads only, so the caches are left holding clean lines."""

    def __init__(self, torch, device, stream):
        self.buf = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device=device)
        self.acc = torch.zeros((), dtype=torch.float32, device=device)
        self.stream = stream
        self.torch = torch

    def __call__(self):
        with self.torch.cuda.stream(self.stream):
            self.torch.sum(self.buf, dim=0, out=self.acc)


def stream_ceiling(torch, qd, kd, vd, out, stream, flush) -> dict:
    """A plain streaming kernel over the layer's own bytes: torch.addcmul reading as many bytes
    of q, k and v as the layer reads and writing out once, warm (back to back) and cold (after
    the same read-only flush).  It is the practical HBM rate for this traffic pattern."""
    n = out.numel()
    a, b, c, o = qd.view(-1)[:n], kd.view(-1)[:n], vd.view(-1)[:n], out.view(-1)

    def run():
        torch.addcmul(a, b, c, out=o)

    for _ in range(200):
        run()
    warm = per_call_us(run, stream, 200)
    cold = per_call_us(run, stream, 100, before=flush)
    nbytes = 4 * n * out.element_size()
    return {"kernel": "torch.addcmul (3 reads, 1 write)", "bytes": nbytes,
            "warm_p50_us": percentiles(warm)[1], "cold_p50_us": percentiles(cold)[1],
            "warm_gbs": round(nbytes / (percentiles(warm)[1] * 1e3), 1),
            "cold_gbs": round(nbytes / (percentiles(cold)[1] * 1e3), 1)}


def backward_leg(binding, synth, wl, qd, kd, vd, stream, steps: int, mode: str, flush) -> dict:
    """Training on the same layer: the forward that keeps the log-sum-exp, then the backward
    (dq, dk, dv for a seeded upstream gradient), each timed with events on the stream.  The
    roofline is that of the backward's kernel: swin_bwd_bf16_window_kernel, or for windows of
    more than 256 tokens swin_bwd_bf16_block_kernel."""
    import torch
    grids = list(wl.grid_list)
    B, L, heads, d = qd.shape
    dout = synth.make_grad(wl).to(qd.device)
    out = torch.empty_like(qd)
    lse = torch.empty((B, heads, L), dtype=torch.float32, device=qd.device)
    dq, dk, dv = torch.empty_like(qd), torch.empty_like(kd), torch.empty_like(vd)
    nws = binding.fla_swin_attn_bwd_workspace(B, heads, grids, wl.window, wl.shift, wl.pad_mode)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=qd.device)

    if wl.rope:   # RoPE training: rotation fused into the training forward and the backward
        theta, scale = wl.rope
        (H, W), = grids

        def fwd():
            binding.fla_swin_attn_rope_fwd_lse(qd, kd, vd, out, lse, B, heads, H, W, d, wl.window, wl.shift,
                                               wl.pad_mode, theta, scale, stream)

        def bwd():
            binding.fla_swin_attn_rope_bwd(qd, kd, vd, out, dout, lse, dq, dk, dv, ws, nws, B, heads, H, W, d,
                                           wl.window, wl.shift, wl.pad_mode, theta, scale, stream)
    else:
        def fwd():
            binding.fla_swin_attn_ms_fwd_lse(qd, kd, vd, out, lse, B, heads, grids, d, wl.window, wl.shift,
                                             wl.pad_mode, stream)

        def bwd():
            binding.fla_swin_attn_ms_bwd(qd, kd, vd, out, dout, lse, dq, dk, dv, ws, nws, B, heads, grids, d,
                                         wl.window, wl.shift, wl.pad_mode, stream)

    def mean_us(fn, n):
        for _ in range(max(n // 4, 10)):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    fwd_us = mean_us(fwd, steps)
    fwd()
    clk_warm, clk_cold = ClockSampler(), ClockSampler()
    with clk_warm:
        warm_us = mean_us(bwd, steps)
    p10, p50, p90 = percentiles(per_call_us(bwd, stream, 100))
    with clk_cold:
        cold = per_call_us(bwd, stream, max(steps // 5, 50), before=flush)
    cold_us = statistics.mean(cold)
    c10, c50, c90 = percentiles(cold)
    assert torch.isfinite(dq[:, :64].float()).all() and torch.isfinite(dk[:, :64].float()).all()
    flops, nbytes = binding.fla_swin_attn_bwd_work(B, heads, grids, d, wl.window, wl.shift, wl.pad_mode, 2)
    us = cold_us if mode == "cold" else warm_us
    tflops = flops / (us * 1e-6) / 1e12
    traffic = measured_traffic(wl.name, "bwd")
    return {"us_per_layer": round(us, 3), "mode": mode, "steps": steps, "fwd_lse_us": round(fwd_us, 3),
            "tflops": round(tflops, 2), "frac_mfma_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
            "roofline": roofline(flops, nbytes, us, traffic),
            "roofline_warm": roofline(flops, nbytes, warm_us, traffic),
            "roofline_cold": roofline(flops, nbytes, cold_us, traffic),
            "alg_flops": flops, "alg_bytes": nbytes,
            "timing": {"warm_mean_us": round(warm_us, 3), "warm_p10_us": p10, "warm_p50_us": p50,
                       "warm_p90_us": p90, "cold_mean_us": round(cold_us, 3), "cold_p10_us": c10,
                       "cold_p50_us": c50, "cold_p90_us": c90,
                       "sclk_mhz_p50": {"warm": clk_warm.median(), "cold": clk_cold.median()}}}


def cycle_scan_leg(binding, synth, stream, steps: int, flush) -> dict:
    """Cycle-scan at the token scale of a 4096^2 image: one fla_cycle_scan call (its three
    kernels) timed warm (back to back, between one pair of events) and cold (after the
    read-only flush, each call between its own events).  The work unit is one exponential
    exp(Delta a) per token, channel and state, B L d N per call whatever the number of copies;
    the roofline is the chip's transcendental rate.  The bytes are those a call must move (x,
    Delta, y, B, C, A once each): their rate is reported beside it."""
    import torch
    wl = synth.CYCLE_WORKLOADS["cyclescan_img4096"]
    dev = torch.device("cuda:0")
    x, delta, A, Bm, Cm = (t.to(dev) for t in synth.make_cycle_inputs(wl.B, wl.L, wl.d, wl.N, wl.seed, wl.kind))
    y = torch.empty_like(x)
    nws = binding.fla_cycle_scan_workspace(wl.B, wl.L, wl.d, wl.N, wl.repeats)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=dev)

    def call():
        binding.fla_cycle_scan(x, delta, A, Bm, Cm, y, ws, nws, wl.B, wl.L, wl.d, wl.N, wl.repeats, stream)

    for _ in range(max(steps // 4, 10)):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        call()
    e1.record(stream)
    e1.synchronize()
    warm_us = e0.elapsed_time(e1) * 1e3 / steps
    p10, p50, p90 = percentiles(per_call_us(call, stream, 50))
    cold = per_call_us(call, stream, 30, before=flush)
    cold_us = statistics.mean(cold)
    assert torch.isfinite(y[:, :64]).all()
    exps, nbytes = binding.fla_cycle_scan_work(wl.B, wl.L, wl.d, wl.N, wl.repeats)

    traffic = measured_traffic(wl.name, "cycle")

    def alu(us):
        t = exps / (us * 1e-6) / 1e12
        return {"bound": "alu", "achieved": round(t, 3), "peak": round(PEAK_EXP_TPS, 3), "unit": "Texp/s",
                "frac": round(t / PEAK_EXP_TPS, 4), "traffic": traffic}

    return {"workload": wl.name, "B": wl.B, "L": wl.L, "d": wl.d, "N": wl.N, "repeats": wl.repeats,
            "dtype": "f32", "us_per_call": round(warm_us, 3), "mode": "warm", "steps": steps,
            "roofline": alu(warm_us), "roofline_cold": alu(cold_us),
            "alg_exps": exps, "alg_bytes": nbytes,
            "hbm_gbs": round(nbytes / (warm_us * 1e-6) / 1e9, 1),
            "hbm_frac": round(nbytes / (warm_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "timing": {"warm_mean_us": round(warm_us, 3), "warm_p10_us": p10, "warm_p50_us": p50,
                       "warm_p90_us": p90, "cold_mean_us": round(cold_us, 3)}}


def cycle_scan_cpu_baseline(binding, synth, channels: int = 128) -> dict:
    """The fp64 Cycle-scan oracle on this host: the three copies laid out and scanned, over the
    whole sequence of the 4096^2 workload for `channels` evenly spaced channels (the channels
    are independent), scaled to all of them; and the GPU's output on those channels against it."""
    import numpy as np
    import oracle
    import torch
    wl = synth.CYCLE_WORKLOADS["cyclescan_img4096"]
    ins = synth.make_cycle_inputs(wl.B, wl.L, wl.d, wl.N, wl.seed, wl.kind)
    x, delta, A, Bm, Cm = (t.numpy() for t in ins)
    ch = np.arange(channels) * (wl.d // channels)
    t0 = time.perf_counter()
    ref = oracle.cycle_scan.cycle_scan_channels(x, delta, A, Bm, Cm, ch, wl.repeats)
    dt = time.perf_counter() - t0
    y = binding.cycle_scan(*(t.cuda() for t in ins), repeats=wl.repeats)
    got = y[:, :, torch.as_tensor(ch, device=y.device)].double().cpu().numpy()
    rel = float(np.abs(got - ref).max() / np.abs(ref).max())
    bound = 4.0 * 2.0 ** -24 / float((ins[1].amin(dim=(0, 1))[:, None] * ins[2].abs()).min()) + 1e-6
    return {"value": round(dt * wl.d / channels * 1e6, 1), "unit": "us/call", "cores": 1, "kind": "oracle",
            "sample": "fp64 oracle (sequence laid out %d times, scanned token by token) on %d of %d channels "
                      "over all %d tokens, one run of %.1f s, scaled to all channels; host %s"
                      % (wl.repeats, channels, wl.d, wl.L, dt, cpu_model()),
            "gpu_vs_oracle": {"channels": channels, "max_err_rel_to_max": rel, "bound": bound, "pass": rel <= bound}}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--mode", default="auto", choices=["auto", "cold", "warm"],
                    help="timed mode: cold (caches flushed before each call) or warm (back to back); "
                         "auto = cold when the layer's bytes exceed the 256 MB MALL")
    ap.add_argument("--warmup", type=int, default=20, help="untimed steps before the timed region")
    ap.add_argument("--settle", type=float, default=0.5,
                    help="seconds of untimed calls before the warm-up, so that the clocks have ramped")
    ap.add_argument("--workload", default="img4096",
                    help="img1024 | img2048 | img4096 | img4096_kv | img4096_rope | ragged150x203 | "
                         "ms_img2048 (default: img4096)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle time")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run 512 MiB device copies (for scaling HBM counters)")
    ap.add_argument("--summarize", metavar="PROF_DIR",
                    help="summarise rocprofv3 CSV output into profiles/ and exit (no GPU needed)")
    ap.add_argument("--command", default="", help="profiling command recorded by --summarize")
    ap.add_argument("--summary-dir", default="", help="where --summarize writes (default: profiles/)")
    ap.add_argument("--leg", default="fwd", choices=["fwd", "bwd", "cycle"],
                    help="kernel --summarize is about: the forward, the backward or the Cycle-scan kernels")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward leg")
    ap.add_argument("--bwd-steps", type=int, default=500, help="timed backward calls")
    ap.add_argument("--no-cycle-scan", action="store_true", help="skip the Cycle-scan leg")
    ap.add_argument("--cycle-steps", type=int, default=100, help="timed Cycle-scan calls")
    args = ap.parse_args()

    if args.summarize:
        if args.leg == "cycle":
            summarize_cycle(args.summarize, args.command, args.summary_dir)
        else:
            summarize(args.summarize, args.workload, args.command, args.leg, args.summary_dir)
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: a Flash Swin layer needs no cross-GPU step "
              "(windows, heads and batch entries are independent); run with --gpus 1",
              file=sys.stderr)
        return 2

    import torch
    from paper_2407_02109_amd import binding, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    wl = synth.WORKLOADS[args.workload]
    if wl.dtype != "bf16":
        print("bench.py times the bf16 path; %s is an fp32 parity case" % wl.name, file=sys.stderr)
        return 2
    binding.load_library()
    print("[bench] workload %s: generating inputs" % wl.name, file=sys.stderr, flush=True)
    q, k, v = synth.make_inputs(wl)
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    out = torch.empty_like(qd)
    stream = torch.cuda.current_stream()
    if wl.grids:   # multi-scale: the grids' tokens one after the other, one launch
        grids = list(wl.grid_list)
        flops, nbytes = binding.fla_swin_attn_ms_work(wl.B, wl.heads, grids, wl.head_dim, wl.window,
                                                      wl.shift, wl.pad_mode, wl.elem_bytes)

        def step():
            binding.fla_swin_attn_ms_fwd(qd, kd, vd, out, wl.B, wl.heads, grids, wl.head_dim,
                                         wl.window, wl.shift, wl.pad_mode, stream)
    elif wl.rope:   # 2-D RoPE fused into the prologue: same bytes, same products
        flops, nbytes = binding.fla_swin_attn_work(wl.B, wl.heads, wl.H, wl.W, wl.head_dim,
                                                   wl.window, wl.shift, wl.pad_mode, wl.elem_bytes)
        theta, scale = wl.rope

        def step():
            binding.fla_swin_attn_rope_fwd(qd, kd, vd, out, wl.B, wl.heads, wl.H, wl.W, wl.head_dim,
                                           wl.window, wl.shift, wl.pad_mode, theta, scale, stream)
    else:
        flops, nbytes = binding.fla_swin_attn_work(wl.B, wl.heads, wl.H, wl.W, wl.head_dim,
                                                   wl.window, wl.shift, wl.pad_mode, wl.elem_bytes)

        def step():
            binding.fla_swin_attn_fwd(qd, kd, vd, out, wl.B, wl.heads, wl.H, wl.W, wl.head_dim,
                                      wl.window, wl.shift, wl.pad_mode, stream)

    mode = args.mode if args.mode != "auto" else ("cold" if nbytes > MALL_BYTES else "warm")
    flush = ReadFlush(torch, dev, stream)
    # clocks: run the layer for about half a second before the counted warm-up, so that the
    # engine clock has ramped whatever --warmup is (with a few calls only it has not)
    print("[bench] settling clocks, then warmup %d" % args.warmup, file=sys.stderr, flush=True)
    settle0 = time.perf_counter()
    settle_calls = 0
    while time.perf_counter() - settle0 < args.settle:
        for _ in range(100):
            step()
        settle_calls += 100
        torch.cuda.synchronize()
    settle_s = time.perf_counter() - settle0
    for _ in range(args.warmup):
        step()
    for _ in range(20):
        flush()
    torch.cuda.synchronize()

    def warm_mean(n):
        """Mean of n back-to-back calls between one pair of events."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            step()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    # the timed region: exactly `steps` calls of the headline mode
    print("[bench] timing %d %s steps" % (args.steps, mode), file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    clk_timed = ClockSampler()
    with clk_timed:
        if mode == "cold":
            cold = per_call_us(step, stream, args.steps, before=flush)
            us = statistics.mean(cold)
        else:
            us = warm_mean(args.steps)
        torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    # the other mode, outside the timed region (warm: for about half a second, so that the
    # clock samples cover it)
    clk_other = ClockSampler()
    with clk_other:
        if mode == "cold":
            warm_us = statistics.mean(warm_mean(1000) for _ in range(max(1, round(0.5e6 / (1000 * us)))))
        else:
            cold = per_call_us(step, stream, 100, before=flush)
            warm_us = us
    sclk = {mode: clk_timed.median(), ("warm" if mode == "cold" else "cold"): clk_other.median()}
    cold_us = statistics.mean(cold)
    tflops = flops / (us * 1e-6) / 1e12
    assert torch.isfinite(out[:, :64].float()).all()

    traffic = measured_traffic(wl.name)
    rec = {
        "metric": "us per Flash-Swin attention layer and TFLOP/s (fraction of MFMA peak)",
        "value": round(us, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "heads": wl.heads,
                   "grid": [list(g) for g in wl.grid_list] if wl.grids else [wl.H, wl.W],
                   "head_dim": wl.head_dim, "window": wl.window, "shift": wl.shift,
                   "pad_mode": wl.pad_mode, "parallelism": "none (1 GPU)", "timing": mode},
        "tflops": round(tflops, 2),
        "frac_mfma_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline(flops, nbytes, us, traffic),
        "roofline_warm": roofline(flops, nbytes, warm_us, traffic),
        "roofline_cold": roofline(flops, nbytes, cold_us, traffic),
        "alg_flops": flops,
        "alg_bytes": nbytes,
    }
    # distributions of single warm and cold calls, a streaming kernel over the same bytes
    # (the practical HBM ceiling), and the cost of a launch on a one-token problem
    p10, p50, p90 = percentiles(per_call_us(step, stream, 200))
    c10, c50, c90 = percentiles(cold)
    tq = torch.zeros(1, 1, 1, wl.head_dim, dtype=torch.bfloat16, device=dev)
    tout = torch.empty_like(tq)
    tiny = lambda: binding.fla_swin_attn_fwd(tq, tq, tq, tout, 1, 1, 1, 1, wl.head_dim, wl.window, 0,
                                             0, stream)
    l10, l50, l90 = percentiles(per_call_us(tiny, stream, 200))
    rec["timing"] = {"mode": mode, "warm_mean_us": round(warm_us, 3), "warm_p10_us": p10, "warm_p50_us": p50,
                     "warm_p90_us": p90, "cold_mean_us": round(cold_us, 3), "cold_p10_us": c10,
                     "cold_p50_us": c50, "cold_p90_us": c90, "cold_calls": len(cold),
                     "launch_one_token_p50_us": l50,
                     "flush": "read-only sum over %d MiB before each cold call" % (FLUSH_BYTES >> 20),
                     "settle_s": round(settle_s, 3), "settle_calls": settle_calls,
                     "sclk_mhz_p50": sclk}
    rec["stream_ceiling"] = stream_ceiling(torch, qd, kd, vd, out, stream, flush)
    rec["device"] = device_info(torch)
    rec["build"] = build_info(torch)
    if not args.no_backward:
        print("[bench] backward", file=sys.stderr, flush=True)
        rec["backward"] = backward_leg(binding, synth, wl, qd, kd, vd, stream, args.bwd_steps, mode, flush)
    if not args.no_cycle_scan:
        print("[bench] Cycle-scan", file=sys.stderr, flush=True)
        rec["cycle_scan"] = cycle_scan_leg(binding, synth, stream, args.cycle_steps, flush)
    del flush
    torch.cuda.synchronize()
    if args.copy_calibration:
        copy_calibration()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        step()   # the layer's output again (the streaming probe reused its buffer), for the oracle check
        torch.cuda.synchronize()
        rec["cpu_baseline"] = cpu_baseline(wl, q, k, v, args.cpu_budget, out)
        if "cycle_scan" in rec:
            print("[bench] timing the CPU Cycle-scan oracle", file=sys.stderr, flush=True)
            rec["cycle_scan"]["cpu_baseline"] = cycle_scan_cpu_baseline(binding, synth)
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
