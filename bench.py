#!/usr/bin/env python3
"""Throughput of the octree-CNN hot path (O-CNN, arXiv 1712.01537) on one MI355X.

One step is one pass of the whole path over one batch of synthetic shapes whose
points and normals are already in HBM:
  oc_build (keys, occupancy ranks, labels, signal, sibling-group neighbour
  tables) and the workload's network forward (conv + fused ReLU, max-pool) and
  backward (pool routing, conv input and weight gradients).  Like the paper's
  precomputation of the next iteration's hash table in a separate thread, the
  octree of step i+1 is built during step i: the part that decides the
  per-depth counts (quantisation, occupancy bitmaps, their scan) at the head
  of the step, so that the host has the counts while the network of step i
  runs, the rest (leaf signal, keys, labels, neighbour tables) after it;
  every timed step builds one octree and runs one forward and backward.
The default workload is the 32-shape depth-6 network: conv3 3->16 @d6,
16->32 @d5, 32->64 @d4, 64->128 @d3 (each + ReLU + 2x2x2 max-pool), then
conv3 + ReLU 128->256 @d2, fp32.

The printed JSON line reports:
  value          nominal convolution fwd+bwd GFLOP/s of the whole step
                 (6 N_out K^3 Cin Cout per conv layer, every tap counted as
                 im2col does, divided by the wall time of the step);
  octants_per_s  output octants of all conv layers per second;
  roofline       the dominant kernel (largest share of the step in the
                 warmup): its algorithmic flops (or bytes) per launch over its
                 mean launch time, from HIP events that the library records at
                 the start and end of that kernel (hipExtLaunchKernelGGL) on the
                 stream it runs on, against the MI355X peak.  In the timed
                 steps one launch of it per step is bracketed, its launches
                 (layers) in turn, each layer's mean taken first;
  cpu_baseline   the plain CPU oracle on a bounded sample of the same workload.
  roofline.traffic  HBM bytes per launch of the dominant kernel from rocprofv3
                 FETCH_SIZE and WRITE_SIZE counters (two runs of this script
                 with --copy-probe), each scaled by what the same counter reads
                 for a plain device copy of known size; taken from
                 profiles/hbm_counters_<workload>.md, and null when a source
                 file that defines or launches the kernel (or the shared
                 internal header) differs from the one the counters were
                 taken on.

  ops            every op class's main kernels in the warmup (HIP events)
                 against its work: TFLOP/s of the conv passes, GB/s of the
                 pooling, and conv_fwd_bwd over all conv passes.

Trace summary: python bench.py --summarize-trace PROF_DIR PROF_LOG reads the
  kernel statistics of a rocprofv3 --kernel-trace --stats run of this script
  and that run's own output, and prints each kernel class's time per step
  against its work (build and pooling GB/s, conv fwd+bwd TFLOP/s with and
  without the helper kernels) and the per-kernel table.

Counter summary: python bench.py --summarize-counters FETCH_DIR WRITE_DIR
  --copy-probe MIB --workload NAME reads the counter_collection CSV files of
  the two rocprofv3 runs and prints the summary (markdown with a JSON block).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Networks whose next build starts after the forward of this layer instead
# of at the head of the step.  wide_d7: its first layer is a pair of
# persistent matrix-core kernels that hold every compute unit, and the
# build's kernels beside them stretch both; after its forward the build runs
# beside the stride-2 layer, which leaves the matrix cores mostly idle.
# net_d6: after the depth-4 layer's forward the build runs beside the
# depth-3 and depth-2 layers, the head and their backward (measured: 0.675 ms
# per step, against 0.685-0.695 from the head of the step and 0.674-0.683
# after the depth-5 or depth-3 layer).
BUILD_AFTER = {"wide_d7": 0, "net_d6": 4}

PEAK = {  # MI355X published peaks
    "hbm_GBps": 8000.0,
    "fp32_TFLOPs": 157.3,
    "bf16_TFLOPs": 2500.0,
}

# Per-kernel-class accounting: "flops" (MFMA-bound) or "bytes" (HBM-bound).
BOUND = {
    "conv_fwd": "mfma",
    "conv_bwd_data": "mfma",
    "conv_bwd_weight": "mfma",
    "deconv_fwd": "mfma",
    "deconv_bwd_data": "mfma",
    "deconv_bwd_weight": "mfma",
    "pool_fwd": "hbm",
    "pool_bwd": "hbm",
    "unpool_fwd": "hbm",
    "unpool_bwd": "hbm",
    "gpool_fwd": "hbm",
    "gpool_bwd": "hbm",
    "bn_fwd": "hbm",
    "bn_bwd": "hbm",
    "fc_fwd": "hbm",
    "fc_bwd": "hbm",
    "dropout": "hbm",
    "softmax": "hbm",
    "sgd": "hbm",
    "build": "hbm",
    "build_emit": "hbm",
    "round": "hbm",
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="net_d6")
    ap.add_argument("--cpu-shapes", type=int, default=32,
                    help="shapes of the batch the CPU oracle runs (0: skip)")
    ap.add_argument("--layers", action="store_true", help="also print per-layer timings to stderr")
    ap.add_argument("--streams", type=int, default=1, choices=(1, 2),
                    help="2: weight gradients on a second stream beside the rest of the backward")
    ap.add_argument("--build-inline", action="store_true",
                    help="run the next batch's build on the network's stream, between "
                         "steps, instead of on its own stream beside the network")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the steps, run an elementwise copy (y = -x) of MIB MiB three "
                         "times: the known-size kernel that calibrates the HBM byte counters")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM counter summary of two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-mfma", nargs=2, metavar=("PMC_DIR", "PROF_DIR"),
                    help="print the matrix-core counters of a --pmc run (MFMA_COUNTERS) "
                         "against a --kernel-trace --stats run, and exit")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("PROF_DIR", "PROF_LOG"),
                    help="print the per-class kernel time of a rocprofv3 --kernel-trace --stats "
                         "run of this script (its output directory and its stdout) and exit")
    return ap.parse_args()


SRC_GLOBS = ("paper_1712_01537_amd/csrc/*", "include/*.h")


def source_hashes():
    """sha256 of each source file liboc.so is built from, by repository path."""
    out = {}
    for pat in SRC_GLOBS:
        for f in sorted(glob.glob(os.path.join(ROOT, pat))):
            with open(f, "rb") as fh:
                out[os.path.relpath(f, ROOT)] = hashlib.sha256(fh.read()).hexdigest()
    return out


def kernel_sources(kernel):
    """Source files a kernel's code depends on: the files that define or launch
    it (its base name followed by '<' or '(') and the shared header."""
    base = kernel.split("<")[0]
    deps = set()
    for f in source_hashes():
        with open(os.path.join(ROOT, f)) as fh:
            text = fh.read()
        if re.search(re.escape(base) + r"\s*[<(]", text):
            deps.add(f)
    if deps:
        deps.add("paper_1712_01537_amd/csrc/common.h")
    return sorted(deps)


def counters_path(workload):
    return os.path.join(ROOT, "profiles", f"hbm_counters_{workload}.md")


def load_traffic(workload, kernel):
    """Calibrated HBM bytes per launch of `kernel` (read + write) from the
    committed counter summary, or None when there is none for this kernel or
    the library sources changed since the counters were taken."""
    try:
        with open(counters_path(workload)) as fh:
            text = fh.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    k = rec.get("kernels", {}).get(kernel)
    if not k:
        return None
    now, then = source_hashes(), rec.get("sources", {})
    deps = kernel_sources(kernel)
    if not deps or any(now.get(f) is None or now.get(f) != then.get(f) for f in deps):
        return None
    return {"read_bytes": k["fetch_bytes_per_launch"], "write_bytes": k["write_bytes_per_launch"],
            "bytes": k["fetch_bytes_per_launch"] + k["write_bytes_per_launch"],
            "source": os.path.relpath(counters_path(workload), ROOT)}


def _counter_rows(d, counter):
    """(kernel name, value) per dispatch from the counter_collection CSV files
    under directory d."""
    rows = []
    for f in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                if r.get("Counter_Name") == counter:
                    rows.append((int(r.get("Dispatch_Id", 0)), r["Kernel_Name"],
                                 float(r["Counter_Value"])))
    rows.sort()
    return [(k, v) for _, k, v in rows]


def _short_name(k):
    """Kernel name with its template arguments, without namespaces of the
    anonymous kind and without the argument list."""
    k = k.replace("(anonymous namespace)::", "")
    k = re.sub(r"^void ", "", k)
    depth = 0
    for i, ch in enumerate(k):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return k[:i].strip()
    return k.strip()


def summarize_counters(fetch_dir, write_dir, copy_mib, workload):
    """Per-kernel mean FETCH_SIZE / WRITE_SIZE per dispatch (KiB, as rocprofv3
    reports them), calibrated by the copy probe: a copy of S bytes must read S
    and write S bytes, so bytes = counter * 1024 / (copy counter * 1024 / S)."""
    out = {}
    for name, d, ctr in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        for k, v in _counter_rows(d, ctr):
            e = out.setdefault(_short_name(k), {}).setdefault(name, [])
            e.append(v)
    size = copy_mib * 2 ** 20
    copy = [k for k in out if "neg" in k.lower() and "fetch" in out[k] and "write" in out[k]
            and max(out[k]["fetch"]) * 1024 > 0.5 * size]
    if not copy or size <= 0:
        raise SystemExit("no copy-probe kernel of the given size in the counter runs")
    ck = copy[0]
    # the probe's largest dispatches are the copies of `size` bytes
    cf = max(out[ck]["fetch"]) * 1024 / size
    cw = max(out[ck]["write"]) * 1024 / size
    kernels = {}
    for k, v in sorted(out.items()):
        # the bench's own input generation (torch kernels) is not the library's
        if "fetch" not in v or "write" not in v or k == ck or k.startswith("at::"):
            continue
        f = sum(v["fetch"]) / len(v["fetch"]) * 1024 / cf
        w = sum(v["write"]) / len(v["write"]) * 1024 / cw
        kernels[k] = {"dispatches": len(v["fetch"]), "fetch_bytes_per_launch": round(f),
                      "write_bytes_per_launch": round(w)}
    rec = {"workload": workload, "sources": source_hashes(),
           "copy_probe": {"kernel": ck, "bytes": size, "fetch_factor": round(cf, 4),
                          "write_factor": round(cw, 4)},
           "kernels": kernels}
    print(f"Copy probe `{ck}` of {copy_mib} MiB: FETCH_SIZE reads {cf:.4f} x and WRITE_SIZE "
          f"{cw:.4f} x the bytes copied; every figure below is divided by these factors.\n")
    print("| kernel | dispatches | read MB / launch | write MB / launch |")
    print("|---|---|---|---|")
    for k, v in sorted(kernels.items(), key=lambda kv: -(kv[1]["fetch_bytes_per_launch"]
                                                          + kv[1]["write_bytes_per_launch"])):
        print(f"| `{k}` | {v['dispatches']} | {v['fetch_bytes_per_launch'] / 1e6:.3f} | "
              f"{v['write_bytes_per_launch'] / 1e6:.3f} |")
    print("\n```json\n" + json.dumps(rec, indent=1) + "\n```")


MFMA_COUNTERS = ("MfmaUtil", "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                 "SQ_WAVE_CYCLES", "SQ_WAIT_INST_LDS", "SQ_LDS_BANK_CONFLICT",
                 "SQ_ACTIVE_INST_LDS")


def summarize_mfma(pmc_dir, prof_dir):
    """Matrix-core use of each kernel from a rocprofv3 --pmc run with
    MFMA_COUNTERS (MfmaUtil: the share of the run's busy cycles during which
    the matrix units of all SIMDs were busy, rocprofv3's own derived counter)
    and the kernel time of a --kernel-trace --stats run of the same command:
    the MFMA flops the hardware executed (MOPS x 512) per second of kernel
    time, padding included, against the dense fp32 or bf16 peak; and the
    share of wave cycles spent waiting on LDS and LDS bank conflicts per LDS
    instruction."""
    per = {}
    for ctr in MFMA_COUNTERS:
        for k, v in _counter_rows(pmc_dir, ctr):
            per.setdefault(_short_name(k), {}).setdefault(ctr, []).append(v)
    avg_us = {}
    for f in glob.glob(os.path.join(prof_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                avg_us[_short_name(r["Name"])] = float(r["AverageNs"]) / 1e3

    def mean(v, c):
        x = v.get(c)
        return sum(x) / len(x) if x else 0.0

    print("| kernel | dispatches | avg us | MfmaUtil % | MFMA TFLOP/s (MOPS x 512 / time) | "
          "share of peak | LDS wait / wave cycles | bank conflicts / LDS instr |")
    print("|---|---|---|---|---|---|---|---|")
    rows = []
    for k, v in per.items():
        mops32, mops16 = mean(v, "SQ_INSTS_VALU_MFMA_MOPS_F32"), mean(v, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        if mops32 + mops16 <= 0 or k not in avg_us:
            continue
        t = avg_us[k]
        bf16 = mops16 > mops32
        tf = (mops32 + mops16) * 512 / (t * 1e-6) / 1e12
        peak = PEAK["bf16_TFLOPs" if bf16 else "fp32_TFLOPs"]
        wc = mean(v, "SQ_WAVE_CYCLES")
        lds = mean(v, "SQ_ACTIVE_INST_LDS")
        rows.append((k, len(v.get("MfmaUtil", [])), t, mean(v, "MfmaUtil"), tf, tf / peak,
                     mean(v, "SQ_WAIT_INST_LDS") / wc if wc else 0.0,
                     mean(v, "SQ_LDS_BANK_CONFLICT") / lds if lds else 0.0, bf16))
    for k, n, t, util, tf, frac, lw, bc, bf16 in sorted(rows, key=lambda r: -r[2] * r[1]):
        print(f"| `{k}` | {n} | {t:.2f} | {util:.1f} | {tf:.1f} ({'bf16' if bf16 else 'fp32'}) | "
              f"{100 * frac:.1f}% | {100 * lw:.1f}% | {bc:.2f} |")


def op_rate(cls, work, us, bf16):
    """Achieved rate of an op class from its algorithmic work (flops of a conv
    class, HBM bytes otherwise) and its time per step, against the peak."""
    if cls.startswith(("conv", "deconv")):
        a = work / (us * 1e-6) / 1e12
        peak, unit = PEAK["bf16_TFLOPs" if bf16 else "fp32_TFLOPs"], "TFLOP/s"
    else:
        a = work / (us * 1e-6) / 1e9
        peak, unit = PEAK["hbm_GBps"], "GB/s"
    return {"us_per_step": round(us, 2), "achieved": round(a, 3), "unit": unit, "peak": peak,
            "frac": round(a / peak, 4)}


# Kernel classes of a rocprofv3 trace of this script, by kernel name: the
# build's kernels, the pooling/unpooling kernels, the convolutions' main
# kernels (the MFMA contractions, the pooled forwards among them) and their
# helpers (split sums, the pooled split sum included, ReLU masks, operand
# conversion, gathers and tables).  Anything else (the bench's own torch
# casts) is "other".
TRACE_CLASSES = (
    ("build", ("k_quant", "k_mark", "k_reduce", "k_scan_a", "k_scan_c", "k_leaf_mean", "k_emit",
               "__amd_rocclr_copyBuffer")),
    ("pool", ("k_pool_fwd", "k_route_down", "k_route_up", "k_gpool_", "k_route_parts")),
    ("conv_main", ("k_conv_", "k_cin_", "k_sr_mm<", "k_sr_dw<")),
    ("conv_helper", ("k_sum_", "k_relu_mask", "k_bf_", "k_bf16_to_f32", "k_sr_", "k_dc_",
                     "k_fill_u32")),
)


def trace_class(name):
    for cls, prefixes in TRACE_CLASSES:
        if any(name.startswith(p) for p in prefixes):
            return cls
    return "other"


def pooled_pair(wl, li):
    """True when conv layer li and the 2x2x2 max-pool after it run as one
    conv + pool call (stride 1, fp32)."""
    ls = wl.layers
    L = ls[li]
    return (L.op == "conv" and L.stride == 1 and L.dtype == "f32" and li + 1 < len(ls)
            and ls[li + 1].op == "pool" and ls[li + 1].depth == L.depth)


def summarize_trace(prof_dir, prof_log):
    """Time per step of each kernel class of a rocprofv3 --kernel-trace --stats
    run of this script, against the algorithmic work of the class: conv
    fwd+bwd flops (every kernel of the conv passes, helpers included, and the
    main kernels alone), HBM bytes of the build and of the pooling.  The
    profiled run's own JSON line (in prof_log) gives the workload's sizes and
    step counts."""
    import synth

    line = None
    with open(prof_log) as fh:
        for ln in fh:
            ln = ln.strip()
            if ln.startswith("{") and '"metric"' in ln:
                line = json.loads(ln)
    if line is None:
        raise SystemExit(f"no bench JSON line in {prof_log}")
    cfg = line["config"]
    wl = synth.WORKLOADS[cfg["workload"]]
    acc = Accounting(wl, cfg["octants_per_depth"], cfg["nonempty_per_depth"], cfg["points"])
    nsteps = max(line["warmup"], 2) + line["steps"]
    files = glob.glob(os.path.join(prof_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {prof_dir}")
    kern, table = {}, []
    for f in files:
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                k = _short_name(r["Name"])
                c = kern.setdefault(k, [0, 0.0])
                c[0] += int(r["Calls"])
                c[1] += float(r["TotalDurationNs"]) / 1e3
                table.append((k, int(r["Calls"]), float(r["AverageNs"]) / 1e3,
                              float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
                              float(r["TotalDurationNs"]) / 1e6, float(r["Percentage"])))
    builds = kern.get("k_quant", [0])[0]
    if builds <= 0:
        raise SystemExit("no build kernel (k_quant) in the trace")
    us, names = {}, {}
    for k, (calls, tot) in kern.items():
        cls = trace_class(k)
        us[cls] = us.get(cls, 0.0) + tot / (builds if cls == "build" else nsteps)
        names.setdefault(cls, []).append(k)
    bf16 = any(L.op == "conv" and L.dtype == "bf16" for L in wl.layers)
    flops, _ = acc.conv_flops()
    # a pooling run inside the convolution below it (conv + pool calls) has no
    # forward kernel of its own: its bytes are not the pooling kernels' work
    fused = {i + 1 for i, L in enumerate(wl.layers) if pooled_pair(wl, i)}
    pool_bytes = sum(acc.work(t, L) for i, L in enumerate(wl.layers)
                     if L.op in ("pool", "unpool", "gpool")
                     for t in (L.op + "_fwd", L.op + "_bwd")
                     if not (t == "pool_fwd" and i in fused))
    rows = []
    if us.get("build"):
        rows.append(("build", "build", acc.work("build", None), us["build"]))
    if us.get("pool"):
        rows.append(("pool + unpool, fwd + bwd", "pool", pool_bytes, us["pool"]))
    conv_all = us.get("conv_main", 0.0) + us.get("conv_helper", 0.0)
    rows.append(("conv fwd + bwd, every kernel", "conv", flops, conv_all))
    rows.append(("conv fwd + bwd, main kernels", "conv", flops, us.get("conv_main", 0.0)))
    print(f"Workload `{wl.name}`: {nsteps} network steps and {builds} builds in the trace; "
          f"per-step figures divide each class's total kernel time by those counts. The "
          f"profiled run's own line: {line['ms_per_step']} ms/step.\n")
    print("| class | kernel time per step (us) | algorithmic work per step | achieved | peak | "
          "share of peak |")
    print("|---|---|---|---|---|---|")
    for label, cls, work, t in rows:
        r = op_rate(cls, work, t, bf16)
        w = f"{work / 1e9:.3f} GFLOP" if cls == "conv" else f"{work / 1e6:.2f} MB"
        print(f"| {label} | {t:.1f} | {w} | {r['achieved']:.1f} {r['unit']} | {r['peak']:g} | "
              f"{100 * r['frac']:.1f}% |")
    for cls in ("conv_helper", "other"):
        if us.get(cls):
            print(f"| {cls.replace('_', ' ')} kernels ({', '.join(sorted(names[cls]))}) | "
                  f"{us[cls]:.1f} | | | | |")
    print(f"\nSum of kernel time per step: {sum(us.values()):.1f} us.\n")
    print("Per kernel (rocprofv3 statistics; names longer than 90 characters cut):\n")
    print("| kernel | calls | avg us | min us | max us | total ms | % |")
    print("|---|---|---|---|---|---|---|")
    for k, n, avg, mn, mx, tot, pc in sorted(table, key=lambda r: -r[5]):
        k = k if len(k) <= 90 else k[:87] + "..."
        print(f"| `{k}` | {n} | {avg:.2f} | {mn:.2f} | {mx:.2f} | {tot:.3f} | {pc:.2f} |")


class Accounting:
    """Algorithmic work of a workload's ops from its per-depth sizes: N[l]
    octants and M[l] non-empty octants at depth l, npoints points."""

    def __init__(self, wl, N, M, npoints):
        self.wl, self.N, self.M, self.npoints = wl, list(N), list(M), npoints

    def _n_out(self, L):
        if L.op == "conv":  # stride 2^r: depth - r
            return self.N[L.depth - (L.stride.bit_length() - 1)]
        if L.op == "pool":
            return self.N[L.depth - 1]
        if L.op == "gpool":  # stride 2^r: depth - r
            return self.N[L.depth - (L.stride.bit_length() - 1)]
        return self.N[L.depth]

    def _n_in(self, L):
        if L.op == "conv" or L.stride == 1:
            return self.N[L.depth]
        return self.N[L.depth - (L.stride.bit_length() - 1)]  # strided deconvolution

    def _n_conv(self, L):
        """Rows at which the convolution a conv or deconv layer runs is
        evaluated (a deconvolution runs the passes of the convolution it
        transposes): every depth-l row at stride 1; at stride 2^r only the
        M[l-r] non-empty depth-(l-r) octants (the empty ones get zero rows
        without any arithmetic)."""
        r = L.stride.bit_length() - 1
        return self.N[L.depth] if r == 0 else self.M[L.depth - r]

    def conv_flops(self):
        """Algorithmic flops of the step's conv passes (forward, weight gradient,
        and input gradient except for the first layer, whose input is the
        octree's signal) and the output octants of every conv layer."""
        f = o = 0
        for li, L in enumerate(self.wl.layers):
            if L.op in ("conv", "deconv"):
                n = self._n_conv(L)
                f += (6 if li > 0 else 4) * n * L.ksize ** 3 * L.cin * L.cout
                o += self._n_out(L)
        return f, o

    def work(self, tag, L):
        """Algorithmic flops (MFMA-bound classes) or HBM bytes of one launch."""
        N, M = self.N, self.M
        if tag in ("build_emit", "dw_sum"):  # counted with the first half; no flops
            return 0
        if tag == "build":
            d = self.wl.depth
            return (self.npoints * 24 + sum(8 * N[k] + 4 * M[k] for k in range(d + 1))
                    + 16 * N[d] + sum(108 * M[k - 1] for k in range(1, d + 1)))
        if tag.startswith(("conv", "deconv")):
            return 2 * self._n_conv(L) * L.ksize ** 3 * L.cin * L.cout
        if tag == "round":  # the layer's input: f32 in, bf16 out
            return N[L.depth] * L.cin * 6
        if L is None:  # the head and the update: small, counted as their bytes
            return self.head_bytes(tag)
        l, c = L.depth, L.cin
        if tag == "pool_fwd":
            return N[l] * c * 4 + N[l - 1] * 4 + N[l - 1] * c * 4 + M[l - 1] * c
        if tag == "pool_bwd":
            # per non-empty parent: its gradient row, switches, row index and
            # (a ReLU'd conv below: its pooled output, the ReLU's mask); every
            # child row out
            ls = self.wl.layers
            i = next(k for k, X in enumerate(ls) if X is L)
            P = ls[i - 1] if i > 0 else None
            masked = P is not None and P.op == "conv" and P.relu
            return M[l - 1] * c * (9 if masked else 5) + M[l - 1] * 4 + N[l] * c * 4
        if tag == "unpool_fwd":  # parent rows and switches in, every child row out
            return M[l - 1] * c * 5 + M[l - 1] * 4 + N[l] * c * 4
        if tag == "unpool_bwd":  # the routed child of each (parent, channel) in, parent rows out
            return M[l - 1] * c * 5 + N[l - 1] * 4 + N[l - 1] * c * 4
        if tag == "bn_fwd":  # (with the pooling) one statistics pass over z, then z in,
            # the pooled rows, switches and labels out / in
            c = L.cout
            return N[l] * c * 8 + N[l - 1] * c * 4 + M[l - 1] * c + N[l - 1] * 4
        if tag == "bn_bwd":  # z and dy in for the sums, then z, dy in and dx out
            return N[l] * L.cout * 4 * 5
        if tag in ("gpool_fwd", "gpool_bwd"):
            r = L.stride.bit_length() - 1
            if r == 0:  # rows in and out, switches (max), 27 ints per group
                return N[l] * c * 8 + (N[l] * c if L.mode == "max" else 0) + M[l - 1] * 108
            # strided: the depth-l rows and the depth-(l-r) rows, switches (max),
            # the 8 group-table entries of every output and its label
            return ((N[l] + N[l - r]) * c * 4 + (N[l - r] * c if L.mode == "max" else 0)
                    + N[l - r] * 4 + M[l - r] * 32)
        return 0


    def head_bytes(self, tag):
        """Bytes per launch of the classification head's ops and of the SGD
        update (a rough count for ops of a few microseconds)."""
        wl = self.wl
        if not getattr(wl, "train", False):
            return 0
        B, c2 = wl.batch, wl.layers[-1].cout
        if tag == "sgd":  # w, g, v in; w, v out: all parameters over the two launches / 2
            n = sum(27 * L.cin * L.cout + 2 * L.cout for L in wl.layers)
            n += 8 * c2 * 128 + 128 + 128 * wl.classes + wl.classes
            return 5 * 4 * n // 2
        if tag in ("fc_fwd", "fc_bwd"):
            return 4 * (B * 8 * c2 + 8 * c2 * 128 + B * 128) // 2
        if tag == "dropout":
            return 9 * B * (8 * c2 + 128) // 2
        return 4 * B * wl.classes * 2  # softmax

    def op_class(self, tag):
        """Op class of a tag: the build's two halves are one class."""
        return "build" if tag.startswith("build") else tag


class Step(Accounting):
    """Enqueue one build + forward + backward of a workload's network."""

    def __init__(self, oc, torch, synth, wl):
        self.oc, self.torch, self.wl = oc, torch, wl
        pts, nrm, offs = synth.make_points(wl)
        dev = "cuda"
        self.pts = torch.as_tensor(pts).to(dev)
        self.nrm = torch.as_tensor(nrm).to(dev)
        self.offs = offs
        self.npoints = len(pts)
        self.dtype = torch.float32
        # the weight gradients' partial sums are added by one launch at the end
        # of the backward when every conv layer is stride 1; with a strided
        # layer in the network (stride 4 at depth 6) the deferred pattern made
        # the step's host launches intermittently several times slower, so
        # such networks add each layer's sums in its own call
        self.defer_dw = all(L.stride == 1 for L in wl.layers if L.op == "conv")
        self.weights = {}
        for li, L in enumerate(wl.layers):
            if L.op == "deconv":  # the weight of the convolution it transposes
                w = synth.make_weights(wl, li, L.ksize, L.cout, L.cin)
                self.weights[li] = torch.as_tensor(w).to(dev)
            if L.op == "conv":
                w = synth.make_weights(wl, li, L.ksize, L.cin, L.cout)
                t = torch.as_tensor(w).to(dev)
                if L.dtype == "bf16":
                    t = t.to(torch.bfloat16)
                self.weights[li] = t
        # sizes come from a first build; the upstream gradient of the last
        # layer and the input features of layers that do not read the signal
        # are drawn once and stay resident
        tree = oc.oc_build(self.pts, self.nrm, offs, wl.depth, wl.full_depth)
        self.N = [tree.num(l) for l in range(wl.depth + 1)]
        self.M = [tree.nonempty(l) for l in range(wl.depth + 1)]
        tree.free()
        last = len(wl.layers) - 1
        Ll = wl.layers[last]
        n_last = self._n_out(Ll)
        self.dy_last = torch.as_tensor(
            synth.make_upstream(wl, last, n_last, Ll.cout)).to(dev)
        self.x0 = None
        if not wl.signal_input:
            L0 = wl.layers[0]
            self.x0 = torch.as_tensor(synth.make_features([wl.seed_id, 3000], self._n_in(L0),
                                                          L0.cin)).to(dev)
            if L0.dtype == "bf16":
                self.x0 = self.x0.to(torch.bfloat16)
        self.side = None  # stream for the weight gradients (None: all on one stream)
        # stream for the next batch's build (None: on the network's stream)
        self.bstream = None
        # with a build stream: the layer after whose forward the next build
        # starts (None: at the head of the step)
        self.build_after = BUILD_AFTER.get(wl.name)
        self._job, self._in_step = None, False
        self.cur_ready = None  # event: the current octree's build is done
        self.events = None  # {key: [(start, end, layer), ...]} when recording
        # when a list: every op of the step (not the build) is run with all of
        # its kernels bracketed (oc_profile_calls), one CallProfile per op
        self.calls = None
        self.record = None  # a dict: network() keeps its tensors there
        self.call_pool = [oc.CallProfile(32) for _ in range(3 * len(wl.layers) + 2)]
        self.traced = set()
        # when set: only the (step number % rotate)-th launch of a traced key
        # in each step is bracketed (each bracketing costs the step time)
        self.rotate = None
        self.nstep = 0
        self.ncall = {}
        # the kernel that does the arithmetic of each conv pass, as profilers name it
        tree = oc.oc_build(self.pts, self.nrm, offs, wl.depth, wl.full_depth)
        self.kname = {}
        for li, L in enumerate(wl.layers):
            if L.op == "conv":
                dt = torch.bfloat16 if L.dtype == "bf16" else torch.float32
                for ps, tag in enumerate(("conv_fwd", "conv_bwd_data", "conv_bwd_weight")):
                    # the forward of a conv + pool pair: the pooled kernel
                    pp = 3 if (ps == 0 and self.pooled(li)) else ps
                    self.kname[(li, tag)] = oc.oc_conv_kernel(tree, L.depth, L.ksize, L.stride,
                                                              L.cin, L.cout, pp, dt)
            elif L.op == "deconv":  # the transposed convolution's passes, swapped
                for ps, tag in ((1, "deconv_fwd"), (0, "deconv_bwd_data"), (2, "deconv_bwd_weight")):
                    self.kname[(li, tag)] = oc.oc_conv_kernel(tree, L.depth, L.ksize, L.stride,
                                                              L.cout, L.cin, ps)
        tree.free()

    def pooled(self, li):
        """True when conv layer li and the pooling after it run as one call."""
        return pooled_pair(self.wl, li)

    def routed_pool(self, li):
        """The 2x2x2 max-pool layer right below conv layer li (which made its
        input) when the conv's input gradient is routed through it in the
        same call (stride 1, fp32), else None."""
        ls = self.wl.layers
        L = ls[li]
        if (li >= 1 and L.op == "conv" and L.stride == 1 and L.dtype == "f32"
                and ls[li - 1].op == "pool" and ls[li - 1].depth == L.depth + 1):
            return li - 1
        return None

    def pool_mask(self, li):
        """True when pool layer li sits on a ReLU'd conv: its backward applies
        that ReLU's backward (the pooled values mask the routed gradient)."""
        P = self.wl.layers[li - 1] if li > 0 else None
        return P is not None and P.op == "conv" and P.relu

    # --- one step ----------------------------------------------------------
    def key(self, tag, li):
        """Kernel name of a conv pass; the op class for the other ops."""
        return self.kname.get((li, tag), tag)

    def _run(self, tag, li, fn):
        L = self.wl.layers[li] if li is not None else None
        k = self.key(tag, li)
        if self.calls is not None and not tag.startswith("build"):
            # every kernel of the call, each bracketed by its own events
            if len(self.calls) == len(self.call_pool):
                self.call_pool.append(self.oc.CallProfile(32))
            prof = self.call_pool[len(self.calls)]
            prof.arm()
            try:
                r = fn()
            finally:
                prof.disarm()
            self.calls.append((prof, li, tag))
            return r
        if self.events is not None and (k in self.traced or "*" in self.traced):
            if self.rotate:
                n = self.ncall.get(k, 0)
                self.ncall[k] = n + 1
                if n != self.nstep % self.rotate:
                    return fn()
            torch = self.torch
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            if not tag.startswith("build"):
                # recorded by the library at the start and end of the kernel itself
                a.record()
                b.record()  # instantiates the events
                self.oc.oc_profile_next(a, b)
                r = fn()
            else:
                a.record()
                r = fn()
                b.record()
            self.events.setdefault(k, []).append((a, b, L, tag))
            return r
        return fn()

    def _begin(self):
        """First half of the next batch's build (up to the per-depth counts),
        enqueued at the head of the step."""
        oc, wl = self.oc, self.wl
        return self._run("build", None, lambda: oc.oc_build_async(
            self.pts, self.nrm, self.offs, wl.depth, wl.full_depth))

    def _finish(self, job):
        """Wait for the counts of `job` (queued at the head of the step, so
        they are known while the network still runs) and enqueue the rest of
        its build (leaf signal, keys, labels, neighbour tables) after the
        network, on the same stream."""
        return self._run("build_emit", None, lambda: job.finish())

    def __call__(self):
        """One step: the first half of the next batch's build, the network
        forward and backward on the octree built during the previous step,
        then the rest of the next build.  As in the paper's training (Sec. 3.2,
        last paragraph) the next batch's octree is prepared while the current
        one trains: the host waits for the next build's counts while the device
        runs the network.  With a build stream (bstream) the build's kernels
        run beside the network's (the build is a chain of short,
        latency-bound kernels); the network waits for the build of its octree
        through an event, and the octree's arrays are marked as used on the
        network's stream before it is freed."""
        self.ncall = {}
        torch = self.torch
        B = self.bstream
        if getattr(self, "cur", None) is None:
            self.cur = self._finish(self._begin())
            self.cur_ready = None
        A = torch.cuda.current_stream()
        self._job = None
        if B is None:
            job = self._begin()
        elif self.build_after is None:
            job = self._start_build()
        tree = self.cur
        if self.cur_ready is not None:
            A.wait_event(self.cur_ready)
        self._in_step = B is not None and self.build_after is not None
        try:
            g = self.network(tree)
        finally:
            self._in_step = False
        if B is not None and self.build_after is not None:
            job = self._job if self._job is not None else self._start_build()
        if B is None:
            tree.free()
            self.cur = self._finish(job)
        else:
            tree.record_stream(A)
            tree.free()
            with torch.cuda.stream(B):
                self.cur = self._finish(job)
                self.cur_ready = torch.cuda.Event()
                self.cur_ready.record(B)
        self.nstep += 1
        return g

    def _start_build(self):
        """Queue the first half of the next build on the build stream, after
        everything queued so far on the network's stream (the previous step,
        and with build_after that layer's forward)."""
        torch, B = self.torch, self.bstream
        B.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(B):
            return self._begin()

    def _layer_done(self, li):
        """Called after the forward of layer li: start the next build there
        when it is build_after's layer."""
        if self._in_step and li == self.build_after and self._job is None:
            self._job = self._start_build()

    def drain(self):
        """Nothing of a step is left on the host once it returns."""
        return None

    def network(self, tree):
        oc, wl = self.oc, self.wl
        x = tree.signal() if wl.signal_input else self.x0
        saved = []
        sws = {}  # switches of the pooling at each depth, for the unpooling
        done = -1  # a pool layer already run with the conv below it
        for li, L in enumerate(wl.layers):
            if li > 0:
                self._layer_done(li - 1)
            if li == done:
                continue
            if L.op == "conv" and self.pooled(li):
                # conv + ReLU + pool in one call: the depth-l output is not kept
                w = self.weights[li]
                p, sw = self._run("conv_fwd", li, lambda: oc.oc_conv_pool_fwd(
                    tree, L.depth, L.ksize, x, w, relu=L.relu))
                saved.append((li, x, None, None))
                saved.append((li + 1, None, p, sw))
                sws[L.depth] = sw
                done = li + 1
                x = p
            elif L.op == "conv":
                w = self.weights[li]
                if x.dtype != w.dtype:  # a bf16 layer after an fp32 output
                    x = self._run("round", li, lambda: oc.oc_round_bf16(x))
                y = self._run("conv_fwd", li, lambda: oc.oc_conv_fwd(
                    tree, L.depth, L.ksize, L.stride, x, w, relu=L.relu))
                saved.append((li, x, y, None))
                x = y
            elif L.op == "deconv":
                w = self.weights[li]
                y = self._run("deconv_fwd", li, lambda: oc.oc_deconv_fwd(
                    tree, L.depth, L.ksize, L.stride, x, w))
                saved.append((li, x, y, None))
                x = y
            elif L.op == "gpool":
                mode = oc.OC_POOL_MAX if L.mode == "max" else oc.OC_POOL_AVG
                y, sw = self._run("gpool_fwd", li, lambda: oc.oc_gpool_fwd(
                    tree, L.depth, L.ksize, mode, x, stride=L.stride))
                saved.append((li, x, y, sw))
                x = y
            elif L.op == "pool":
                p, sw = self._run("pool_fwd", li, lambda: oc.oc_pool_fwd(tree, L.depth, x))
                saved.append((li, x, p, sw))
                sws[L.depth] = sw
                x = p
            elif L.op == "unpool":
                sw = sws[L.depth]
                u = self._run("unpool_fwd", li, lambda: oc.oc_unpool_fwd(tree, L.depth, x, sw))
                saved.append((li, x, u, sw))
                x = u
        g = self.dy_last
        masked = False  # g already went through the ReLU of the conv below it
        rec = self.record
        if rec is not None:  # the tensors of this step, for a parity test
            rec["fwd"] = {li: (xin, yout, sw) for li, xin, yout, sw in saved}
            rec["bwd"] = {}
        saved_sw = {li: sw for li, xin, yout, sw in saved}
        routed = set()  # pool layers whose backward ran with the conv above them
        # the weight gradients' partial sums, added by one launch at the end
        pending = []
        for li, xin, yout, sw in reversed(saved):
            L = wl.layers[li]
            g_in, dw = g, None
            if li in routed:
                continue
            if L.op == "conv":
                w = self.weights[li]
                relu = L.relu and not masked
                below = self.routed_pool(li)
                if below is not None:
                    # the input gradient goes straight on through the pooling
                    # that made x (and the ReLU under it): one call, no
                    # depth-l gradient
                    psw, mask = saved_sw[below], self.pool_mask(below)
                    # the ReLU's backward once: the masked dy serves the weight gradient too
                    dym = self.torch.empty_like(g) if relu else None
                    dxf = self._run("conv_bwd_data", li, lambda: oc.oc_conv_bwd_pool(
                        tree, L.depth, L.ksize, w, g, psw, xp=xin if mask else None, y=yout,
                        relu=relu, dym=dym))
                    if dym is not None:
                        g, relu = dym, False
                    routed.add(below)
                    if rec is not None:
                        rec["bwd"][below] = (None, dxf, None)
                    dx = None
                elif li > 0:  # the first layer's input, the signal, needs no gradient
                    dx, _ = self._run("conv_bwd_data", li, lambda: oc.oc_conv_bwd(
                        tree, L.depth, L.ksize, L.stride, xin, w, g, y=yout, relu=relu,
                        need_dx=True, need_dw=False))
                else:
                    dx = None
                dwf = (lambda: oc.oc_conv_bwd(
                    tree, L.depth, L.ksize, L.stride, xin, w, g, y=yout, relu=relu,
                    need_dx=False, need_dw=True, defer=pending if self.defer_dw else None))
                if self.side is None:
                    _, dw = self._run("conv_bwd_weight", li, dwf)
                else:
                    # the weight gradient depends on nothing that follows: it
                    # runs on the side stream beside the rest of the backward
                    torch = self.torch
                    ev = torch.cuda.Event()
                    ev.record()
                    self.side.wait_event(ev)
                    with torch.cuda.stream(self.side):
                        _, dw = self._run("conv_bwd_weight", li, dwf)
                    for t in (xin, g, yout, w):
                        if t is not None:
                            t.record_stream(self.side)
                    tree.record_stream(self.side)
                if below is not None:
                    g, masked = dxf, self.pool_mask(below)
                else:
                    g, masked = dx, False
            elif L.op == "deconv":
                w = self.weights[li]
                dx, _ = self._run("deconv_bwd_data", li, lambda: oc.oc_deconv_bwd(
                    tree, L.depth, L.ksize, L.stride, xin, w, g, need_dx=True, need_dw=False))
                _, dw = self._run("deconv_bwd_weight", li, lambda: oc.oc_deconv_bwd(
                    tree, L.depth, L.ksize, L.stride, xin, w, g, need_dx=False, need_dw=True))
                g, masked = dx, False
            elif L.op == "gpool":
                mode = oc.OC_POOL_MAX if L.mode == "max" else oc.OC_POOL_AVG
                g = self._run("gpool_bwd", li, lambda: oc.oc_gpool_bwd(
                    tree, L.depth, L.ksize, mode, g, sw, stride=L.stride))
                masked = False
            elif L.op == "pool":
                # a ReLU right below the pooling: its backward goes into the routing
                masked = self.pool_mask(li)
                ym = yout if masked else None
                g = self._run("pool_bwd", li, lambda: oc.oc_pool_bwd(tree, L.depth, g, sw, y=ym))
            elif L.op == "unpool":
                g = self._run("unpool_bwd", li, lambda: oc.oc_unpool_bwd(tree, L.depth, g, sw))
                masked = False
            if rec is not None:  # a routed input gradient is the pooling's record
                rec["bwd"][li] = (g_in, None if li - 1 in routed and L.op == "conv" else g, dw)
        if pending:  # on the stream of the weight gradients
            if self.side is None:
                self._run("dw_sum", None, lambda: oc.oc_sum_partials(pending))
            else:
                with self.torch.cuda.stream(self.side):
                    self._run("dw_sum", None, lambda: oc.oc_sum_partials(pending))
        if self.side is not None:
            self.torch.cuda.current_stream().wait_stream(self.side)
        return g

    def collect_calls(self, acc):
        """Add the kernel time of every op of the last step run with
        self.calls set (the device work must be done) to acc: {(layer, tag):
        [ms, calls, launches]}, and reset the list."""
        for prof, li, tag in self.calls:
            a = acc.setdefault((li, tag), [0.0, 0, 0])
            a[0] += prof.kernel_ms()
            a[1] += 1
            a[2] += prof.used
        self.calls = []

    def collect(self):
        """Per-key (total ms, launches, total work, op) of the recorded events."""
        out = {}
        for key, lst in (self.events or {}).items():
            ms = sum(a.elapsed_time(b) for a, b, _, _ in lst)
            work = sum(self.work(tag, L) for _, _, L, tag in lst)
            out[key] = {"ms": ms, "launches": len(lst), "work": work, "op": lst[0][3],
                        "per_layer": [(f"{tag} d{L.depth}" if L is not None else tag,
                                       a.elapsed_time(b)) for a, b, L, tag in lst]}
        return out


class TrainStep(Step):
    """One O-CNN(d) classification training iteration (Sec. 4 "Network
    structure", Sec. 5 "Training details") on the octree built during the
    previous step: units U_d .. U_2 (conv, then batch normalisation, ReLU and
    the 2x2x2 max-pool in one call), the depth-1 features of each shape (8 C_2 values)
    through dropout, FC(128), dropout, FC(classes), softmax cross-entropy on
    synthetic labels; the backward of all of it; one SGD step with momentum
    0.9, weight decay 5e-4 (convolution and FC weights) and learning rate 0.1.
    The parameters live in two flat buffers (with and without weight decay),
    as do their gradients and velocities, so the update is two launches."""

    P_DROP, LR, MOMENTUM, DECAY = 0.5, 0.1, 0.9, 5e-4

    def __init__(self, oc, torch, synth, wl):
        super().__init__(oc, torch, synth, wl)
        d = synth.make_train_inputs(wl)
        dev = "cuda"

        def T(a):
            return torch.as_tensor(a).to(dev)

        self.labels, self.keep1, self.keep2 = T(d["labels"]), T(d["keep1"]), T(d["keep2"])
        # flat buffers: decayed = conv weights, fc1_w, fc2_w; plain = gammas, betas, biases
        dec = [self.weights[li] for li in range(len(wl.layers))] + [T(d["fc1_w"]), T(d["fc2_w"])]
        pla = [T(a) for g_b in d["bn"] for a in g_b] + [T(d["fc1_b"]), T(d["fc2_b"])]
        self.flat = {}
        views = {}
        for key, lst in (("dec", dec), ("pla", pla)):
            n = sum(t.numel() for t in lst)
            buf = {k: torch.zeros(n, dtype=torch.float32, device=dev) for k in ("w", "g", "v")}
            off, vs = 0, []
            for t in lst:
                sl = slice(off, off + t.numel())
                buf["w"][sl].copy_(t.reshape(-1))
                vs.append({k: buf[k][sl].view(t.shape) for k in ("w", "g", "v")})
                off += t.numel()
            self.flat[key] = buf
            views[key] = vs
        nl = len(wl.layers)
        self.conv_p = views["dec"][:nl]
        self.fc1_w, self.fc2_w = views["dec"][nl], views["dec"][nl + 1]
        self.gamma = [views["pla"][2 * i] for i in range(nl)]
        self.beta = [views["pla"][2 * i + 1] for i in range(nl)]
        self.fc1_b, self.fc2_b = views["pla"][2 * nl], views["pla"][2 * nl + 1]
        for li in range(nl):
            self.weights[li] = self.conv_p[li]["w"]
        self.loss = None

    def network(self, tree):
        oc, wl, torch, P = self.oc, self.wl, self.torch, self.P_DROP
        rec = self.record
        x = tree.signal()
        units = []
        for li, L in enumerate(wl.layers):
            w = self.conv_p[li]["w"]
            z = self._run("conv_fwd", li, lambda: oc.oc_conv_fwd(tree, L.depth, 3, 1, x, w))
            # normalisation, ReLU and pooling in one call (the depth-l
            # activations are not kept: the backward needs z and the pooled
            # output only)
            p, sw, mean, invstd = self._run("bn_fwd", li, lambda: oc.oc_bn_pool_fwd(
                tree, L.depth, z, self.gamma[li]["w"], self.beta[li]["w"], relu=True))
            units.append((li, x, z, None, mean, invstd, p, sw))
            x = p
        feat = x.view(wl.batch, -1)
        h0 = self._run("dropout", None, lambda: oc.oc_dropout(feat, self.keep1, P))
        h1 = self._run("fc_fwd", None, lambda: oc.oc_fc_fwd(h0, self.fc1_w["w"], self.fc1_b["w"]))
        h2 = self._run("dropout", None, lambda: oc.oc_dropout(h1, self.keep2, P))
        zl = self._run("fc_fwd", None, lambda: oc.oc_fc_fwd(h2, self.fc2_w["w"], self.fc2_b["w"]))
        loss, dz = self._run("softmax", None, lambda: oc.oc_softmax_ce(zl, self.labels))
        dh2, _, _ = self._run("fc_bwd", None, lambda: oc.oc_fc_bwd(
            h2, self.fc2_w["w"], dz, dw=self.fc2_w["g"], db=self.fc2_b["g"]))
        dh1 = self._run("dropout", None, lambda: oc.oc_dropout(dh2, self.keep2, P))
        dh0, _, _ = self._run("fc_bwd", None, lambda: oc.oc_fc_bwd(
            h0, self.fc1_w["w"], dh1, dw=self.fc1_w["g"], db=self.fc1_b["g"]))
        g = self._run("dropout", None, lambda: oc.oc_dropout(dh0, self.keep1, P)).view(x.shape)
        if rec is not None:
            rec.update(units=units, feat=feat, h0=h0, h1=h1, h2=h2, logits=zl, loss=loss,
                       dlogits=dz, dh1=dh1, dfeat=g, bwd={})
        da_up = None  # the unit above routed its input gradient into this unit's pooling
        pending = []  # the weight gradients' partial sums, added by one launch
        for li, xin, z, a, mean, invstd, p, sw in reversed(units):
            L = wl.layers[li]
            w = self.conv_p[li]["w"]
            g_in = g
            if da_up is None:
                # the ReLU's backward rides on the routing (the pooled output)
                da = self._run("pool_bwd", li, lambda: oc.oc_pool_bwd(tree, L.depth, g, sw, y=p))
            else:
                da = da_up
            dz_, _, _ = self._run("bn_bwd", li, lambda: oc.oc_bn_bwd(
                z, da, self.gamma[li]["w"], mean, invstd, dgamma=self.gamma[li]["g"],
                dbeta=self.beta[li]["g"]))
            da_up = None
            if li > 0:  # the signal needs no gradient
                # the input gradient goes on through the pooling (and ReLU) of
                # the unit below in the same call: that unit's da
                _, _, _, _, _, _, p_below, sw_below = units[li - 1]
                da_up = self._run("conv_bwd_data", li, lambda: oc.oc_conv_bwd_pool(
                    tree, L.depth, 3, w, dz_, sw_below, xp=p_below))
            self._run("conv_bwd_weight", li, lambda: oc.oc_conv_bwd(
                tree, L.depth, 3, 1, xin, w, dz_, need_dx=False, need_dw=True,
                dw_out=self.conv_p[li]["g"], defer=pending))
            if rec is not None:
                rec["bwd"][li] = (g_in, da, dz_, None)
            g = None
        if pending:
            self._run("dw_sum", None, lambda: oc.oc_sum_partials(pending))
        if rec is not None:  # parameters and velocities before the update
            rec["before"] = {k: {q: b[q].clone() for q in ("w", "v")} for k, b in self.flat.items()}
        for key, dec in (("dec", self.DECAY), ("pla", 0.0)):
            b = self.flat[key]
            self._run("sgd", None, lambda: oc.oc_sgd(b["w"], b["g"], b["v"], self.LR,
                                                     self.MOMENTUM, dec))
        self.loss = loss
        return loss


def oracle_step(synth, wl, shapes):
    """The oracle on the first `shapes` shapes of the batch: build, neighbour
    search and the network's forward and backward.  Returns (algorithmic conv
    flops of the step, seconds on the host)."""
    import oracle

    pts, nrm, offs = synth.make_points(wl, batch=shapes)
    t0 = time.perf_counter()
    ref = oracle.Octree(pts, nrm, offs, wl.depth, wl.full_depth)
    L0 = wl.layers[0]
    x = ref.signal if wl.signal_input else synth.make_features(
        [wl.seed_id, 3000], ref.num(L0.depth - (L0.op == "deconv" and L0.stride == 2)), L0.cin)
    saved, flops, sws = [], 0, {}
    for li, L in enumerate(wl.layers):
        l = L.depth
        if L.op == "conv":
            nb = ref.neighbors(l, L.ksize, stride=L.stride)
            w = synth.make_weights(wl, li, L.ksize, L.cin, L.cout)
            pre = oracle.conv_fwd(nb, x, w)
            r = L.stride.bit_length() - 1
            if r > 0:
                pre = oracle.renew(ref.labels(l - r), pre)
            y = oracle.relu_fwd(pre) if L.relu else pre
            saved.append((li, nb, x, w, pre))
            flops += (6 if li > 0 else 4) * nb.shape[0] * L.ksize ** 3 * L.cin * L.cout
            x = y
        elif L.op == "deconv":
            w = synth.make_weights(wl, li, L.ksize, L.cout, L.cin)
            if L.stride == 1:
                nb = ref.neighbors(l, L.ksize)
                y = oracle.deconv_fwd(nb, x, w, ref.num(l))
            else:
                y = oracle.deconv_sr_fwd(ref, l, x, w, L.stride)
            saved.append((li, None, x, w, None))
            n = ref.num(l) if L.stride == 1 else ref.nonempty(l - (L.stride.bit_length() - 1))
            flops += 6 * n * L.ksize ** 3 * L.cin * L.cout
            x = y
        elif L.op == "pool":
            y, sw = oracle.pool_fwd(ref.labels(l - 1), x)
            saved.append((li, None, x, sw, None))
            sws[l] = sw
            x = y
        elif L.op == "unpool":
            sw = sws[l]
            y = oracle.unpool_fwd(ref.labels(l - 1), x, sw, ref.num(l))
            saved.append((li, None, x, sw, None))
            x = y
        elif L.op == "gpool":
            mode = oracle.POOL_MAX if L.mode == "max" else oracle.POOL_AVG
            if L.stride == 1:
                nb = ref.neighbors(l, L.ksize)
                y, sw = oracle.gpool_fwd(nb, x, mode)
            else:
                nb = None
                y, sw = oracle.gpool_sr_fwd(ref, l, x, mode, L.stride)
            saved.append((li, nb, x, sw, mode))
            x = y
    g = synth.make_upstream(wl, len(wl.layers) - 1, x.shape[0], x.shape[1])
    for li, nb, xin, w_or_sw, pre in reversed(saved):
        L = wl.layers[li]
        l = L.depth
        if L.op == "conv":
            ge = oracle.relu_bwd(pre, g) if L.relu else g
            r = L.stride.bit_length() - 1
            if r > 0:
                ge = oracle.renew_bwd(ref.labels(l - r), ge, nb.shape[0])
            oracle.conv_bwd_weight(nb, xin, ge, L.ksize ** 3)
            g = oracle.conv_bwd_data(nb, ge, w_or_sw, xin.shape[0]) if li > 0 else None
        elif L.op == "deconv":
            if L.stride == 1:
                g, _ = oracle.deconv_bwd(ref.neighbors(l, L.ksize), xin, w_or_sw, g)
            else:
                g, _ = oracle.deconv_sr_bwd(ref, l, xin, w_or_sw, g, L.stride)
        elif L.op == "unpool":
            g = oracle.unpool_bwd(ref.labels(l - 1), g, w_or_sw)
        elif L.op == "gpool":
            if L.stride == 1:
                g = oracle.gpool_bwd(nb, g, w_or_sw, ref.num(l), pre)
            else:
                g = oracle.gpool_sr_bwd(ref, l, g, w_or_sw, ref.num(l), pre, L.stride)
        else:
            g = oracle.pool_bwd(ref.labels(l - 1), g, w_or_sw, ref.num(l))
    return flops, time.perf_counter() - t0


def oracle_train_step(synth, wl, shapes):
    """The oracle's O-CNN(d) training iteration (oracle/train.py) on the first
    `shapes` shapes: build, forward, backward, SGD.  (conv flops, seconds)."""
    import numpy as np

    import oracle
    from oracle import train as T

    pts, nrm, offs = synth.make_points(wl, batch=shapes)
    d = synth.make_train_inputs(wl, batch=shapes)
    params = []
    for li, L in enumerate(wl.layers):
        params += [synth.make_weights(wl, li, 3, L.cin, L.cout), d["bn"][li][0], d["bn"][li][1]]
    params += [d["fc1_w"], d["fc1_b"], d["fc2_w"], d["fc2_b"]]
    params = [np.asarray(q, np.float64) for q in params]
    vel = [np.zeros_like(q) for q in params]
    t0 = time.perf_counter()
    ref = oracle.Octree(pts, nrm, offs, wl.depth, wl.full_depth)
    T.ocnn_step(ref, params, vel, d["labels"], d["keep1"], d["keep2"])
    flops = sum((6 if li > 0 else 4) * ref.num(L.depth) * 27 * L.cin * L.cout
                for li, L in enumerate(wl.layers))
    return flops, time.perf_counter() - t0


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(synth, wl, max_shapes, budget_s=4.0):
    """The oracle (as it stands, float64) timed on the host: a warm-up run on
    one shape, then, at all threads and at one thread, the median of three
    runs on the first s shapes of the batch, s sized from the warm-up so that
    one run takes about budget_s seconds (at most max_shapes).  The one-thread
    leg is skipped when a single shape would take over 30 s."""
    import oracle

    threads = oracle.num_threads()
    run = oracle_train_step if wl.train else oracle_step
    f1, t1 = run(synth, wl, 1)  # warm-up (page faults, thread start)

    def leg(nthr):
        oracle.set_num_threads(nthr)
        per_shape = t1 * threads / nthr  # an upper bound: perfect scaling over the threads
        if per_shape > 30.0 and nthr == 1:
            return None
        s = max(1, min(max_shapes, int(budget_s / max(per_shape, 1e-3))))
        runs = sorted(run(synth, wl, s) for _ in range(3))
        flops, dt = runs[1]
        return {"value": round(flops / dt / 1e9, 4), "shapes": s, "seconds": round(dt, 3),
                "gflop": round(flops / 1e9, 3)}

    try:
        one = leg(1)
        full = leg(threads)
    finally:
        oracle.set_num_threads(threads)
    return {"value": full["value"], "unit": "GFLOP/s", "cores": threads, "kind": "oracle",
            "value_all": full["value"], "value_1t": one["value"] if one else None,
            "cpu_model": cpu_model(),
            "sample": f"one step (build, neighbour search, forward and backward"
                      f"{', SGD update' if wl.train else ''}, float64) of the "
                      f"first {full['shapes']} of {wl.batch} shapes at {threads} threads "
                      f"({full['gflop']} GFLOP, median of 3: {full['seconds']} s)"
                      + (f", and of the first {one['shapes']} shapes at 1 thread "
                         f"({one['gflop']} GFLOP, median of 3: {one['seconds']} s)" if one else
                         ", 1 thread skipped (over 30 s per shape)")
                      + "; oracle built with g++ -O3"}


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters, args.copy_probe, args.workload)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
              f"(the path would shard by shape with one dW all-reduce per layer, not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1712_01537_amd as oc
    import synth

    oc.load()  # raises if liboc.so is missing: there is no other implementation
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.workload]
    print(f"[bench] workload {wl.name}: generating inputs", file=sys.stderr, flush=True)
    step = (TrainStep if wl.train else Step)(oc, torch, synth, wl)
    if args.streams == 2:
        step.side = torch.cuda.Stream()  # default priority, like the main stream
    if not args.build_inline:
        step.bstream = torch.cuda.Stream()  # default priority, like the main stream
    flops, octants = step.conv_flops()
    print(f"[bench] N_l = {step.N}, M_l = {step.M}", file=sys.stderr, flush=True)

    # warmup, every op timed; the kernel (conv passes) or op class with the
    # largest share of the step is the dominant one
    # (the first step's one-time costs, such as loading GEMM kernels, are not
    # counted)
    # warmup steps 1, 3, ... bracket each op's main kernel (oc_profile_next),
    # steps 2, 4, ... every kernel of each op (oc_profile_calls)
    step.events, step.traced = {}, {"*"}
    nwarm = max(args.warmup, 3)
    allk = {}
    n_main = n_all = 0
    for i in range(nwarm):
        if i == 1:
            torch.cuda.synchronize()
            step.events = {}
        if i >= 1 and i % 2 == 0:
            saved_events, step.events, step.calls = step.events, None, []
            step()
            torch.cuda.synchronize()
            step.collect_calls(allk)
            step.events, step.calls = saved_events, None
            n_all += 1
        else:
            step()
            n_main += i >= 1
    step.drain()
    torch.cuda.synchronize()
    warm = step.collect()
    nwarm = n_main
    # the build (part at the head of the step, part on its own stream) is not a
    # convolution or pooling class, and the deferred weight-gradient sums are
    # counted with their layers' passes
    dominant = max((k for k in warm if warm[k]["op"] in BOUND
                    and not warm[k]["op"].startswith("build")),
                   key=lambda k: warm[k]["ms"])
    print(f"[bench] warmup done; dominant kernel: {dominant}", file=sys.stderr, flush=True)

    # timed region: K steps; events bracket one launch of the dominant kernel
    # per step, the launches taken in turn
    nper = max(1, warm[dominant]["launches"] // nwarm)
    step.events, step.traced, step.rotate, step.nstep = {}, {dominant}, nper, 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    step.drain()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    dom = step.collect()[dominant]
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)

    # mean time of each launch of the step (layer), then their sum against
    # their work: every launch weighs the same however often it was sampled
    by = {}
    for a, b, L, tag in step.events[dominant]:
        t = by.setdefault((tag, L.depth if L is not None else -1), [0.0, 0, step.work(tag, L)])
        t[0] += a.elapsed_time(b)
        t[1] += 1
    per_launch_ms = sum(t[0] / t[1] for t in by.values()) / len(by)
    per_launch_work = sum(t[2] for t in by.values()) / len(by)
    bound = BOUND[dom["op"]]
    if bound == "mfma":
        achieved = per_launch_work / (per_launch_ms * 1e-3) / 1e12
        bf16 = any(L is not None and L.dtype == "bf16" for _, _, L, _ in step.events[dominant])
        peak, unit = PEAK["bf16_TFLOPs" if bf16 else "fp32_TFLOPs"], "TFLOP/s"
    else:
        achieved = per_launch_work / (per_launch_ms * 1e-3) / 1e9
        peak, unit = PEAK["hbm_GBps"], "GB/s"
    traffic = load_traffic(wl.name, dominant)
    roofline = {"bound": bound, "kernel": dominant, "op": dom["op"], "achieved": round(achieved, 3),
                "peak": peak, "unit": unit, "frac": round(achieved / peak, 4),
                "traffic": traffic["bytes"] if traffic else None,
                "launches_per_step": nper,
                "mean_launch_us": round(per_launch_ms * 1e3, 2)}
    if traffic:
        roofline["traffic_detail"] = traffic

    # every op class's main kernels in the warmup, against its work
    ops = {}
    for v in warm.values():
        c = ops.setdefault(step.op_class(v["op"]), [0.0, 0.0])
        c[0] += v["ms"] * 1e3 / nwarm
        c[1] += v["work"] / nwarm
    bf16 = any(L.op == "conv" and L.dtype == "bf16" for L in wl.layers)
    # the build's events also span host work (the wait for its counts): its
    # rate comes from a kernel trace (--summarize-trace) instead
    ops.pop("build", None)
    ops_out = {c: op_rate(c, w, t, bf16) for c, (t, w) in sorted(ops.items()) if t > 0 and w > 0}
    conv = [v for c, v in ops.items() if c.startswith(("conv", "deconv"))]
    if conv:
        ops_out["conv_fwd_bwd"] = op_rate("conv", sum(w for _, w in conv),
                                          sum(t for t, _ in conv), bf16)
    # every kernel of the conv passes (split sums, ReLU masks, operand
    # conversions and gathers included), per layer and in total
    layers, tot_us, tot_work = [], 0.0, 0.0
    for li, L in enumerate(wl.layers):
        if L.op not in ("conv", "deconv"):
            continue
        tags = (("conv_fwd", "conv_bwd_data", "conv_bwd_weight") if L.op == "conv" else
                ("deconv_fwd", "deconv_bwd_data", "deconv_bwd_weight"))
        us, work = {}, 0.0
        for tag in tags:
            a = allk.get((li, tag))
            if a and a[1]:
                us[tag.split("_", 1)[1]] = round(a[0] * 1e3 / a[1], 2)
                work += step.work(tag, L)
        t = sum(us.values())
        if t <= 0:
            continue
        r = op_rate("conv", work, t, L.dtype == "bf16")
        layers.append({"layer": li, "op": L.op, "depth": L.depth, "ksize": L.ksize,
                       "stride": L.stride, "cin": L.cin, "cout": L.cout, "dtype": L.dtype,
                       "rows": step._n_conv(L), "us": us, "us_total": round(t, 2),
                       "gflops": round(work / (t * 1e-6) / 1e9, 1),
                       "octants_per_s": round(step._n_out(L) / (t * 1e-6), 1),
                       "frac": r["frac"]})
        tot_us += t
        tot_work += work
    # the weight gradients' partial sums of all layers, one launch per step
    a = allk.get((None, "dw_sum"))
    if a and a[1]:
        tot_us += a[0] * 1e3 / a[1]
    if tot_us > 0:
        ops_out["conv_fwd_bwd_all"] = op_rate("conv", tot_work, tot_us, bf16)

    if args.layers:
        for key, v in sorted(warm.items(), key=lambda kv: -kv[1]["ms"]):
            per = {}
            for name, t in v["per_layer"]:
                per[name] = per.get(name, 0.0) + t / nwarm
            print(f"[bench] {key:42s} {v['ms'] / nwarm:8.3f} ms/step  "
                  + "  ".join(f"{k}:{t:.3f}" for k, t in per.items()), file=sys.stderr)

    if args.copy_probe > 0:
        n = args.copy_probe * 2 ** 20 // 4
        src = torch.randn(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):  # an elementwise kernel (a plain copy could go to a DMA engine)
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        print(f"[bench] copy probe: 3 copies of {args.copy_probe} MiB", file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_shapes > 0:
        print(f"[bench] cpu oracle, up to {args.cpu_shapes} shapes", file=sys.stderr, flush=True)
        cpu = cpu_baseline(synth, wl, min(args.cpu_shapes, wl.batch))

    line = {
        "metric": "octree-conv fwd+bwd GFLOP/s & octants/s per layer; % HBM/MFMA roofline",
        "value": round(flops / (ms * 1e-3) / 1e9, 3),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if all(L.dtype == "f32" for L in wl.layers) else "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "description": WORKLOAD_TEXT.get(wl.name, ""),
            "batch": wl.batch,
            "depth": wl.depth,
            "points": step.npoints,
            "octants_per_depth": step.N,
            "nonempty_per_depth": step.M,
            "conv_gflop_per_step": round(flops / 1e9, 4),
        },
        "octants_per_s": round(octants / (ms * 1e-3), 1),
        "roofline": roofline,
        "ops": ops_out,
        "ops_scope": "warmup HIP events: per op class around its main kernel; conv_fwd_bwd_all "
                     "and layers around every kernel of the conv passes (split sums, ReLU "
                     "masks, conversions and gathers included); the build is measured from a "
                     "kernel trace",
        "layers": layers,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


WORKLOAD_TEXT = {
    "net_d6": "32 shapes (unions of 1-4 spheres/boxes, 20k surface points each), depth-6 "
              "octree built on the GPU each step; conv3+ReLU+maxpool 3->16 @d6, 16->32 @d5, "
              "32->64 @d4, 64->128 @d3, conv3+ReLU 128->256 @d2; fp32 forward and backward",
    "net_d5": "32 shapes, depth 5; conv3 3->32 @d5 + pool, 32->64 @d4 + pool, 64->128 @d3 + "
              "pool, 128->256 @d2; fp32 forward and backward",
    "sphere_d5": "one sphere, 20k points, depth 5; conv3 3->32 + pool; fp32 fwd+bwd",
    "deep_d8": "8 shapes, 100k points each, depth 8; conv3 16->16 @d8, pool, unpool; fp32",
    "wide_d7": "16 shapes, 100k points each, depth 7; conv5 64->64 and stride-2 conv3 "
               "64->128, bf16 inputs with fp32 accumulation",
    "gpool_d6": "32 shapes, depth 6; conv3+ReLU 3->16 @d6, stride-1 3x3x3 max-pool and 5x5x5 "
                "average-pool @d6 (the convolution's neighbourhood), 2x2x2 max-pool d6->d5, "
                "3x3x3 max-pool stride 2 d5->d4, 3x3x3 average-pool stride 4 d4->d2; fp32 "
                "forward and backward",
    "ocnn_d6": "O-CNN(6) classification training iteration on 32 shapes (20k surface points "
               "each), octree built on the GPU each step: U_6 .. U_2 (conv3 + batch norm + ReLU "
               "+ 2x2x2 max-pool; 3->8, 8->16, 16->32, 32->64, 64->128), dropout 0.5, FC(128), "
               "dropout, FC(40), softmax cross-entropy on synthetic labels, backward, SGD "
               "(momentum 0.9, weight decay 5e-4); fp32",
    "s4_d6": "32 shapes, depth 6; conv3+ReLU 3->16 @d6, stride-4 conv3+ReLU 16->64 d6->d4, "
             "conv3 64->128 @d4; fp32 forward and backward",
    "seg_d6": "32 shapes, depth 6; encoder conv3+ReLU+maxpool 3->16 @d6, 16->32 @d5; decoder "
              "stride-2 deconv3 32->16 d4->d5, max-unpool d5->d6, deconv3 16->16 @d6; fp32 "
              "forward and backward",
}


if __name__ == "__main__":
    main()
