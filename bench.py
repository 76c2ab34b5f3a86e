#!/usr/bin/env python3
"""Throughput of carry-through protected CNN inference on one MI355X.

A step is one pass of the whole protected path over one batch: input
staging, every conv / pool / FC layer (the carry-through channels computed
inside the normal conv tiles), the detector, and re-execution of flagged
images (deferred: they join the batch two steps later; the run ends with a
flush).  The threshold is calibrated first from fault-free inferences
(distribution-based, alpha = 1%), so about alpha of the images are re-run.

Default workload: VGG-16, fp16, batch 32, 3x224x224 synthetic inputs and
seeded random weights (the largest single-GPU configuration).  Prints one
JSON line (rank 0).  Other measurements:
  overhead_pct    protected vs the same kernels without carry-through
                  channels: ABAB-interleaved blocks of a test-set-sized
                  stream (--abab-images per block, independent of --steps),
                  each protected block ending with its flush; medians
  flush_ms        the end-of-stream flush of the timed region on its own
  mfma_util       dense-conv algorithmic FLOPs / their kernel time / peak
  roofline        the kernel with the most device time: HIP events that
                  the library records on its own stream around every
                  launch of a profiled run of full-batch passes (every
                  launch processes exactly `batch` images)
  cpu_baseline    the CPU oracle on the host cores, on a bounded sample
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("images/sec with carry-through checksum; % overhead vs "
          "unprotected; MFMA util")
PEAK = {"f32": 157.3e12, "f16": 2.5e15}     # dense MFMA, per GPU
HBM_PEAK = 8.0e12                            # bytes/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the first ~100 passes of a protected run are up to ~8% slower than
    # later ones: the default timed region is long enough to be steady
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="vgg16_f16_b32")
    ap.add_argument("--alpha", type=float, default=0.01)
    ap.add_argument("--no-fuse", action="store_true",
                    help="run every op as its own kernel (fusion off)")
    ap.add_argument("--mode", choices=("replace", "append"), default="replace",
                    help="carry-through channel replaces each layer's last "
                         "channel (the paper's construction) or is appended")
    ap.add_argument("--ncal", type=int, default=2048)
    ap.add_argument("--pool", type=int, default=8,
                    help="distinct input batches resident in HBM")
    ap.add_argument("--abab", type=int, default=7,
                    help="protected/unprotected block pairs")
    ap.add_argument("--abab-images", type=int, default=10000,
                    help="images per ABAB block (a test-set-sized stream)")
    ap.add_argument("--prof-steps", type=int, default=50,
                    help="full-batch passes of the profiled run")
    ap.add_argument("--graph-passes", type=int, default=None,
                    help="passes captured per HIP graph for the graph-replay "
                         "figure (default: 2000 for batch-1 workloads, "
                         "otherwise none)")
    ap.add_argument("--graph-reps", type=int, default=9,
                    help="protected/unprotected graph replay pairs")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="also time the library GEMM (torch.matmul) of each "
                         "dense conv's implicit-GEMM shape and print it "
                         "beside the conv kernel's profiled time")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also run a 256 MiB device copy (HBM counter "
                         "calibration under rocprofv3 --pmc)")
    ap.add_argument("--summarize-trace", metavar="DB",
                    help="print a markdown table of per-kernel device time "
                         "from a rocprofv3 --kernel-trace database and exit")
    ap.add_argument("--summarize-sq", metavar="DIR",
                    help="print a markdown table of MFMA and LDS counters "
                         "from a rocprofv3 --pmc run and exit")
    ap.add_argument("--summarize-counters", metavar="DIR",
                    help="print a markdown table of every counter of a "
                         "rocprofv3 --pmc run per kernel (dispatch averages; "
                         "with SQ_WAVE_CYCLES, also per wave-cycle) and exit")
    ap.add_argument("--traffic-table", action="store_true",
                    help="print a markdown table of the committed HBM "
                         "traffic of each kernel of --workload against its "
                         "algorithmic bytes per launch (no GPU needed)")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, "
                         "WRITE_SIZE) under DIR into a traffic summary in "
                         "profiles/ and exit")
    return ap.parse_args()


def layer_flops(net):
    """Algorithmic FLOPs per image of every layer (2 per multiply-add;
    conv/FC only), with the deployed output widths."""
    shp = net.shapes()
    out = []
    for i, L in enumerate(net.layers):
        if L["op"] == "conv":
            c, p, q = shp[i + 1]
            out.append(2.0 * p * q * c * (L["c_in"] // L["groups"])
                       * L["k"] * L["k"])
        elif L["op"] == "fc":
            rows = L["out_f"] + (1 if L["final"] else 0)
            out.append(2.0 * rows * L["in_f"])
        else:
            out.append(0.0)
    return out


def layer_bytes(net):
    """Algorithmic HBM bytes per image of every layer: read input (and
    residual) once, write output once, plus the layer's weights read once
    per pass of net.batch images."""
    shp = net.shapes()
    eb = 2 if net.dtype == "f16" else 4
    out = []
    for i, L in enumerate(net.layers):
        ci = math.prod(shp[L["inp"]])
        co = math.prod(shp[i + 1])
        r = co if (L["op"] == "conv" and L["residual"] >= 0) else 0
        if L["op"] == "conv":
            w = L["c_out"] * (L["c_in"] // L["groups"]) * L["k"] * L["k"]
        elif L["op"] == "fc":
            w = (L["out_f"] + (1 if L["final"] else 0)) * L["in_f"]
        else:
            w = 0
        out.append(float((ci + co + r) * eb + w * eb / net.batch))
    return out


def kernels_hash():
    h = hashlib.sha256()
    for f in ("kernels.hip", "kernels.h"):
        with open(os.path.join(ROOT, "paper_2609_16742_amd", "csrc", f),
                  "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_file(kernel, workload):
    safe = "".join(ch if ch.isalnum() else "_" for ch in kernel).strip("_")
    return os.path.join(ROOT, "profiles", "traffic_%s_%s.json"
                        % (safe, workload))


def load_traffic(kernel, workload):
    f = traffic_file(kernel, workload)
    if not os.path.exists(f):
        return None
    d = json.load(open(f))
    if d.get("kernels_sha") != kernels_hash():
        return None           # kernel changed since the counters were read
    return d.get("bytes_per_launch")


# --------------------------------------------------------------- CPU leg

def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(net, params, ref, tau, seconds, max_images=4096):
    """The oracle as it stands on the host cores, on the bench's own input
    stream: chunks of one image per thread until `seconds` have passed (at
    least one chunk, at most max_images images)."""
    import numpy as np
    import oracle
    from workloads import gen
    threads = min(16, os.cpu_count() or 1)
    dp = oracle.protect_params(net, params)
    n_done, t0 = 0, time.perf_counter()
    chunk = threads
    while n_done < max_images and (n_done == 0 or
                                   time.perf_counter() - t0 < seconds):
        xb = gen.make_inputs(net, min(chunk, max_images - n_done),
                             offset=n_done)
        out = oracle.forward_batch(net, dp, xb, threads=threads)
        fl = oracle.verify(out[:, -1], ref, tau)
        for j in np.nonzero(fl)[0]:          # re-execute flagged images
            oracle.forward_image(net, dp, xb[j])
        n_done += len(xb)
    dt = time.perf_counter() - t0
    return {"value": n_done / dt, "unit": "images/s", "cores": threads,
            "kind": "oracle",
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": "%d images of the same workload (protected forward, "
                      "detector, re-execution of flagged images), one "
                      "image per thread in flight, %d threads, %.1f s"
                      % (n_done, threads, dt)}


# ------------------------------------------------------- PMC summarising

def _counter_rows(d):
    """(demangled kernel name, counter, value, duration ns) of every
    dispatch in the rocprofv3 databases under d."""
    import glob
    import sqlite3
    names = {}
    for f in glob.glob(os.path.join(d, "**", "*_results.db"), recursive=True):
        c = sqlite3.connect(f)
        cols = [r[1] for r in c.execute("pragma table_info(counters_collection)")]
        dur = "duration" if "duration" in cols else "0"
        for name, counter, val, ns in c.execute(
                "select kernel_name, counter_name, value, %s from "
                "counters_collection" % dur):
            if name not in names:
                names[name] = _demangle(name) if name.startswith("_Z") else name
            yield names[name], counter, val, ns


def _short(name):
    return name.split("(")[0].replace("void ", "").replace("ctc::", "")


# The short bench run every counter pass profiles.
PMC_FLAGS = ("--steps 5 --warmup 2 --abab 1 --abab-images 64 --ncal 64 "
             "--prof-steps 5 --no-cpu-baseline --copy-calib")


def summarize_pmc(d, workload):
    """Reads the rocprofv3 databases of a FETCH_SIZE run and a WRITE_SIZE
    run (anywhere under d; counters in KiB per dispatch) of
    `bench.py --copy-calib`, scales each counter so that the three 256 MiB
    device copies read (and write) 3 x 256 MiB, and returns per kernel of
    the library {counter: (bytes per launch, scale)}."""
    agg = {}
    copies = {}
    for name, counter, val, _ in _counter_rows(d):
        if "copyBuffer" in name or "direct_copy" in name:
            if val > 32 * 1024:                 # the calibration copies
                copies[counter] = copies.get(counter, 0.0) + val
            continue
        if "ctc::" in name:
            agg.setdefault((counter, name), []).append(val)
    res = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        if counter not in copies:
            continue
        cal = 3 * 256 * 2 ** 20 / (copies[counter] * 1024.0)
        for (cn, k), vs in agg.items():
            if cn == counter:
                res.setdefault(k, {})[counter] = (
                    sum(vs) / len(vs) * 1024.0 * cal, cal)
    return res


# MI355X: 8 XCDs of 32 CUs, 4 SIMDs per CU.  GRBM_GUI_ACTIVE counts GPU
# cycles summed over the XCDs; SQ_VALU_MFMA_BUSY_CYCLES counts busy cycles
# of every SIMD's matrix core.
XCDS, SIMDS = 8, 256 * 4


SQ_COUNTERS = ("SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_F16 "
               "SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS "
               "SQ_WAIT_INST_LDS GRBM_GUI_ACTIVE")


def summarize_sq(d):
    """Per-kernel SQ / GRBM counter averages from a rocprofv3 --pmc run
    (anywhere under d): MFMA busy fraction, the MFMA FLOPs the counters saw
    (512 per F16 MOP), LDS bank-conflict cycles per LDS-active cycle, the
    clock.  Returns {kernel: {...}} and a markdown table of it."""
    agg = {}
    for name, counter, val, ns in _counter_rows(d):
        if "ctc::" not in name:
            continue
        a = agg.setdefault(_short(name), {})
        a.setdefault(counter, []).append(val)
        a.setdefault("_ns", []).append(ns)
    out = ["| kernel | dispatches | MFMA busy | MFMA TFLOP/s (counters) | "
           "LDS conflict / active | clock GHz |",
           "|---|---:|---:|---:|---:|---:|"]
    res = {}
    for k, a in agg.items():
        m = {c: sum(v) / len(v) for c, v in a.items()}
        g = m.get("GRBM_GUI_ACTIVE", 0.0) / XCDS
        busy = m.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        ns = m.get("_ns", 0.0)
        ldsa = m.get("SQ_LDS_IDX_ACTIVE", 0.0)
        res[k] = {
            "dispatches": len(a["_ns"]) // max(1, len(a) - 1),
            "mfma_busy": busy / (g * SIMDS) if g else None,
            "mfma_tflops": (m.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) * 512
                            / (ns * 1e-9) / 1e12) if ns else None,
            "lds_conflict": (m.get("SQ_LDS_BANK_CONFLICT", 0.0) / ldsa
                             if ldsa else None),
            "clock_ghz": g / ns if ns else None,
            "_busy": busy}
    nan = float("nan")
    for k, r in sorted(res.items(), key=lambda kv: -kv[1]["_busy"]):
        out.append("| `%s` | %d | %.3f | %.1f | %.3f | %.2f |" % (
            k, r["dispatches"],
            *(nan if r[f] is None else r[f] for f in
              ("mfma_busy", "mfma_tflops", "lds_conflict", "clock_ghz"))))
        del r["_busy"]
    return res, "\n".join(out)


def summarize_counters(d):
    """Markdown table of the dispatch-averaged value of every counter of a
    rocprofv3 --pmc run (anywhere under d), per kernel of this library,
    slowest first.  SQ_WAVE_CYCLES (summed over the waves, in units of 4
    cycles like the SQ's other cycle counters) is the denominator of a
    second row per kernel: the fraction of a wave's resident cycles spent
    issuing or waiting."""
    agg = {}
    for name, counter, val, ns in _counter_rows(d):
        if "ctc::" not in name:
            continue
        a = agg.setdefault(_short(name), {})
        a.setdefault(counter, []).append(val)
        a.setdefault("_ns", []).append(ns)
    cols = sorted({c for a in agg.values() for c in a if c != "_ns"})
    out = ["| kernel | us | " + " | ".join(cols) + " |",
           "|---|---:|" + "---:|" * len(cols)]
    for k, a in sorted(agg.items(), key=lambda kv: -sum(kv[1]["_ns"])
                       / len(kv[1]["_ns"])):
        m = {c: sum(v) / len(v) for c, v in a.items()}
        out.append("| `%s` | %.1f | %s |" % (k, m["_ns"] / 1e3, " | ".join(
            "%.4g" % m.get(c, 0.0) for c in cols)))
        wc = m.get("SQ_WAVE_CYCLES")
        if wc:
            out.append("| (per wave-cycle) | | %s |" % " | ".join(
                "" if c in ("SQ_WAVE_CYCLES", "SQ_WAVES", "GRBM_GUI_ACTIVE")
                else "%.3f" % (m.get(c, 0.0) / wc) for c in cols))
    return "\n".join(out)


def sq_file(workload):
    return os.path.join(ROOT, "profiles", "sq_%s.json" % workload)


def load_sq(kernel, workload):
    """Counter-measured MFMA busy fraction of a kernel, when the committed
    counters were read from the kernels as they are now."""
    f = sq_file(workload)
    if not os.path.exists(f):
        return None
    d = json.load(open(f))
    if d.get("kernels_sha") != kernels_hash():
        return None
    return d["kernels"].get(kernel, {}).get("mfma_busy")


# ------------------------------------------------------------------ main

def _demangle(name):
    """Readable name of a mangled kernel symbol (rocprofv3 leaves those with
    _Float16 template arguments mangled): the _Float16 code is swapped for
    the half-float one, which the system c++filt knows, and renamed back."""
    import subprocess
    try:
        r = subprocess.run(["c++filt"], input=name.replace("DF16_", "Dh"),
                           capture_output=True, text=True, timeout=10)
        out = r.stdout.strip()
        return out.replace("half", "_Float16") if out else name
    except (OSError, subprocess.SubprocessError):
        return name


def summarize_trace(db):
    """Per-kernel calls / total / average duration from a rocprofv3
    --kernel-trace --stats SQLite output (its top_kernels view)."""
    import sqlite3
    c = sqlite3.connect(db)
    rows = list(c.execute("select name, total_calls, total_duration, "
                          "average, percentage from top_kernels"))
    out = ["| kernel | calls | total us | avg us | % |",
           "|---|---:|---:|---:|---:|"]
    for name, n, tot, avg, pct in rows:
        if name.startswith("_Z"):
            name = _demangle(name)
        short = name.split("(")[0].replace("void ", "")
        if len(short) > 90:
            short = short[:87] + "..."
        out.append("| `%s` | %d | %.1f | %.3f | %.2f |"
                   % (short, n, tot, avg, pct))
    return "\n".join(out)


def kernel_roof(d, peak):
    """Bound, achieved and fraction of peak of one kernel from its profiled
    launches: MFMA-bound above the ridge point (flops per byte of the MFMA
    peak over the HBM peak), else HBM-bound."""
    n = max(d["launches"], 1)
    us = d["ms"] / n * 1e3
    ai = d["flops"] / d["bytes"] if d["bytes"] > 0 else float("inf")
    if d["ms"] <= 0:
        return {"avg_launch_us": us, "launches": d["launches"]}
    if ai >= peak / HBM_PEAK:
        a = d["flops"] / (d["ms"] * 1e-3)
        return {"bound": "mfma", "avg_launch_us": round(us, 3),
                "launches": d["launches"], "achieved_tflops": round(a / 1e12, 1),
                "alg_mb_per_launch": round(d["bytes"] / n / 1e6, 3),
                "frac": round(a / peak, 4)}
    a = d["bytes"] / (d["ms"] * 1e-3)
    return {"bound": "hbm", "avg_launch_us": round(us, 3),
            "launches": d["launches"], "achieved_gbs": round(a / 1e9, 1),
            "alg_mb_per_launch": round(d["bytes"] / n / 1e6, 3),
            "frac": round(a / HBM_PEAK, 4)}


def merge_fused(net, names, launches, lf, lb):
    """Ops that run inside the kernel of an earlier op (the library names
    them by that kernel and launches nothing for them: a conv's fused 2x2
    pool, the second conv of a fused residual block, a fused GAP + FC ...)
    add their flops and bytes to the launching op, less the write and read
    of each tensor passed between them inside the kernel.  Returns the set
    of merged ops."""
    shp = net.shapes()
    eb = 2 if net.dtype == "f16" else 4
    merged = set()
    owner = None
    for i in range(len(net.layers)):
        if launches[i] == 0 and owner is not None and names[i] == names[owner]:
            lf[owner] += lf[i]
            lb[owner] += lb[i] - 2.0 * math.prod(shp[net.layers[i]["inp"]]) * eb
            lf[i] = lb[i] = 0.0
            merged.add(i)
        elif launches[i] > 0:
            owner = i
    return merged


def alg_bytes_by_kernel(net, names):
    """Algorithmic HBM bytes of every kernel per launch at the net's batch:
    the layer_bytes of the ops it runs, averaged over its launches per pass.
    Without a GPU the launches are not measured: a max pool named by the
    kernel of the conv before it counts as fused into it (the fused pools
    of the fp16 networks), and so do the depthwise and project convs of a
    fused inverted residual block; every other op as a launch of its own
    (not true of the fused residual blocks of the fp32 networks)."""
    lb = layer_bytes(net)
    lf = layer_flops(net)
    nops = len(net.layers)

    def inside(i):
        L = net.layers[i]
        if i == 0 or names[i] != names[i - 1]:
            return False
        if L["op"] == "maxpool":
            return True
        if names[i].startswith("conv_ir"):
            prev = net.layers[i - 1]
            return L["groups"] > 1 or (prev["op"] == "conv" and prev["groups"] > 1)
        return False

    launches = [0 if inside(i) else 1 for i in range(nops)]
    fused = merge_fused(net, names, launches, lf, lb)
    out = {}
    for i in range(nops):
        if i in fused:
            continue
        d = out.setdefault(names[i], [0.0, 0])
        d[0] += lb[i] * net.batch
        d[1] += 1
    return {k: (v[0] / v[1], v[1]) for k, v in out.items()}


def traffic_table(workload):
    from paper_2609_16742_amd import ctc
    from workloads import config
    net = config(workload)
    h = ctc.ctc_net_create(ctc.ops_from_layers(net.layers), net.in_shape[0],
                           net.in_shape[1], net.in_shape[2], net.classes,
                           ctc.DTYPES[net.dtype], 1)
    names = [ctc.ctc_net_op_kernel(h, i, net.batch)
             for i in range(len(net.layers))]
    alg = alg_bytes_by_kernel(net, names)
    out = ["| kernel | launches / pass | algorithmic MB / launch | FETCH MB | "
           "WRITE MB | counted / algorithmic |",
           "|---|---:|---:|---:|---:|---:|"]
    for k, (b, n) in sorted(alg.items(), key=lambda kv: -kv[1][0] * kv[1][1]):
        f = traffic_file(k, workload)
        if not os.path.exists(f):
            out.append("| `%s` | %d | %.1f | - | - | - |" % (k, n, b / 1e6))
            continue
        d = json.load(open(f))
        stale = d.get("kernels_sha") != kernels_hash()
        out.append("| `%s` | %d | %.1f | %.1f | %.1f | %.2f%s |" % (
            k, n, b / 1e6, d["fetch_bytes_per_launch"] / 1e6,
            d["write_bytes_per_launch"] / 1e6, d["bytes_per_launch"] / b,
            " (stale)" if stale else ""))
    return "\n".join(out)


def gemm_reference(net, B, names, launches, ms, reps=20):
    """Per dense conv op run by a single-conv kernel: its implicit GEMM
    (M = B P Q pixels, K = C R S, N output channels) timed as a plain
    library GEMM (torch.matmul, operands resident, no im2col) against the
    op's own profiled launch time."""
    import torch

    shp = net.shapes()
    lf = layer_flops(net)
    tdt = torch.float16 if net.dtype == "f16" else torch.float32
    seen, rows = {}, []
    for i, L in enumerate(net.layers):
        n_l = int(launches[1 + i])
        if (L["op"] != "conv" or L["groups"] != 1 or n_l == 0 or
                not names[i].startswith(("conv_pp", "conv_dma", "conv_img"))):
            continue
        c, p, q = shp[i + 1]
        M, K, N = B * p * q, L["c_in"] * L["k"] * L["k"], c
        if (M, K, N) not in seen:
            a = torch.randn(M, K, device="cuda", dtype=tdt)
            b = torch.randn(K, N, device="cuda", dtype=tdt)
            for _ in range(3):
                a @ b
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                a @ b
            e1.record()
            torch.cuda.synchronize()
            seen[(M, K, N)] = e0.elapsed_time(e1) / reps * 1e3
            del a, b
        g = seen[(M, K, N)]
        ours = ms[1 + i] / n_l * 1e3
        rows.append({"op": i, "kernel": names[i], "M": M, "K": K, "N": N,
                     "gemm_us": g, "gemm_tflops": 2.0 * M * N * K / g * 1e-6,
                     "ours_us": ours, "ours_tflops": lf[i] * B / ours * 1e-6})
    print("| op | kernel | M x K x N | library GEMM us (TF/s) | conv kernel us "
          "(TF/s) |", file=sys.stderr)
    print("|---:|---|---|---:|---:|", file=sys.stderr)
    for r in rows:
        print("| %d | `%s` | %d x %d x %d | %.1f (%.0f) | %.1f (%.0f) |"
              % (r["op"], r["kernel"], r["M"], r["K"], r["N"], r["gemm_us"],
                 r["gemm_tflops"], r["ours_us"], r["ours_tflops"]),
              file=sys.stderr)
    return rows


def graph_figures(ctc, net, prot, unprot, B, passes, reps, stream):
    """Microseconds per inference with `passes` passes of B images captured
    as one HIP graph (ctc_graph_*): protected replays re-execute their
    flagged images before returning (CTC_REEXEC_SYNC, the host waits),
    unprotected replays are waited for; ABAB-interleaved, medians."""
    import numpy as np
    import torch
    from workloads import gen

    n = B * passes
    x = torch.from_numpy(gen.make_inputs(net, n, offset=10 ** 6)).to(
        prot.ws.device)
    fl = torch.zeros(n, dtype=torch.uint8, device=x.device)
    g_p = prot.graph(x, B, flags=fl)
    g_u = unprot.graph(x, B)
    g_p.launch(ctc.CTC_REEXEC_SYNC, stream)
    g_u.launch(ctc.CTC_REEXEC_NONE, stream)
    torch.cuda.synchronize()
    tp, tu, nf = [], [], []
    for _ in range(reps):
        torch.cuda.synchronize()
        a0 = time.perf_counter()
        nf.append(g_p.launch(ctc.CTC_REEXEC_SYNC, stream))
        torch.cuda.synchronize()
        a1 = time.perf_counter()
        g_u.launch(ctc.CTC_REEXEC_NONE, stream)
        torch.cuda.synchronize()
        a2 = time.perf_counter()
        tp.append(a1 - a0)
        tu.append(a2 - a1)
    tpm, tum = float(np.median(tp)), float(np.median(tu))
    return {"passes": passes, "batch": B, "images": n, "replays": reps,
            "us_per_inference": tpm / n * 1e6,
            "us_per_inference_unprotected": tum / n * 1e6,
            "images_per_s": n / tpm,
            "overhead_pct": (tpm - tum) / tum * 100.0,
            "flagged_per_replay": float(np.median(nf)),
            "reexec": "sync (flagged images re-run before the replay "
                      "returns)"}


def main():
    args = parse()
    if args.traffic_table:
        print(traffic_table(args.workload))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters))
        return
    if args.summarize_sq:
        res, table = summarize_sq(args.summarize_sq)
        rec = {"workload": args.workload, "kernels_sha": kernels_hash(),
               "commands": [
                   "timeout -s KILL 150 rocprofv3 --pmc %s -d DIR -o p -- "
                   "python -u bench.py --workload %s %s"
                   % (SQ_COUNTERS, args.workload,
                      PMC_FLAGS.replace(" --copy-calib", "")),
                   "python bench.py --workload %s --summarize-sq DIR"
                   % args.workload],
               "kernels": res}
        with open(sq_file(args.workload), "w") as fh:
            json.dump(rec, fh, indent=1)
        print(table)
        return
    if args.summarize_pmc:
        res = summarize_pmc(args.summarize_pmc, args.workload)
        for full, d in res.items():
            if "FETCH_SIZE" not in d or "WRITE_SIZE" not in d:
                continue
            short = _short(full)
            rec = {"kernel": short, "workload": args.workload,
                   "kernels_sha": kernels_hash(),
                   "fetch_bytes_per_launch": d["FETCH_SIZE"][0],
                   "write_bytes_per_launch": d["WRITE_SIZE"][0],
                   "fetch_scale": d["FETCH_SIZE"][1],
                   "write_scale": d["WRITE_SIZE"][1],
                   "bytes_per_launch": d["FETCH_SIZE"][0] + d["WRITE_SIZE"][0],
                   "source": "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, "
                             "scaled by a 256 MiB device copy",
                   "commands": [
                       "timeout -s KILL 150 rocprofv3 --pmc %s -d DIR/%s_%s "
                       "-o p -- python -u bench.py --workload %s %s"
                       % (c, c, args.workload, args.workload, PMC_FLAGS)
                       for c in ("FETCH_SIZE", "WRITE_SIZE")] + [
                       "python bench.py --workload %s --summarize-pmc DIR"
                       % args.workload]}
            with open(traffic_file(short, args.workload), "w") as fh:
                json.dump(rec, fh, indent=1)
            print(json.dumps(rec))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: there is no multi-GPU path "
              "(every image is independent, so the work would shard as "
              "plain data parallelism with nothing exchanged per "
              "inference).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_16742_amd as P
    from paper_2609_16742_amd import ctc
    from workloads import config, gen

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    net = config(args.workload)
    B = net.batch
    params = gen.make_params(net)
    prot = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                    protect=args.mode, max_batch=B, device=dev)
    if args.no_fuse:
        prot.set_fusion(False)
    unprot = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype,
                      params, protect=False, max_batch=B, device=dev)
    if args.no_fuse:
        unprot.set_fusion(False)

    # distribution-based threshold from fault-free inferences (Sec. II-C)
    S = []
    for s in range(0, args.ncal, B):
        n = min(B, args.ncal - s)
        xc = torch.from_numpy(gen.make_inputs(net, n, stream=gen.S_CALIB,
                                              offset=s)).to(dev)
        S.append(prot.forward(xc)[:, -1].double().cpu().numpy())
    S = np.concatenate(S)
    ref, tau = ctc.ctc_threshold_from_samples(S, args.alpha)
    prot.set_threshold(ref, tau)

    # resident inputs and rotating outputs
    x_host = gen.make_inputs(net, B * args.pool)
    xs = [torch.from_numpy(x_host[i * B:(i + 1) * B]).to(dev)
          for i in range(args.pool)]
    outs_p = [torch.empty((B, net.classes + 1), device=dev)
              for _ in range(args.pool)]
    outs_u = [torch.empty((B, net.classes), device=dev)
              for _ in range(args.pool)]
    flags = [torch.zeros(B, dtype=torch.uint8, device=dev)
             for _ in range(args.pool)]
    stream = torch.cuda.current_stream()
    DEF = ctc.CTC_REEXEC_DEFERRED

    def run_prot(k0, k):
        for i in range(k0, k0 + k):
            j = i % args.pool
            ctc.ctc_network_forward(prot.h, B, xs[j], outs_p[j], flags[j],
                                    DEF, stream)
        ctc.ctc_network_flush(prot.h, stream)

    def run_unprot(k0, k):
        for i in range(k0, k0 + k):
            j = i % args.pool
            ctc.ctc_network_forward(unprot.h, B, xs[j], outs_u[j], None,
                                    ctc.CTC_REEXEC_NONE, stream)

    if args.copy_calib:                      # HBM counter calibration
        a = torch.empty(256 * 2 ** 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    # warmup
    run_prot(0, args.warmup)
    run_unprot(0, max(1, args.warmup // 2))
    torch.cuda.synchronize()

    # timed region: K protected steps (with re-execution) and the flush
    flagged = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        j = i % args.pool
        ctc.ctc_network_forward(prot.h, B, xs[j], outs_p[j], flags[j], DEF,
                                stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctc.ctc_network_flush(prot.h, stream)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for f in flags:                         # last pool's worth of flags
        flagged += int(f.sum().item())
    flag_rate = flagged / float(B * min(args.pool, args.steps))
    elapsed = t2 - t0
    value = B * args.steps / elapsed
    ms_per_step = elapsed / args.steps * 1e3
    flush_ms = (t2 - t1) * 1e3

    # protection overhead: ABAB-interleaved blocks of a test-set-sized
    # stream, medians (each protected block ends with a flush, as a job
    # would); the block length does not depend on --steps
    kb = max(1, -(-args.abab_images // B))
    tp, tu = [], []
    for r in range(args.abab):
        for which in ("p", "u"):
            torch.cuda.synchronize()
            a0 = time.perf_counter()
            (run_prot if which == "p" else run_unprot)(r * kb, kb)
            torch.cuda.synchronize()
            (tp if which == "p" else tu).append(time.perf_counter() - a0)
    tpm, tum = float(np.median(tp)), float(np.median(tu))
    overhead = (tpm - tum) / tum * 100.0

    # profiled run: per-op device time from HIP events the library records
    # around each launch on its stream.  Deferred passes always run exactly
    # B inferences (re-runs join later passes); the flush, whose last pass
    # may be partial, runs after the profile is read, so every profiled
    # launch processed B images.
    kprof = max(1, args.prof_steps)
    ctc.ctc_network_flush(prot.h, stream)
    torch.cuda.synchronize()
    ctc.ctc_net_profile(prot.h, 1)
    for i in range(kprof):
        j = i % args.pool
        ctc.ctc_network_forward(prot.h, B, xs[j], outs_p[j], flags[j], DEF,
                                stream)
    launches, ms = ctc.ctc_net_profile_read(prot.h, len(net.layers))
    ctc.ctc_net_profile(prot.h, 0)
    ctc.ctc_network_flush(prot.h, stream)
    torch.cuda.synchronize()
    nops = len(net.layers)
    gref = None
    if args.gemm_reference:
        gref = gemm_reference(net, B, [ctc.ctc_net_op_kernel(prot.h, i, B)
                                       for i in range(nops)], launches, ms)
    lf = layer_flops(net)
    lb = layer_bytes(net)
    names = [ctc.ctc_net_op_kernel(prot.h, i, B) for i in range(nops)]
    merge_fused(net, names, [int(launches[1 + i]) for i in range(nops)], lf, lb)
    by_kernel = {}
    for i in range(nops):
        name = names[i]
        d = by_kernel.setdefault(name, {"ms": 0.0, "launches": 0,
                                        "flops": 0.0, "bytes": 0.0})
        n_l = int(launches[1 + i])
        d["ms"] += ms[1 + i]
        d["launches"] += n_l
        d["flops"] += lf[i] * B * n_l        # B images per launch
        d["bytes"] += lb[i] * B * n_l
    dom_name, dom = max(by_kernel.items(), key=lambda kv: kv[1]["ms"])
    peak = PEAK[net.dtype]
    # bound by the kernel's own arithmetic intensity against the ridge point
    # (MFMA peak / HBM peak): the 3x3 convs are MFMA-bound, pointwise convs
    # with few channels, depthwise, pooling and the FCs HBM-bound
    ai = dom["flops"] / dom["bytes"] if dom["bytes"] > 0 else float("inf")
    is_conv = ai >= peak / HBM_PEAK
    if is_conv:
        achieved = dom["flops"] / (dom["ms"] * 1e-3)
        roof = {"bound": "mfma", "achieved": achieved / 1e12,
                "peak": peak / 1e12, "unit": "TFLOP/s",
                "frac": achieved / peak}
    else:
        achieved = dom["bytes"] / (dom["ms"] * 1e-3)
        roof = {"bound": "hbm", "achieved": achieved / 1e9,
                "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                "frac": achieved / HBM_PEAK}
    tb = load_traffic(dom_name, args.workload)
    roof["traffic"] = tb
    if is_conv:
        roof["mfma_busy_counters"] = load_sq(dom_name, args.workload)
    roof["kernel"] = dom_name
    roof["arith_intensity"] = ai
    roof["avg_launch_us"] = dom["ms"] / max(dom["launches"], 1) * 1e3
    roof["launches"] = dom["launches"]
    roof["algorithmic_per_launch"] = (dom["flops"] if is_conv else
                                      dom["bytes"]) / max(dom["launches"], 1)
    conv_ms = sum(d["ms"] for k, d in by_kernel.items()
                  if k.startswith("conv_"))
    conv_fl = sum(d["flops"] for k, d in by_kernel.items()
                  if k.startswith("conv_"))
    mfma_util = conv_fl / (conv_ms * 1e-3) / peak if conv_ms > 0 else None
    # passes in the profiled run: the launches of the op that launches
    # most often (every pass runs the first op's kernel; a fused op's
    # launch is counted at the op that starts it)
    passes = max(max(int(launches[1 + i]) for i in range(nops)), 1)
    dev_ms_per_step = float(ms.sum()) / passes

    line = {
        "metric": METRIC, "value": value, "unit": "images/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": net.dtype,
        "data": "synthetic",
        "config": {"workload": args.workload,
                   "description": "%s %s batch %d, input %s, seeded random "
                                  "weights, carry-through filters in every "
                                  "conv (%s mode), deferred re-execution, "
                                  "alpha %g"
                                  % (net.name, net.dtype, B,
                                     "x".join(map(str, net.in_shape)),
                                     args.mode, args.alpha),
                   "batch": B, "parallelism": "single GPU"},
        "overhead_pct": overhead,
        "overhead_block_images": B * kb,
        "overhead_blocks": args.abab,
        "unprotected_images_per_s": B * kb / tum,
        "protected_block_images_per_s": B * kb / tpm,
        "flush_ms": flush_ms,
        "flag_rate": flag_rate,
        "threshold": {"method": "distribution", "alpha": args.alpha,
                      "n_cal": int(args.ncal), "ref": ref, "tau": tau},
        "mfma_util": mfma_util,
        "device_ms_per_step": dev_ms_per_step,
        "per_kernel_ms_per_step": {k: v["ms"] / passes
                                   for k, v in sorted(
                                       by_kernel.items(),
                                       key=lambda kv: -kv[1]["ms"])},
        # every kernel against its own roofline (algorithmic flops or bytes
        # per launch / its event-timed launch), as the dominant one below
        "per_kernel_roofline": {k: kernel_roof(v, peak)
                                for k, v in sorted(
                                    by_kernel.items(),
                                    key=lambda kv: -kv[1]["ms"])},
        "roofline": roof,
    }
    if gref is not None:
        line["gemm_reference"] = gref
    gp = args.graph_passes if args.graph_passes is not None else (
        2000 if B == 1 else 0)
    if gp > 0:
        line["graph"] = graph_figures(ctc, net, prot, unprot, B, gp,
                                      args.graph_reps, stream)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(net, params, ref, tau,
                                            args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
