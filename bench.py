#!/usr/bin/env python3
"""Benchmark of the SAMD b-bit quantized conv2d on one MI355X.

Workload: conv2d 8 x 128 x 56 x 56 -> 128 channels, 3x3, stride 1, pad 1, unsigned b-bit
activations x signed b-bit weights (seeded synthetic values), swept over b = 1..8.

One step = one pass of the whole hot path at every bit width: pack the uint8
activations into b-bit words, spread them into operand words (stage), multiply,
accumulate, decode and store (accumulate).  Each layer's kernel words are prepared once,
before timing, as weights are constant, and each layer's plan is tuned at set-up.  The
8 layers are independent, so the step runs them round-robin on 4 side streams (default
priority) that fork from and join the launching stream.  `value` is the whole sweep's
throughput (all MACs of the 8 layers / wall time of the step) in GMAC/s, with the step
replayed from a captured HIP graph; `eager_ms_per_step` is the same step launched
kernel by kernel from Python.  Per bit width the line also reports each kernel's own duration (HIP events
around a graph of back-to-back launches of that kernel alone), the
native-int8 matrix-core baseline on the same layer, their speedup, and the roofline
fractions; the CPU oracle is timed on the host.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--bits 1,2,...]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

PEAK_VALU_OPS = 256 * 64 * 2.4e9      # int32 VALU lane-ops/s: 256 CUs x 64 lanes x 2.4 GHz
PEAK_HBM = 8.0e12                     # bytes/s
PEAK_I8_MACS = 2.5e15                 # dense int8 matrix-core MAC/s (5.0 POP/s)
PEAK_LDS = 256 * 256 * 2.4e9          # LDS read bytes/s: 256 CUs x 256 B/clk x 2.4 GHz


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--step-warm-s", type=float, default=0.5,
                   help="seconds of back-to-back step replays before the timed steps (at least --warmup replays)")
    p.add_argument("--samples", type=int, default=5,
                   help="timed graph replays per kernel timing (median and min reported)")
    p.add_argument("--no-peak-check", action="store_true",
                   help="skip the short v_mad_i64_i32 issue-rate measurement reported next to the roofline")
    p.add_argument("--peaks", action="store_true",
                   help="instead of the default workload, measure the ceilings: v_mad_i64_i32 and int32 add issue "
                        "rates, int8 MFMA rate, streaming copy and read bandwidth")
    p.add_argument("--bits", default="1,2,3,4,5,6,7,8")
    p.add_argument("--reps", type=int, default=20, help="back-to-back launches per kernel timing")
    p.add_argument("--kernel-warm-s", type=float, default=0.2,
                   help="seconds of back-to-back replays before each kernel's timed replay (clocks settle)")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU oracle sample budget")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-check", action="store_true", help="skip the sampled parity check")
    p.add_argument("--no-tune", action="store_true",
                   help="use the planner's model plans (default: time the top candidates at set-up)")
    p.add_argument("--tune-candidates", type=int, default=16, help="candidate plans timed per bit width")
    p.add_argument("--no-tune-int8", action="store_true",
                   help="use the int8 baseline's own launch choice (default: time every candidate launch at "
                        "set-up and keep the fastest, as the SAMD plans are tuned)")
    p.add_argument("--streams", type=int, default=4,
                   help="streams the step's independent bit widths are spread over (every stream at the "
                        "default priority)")
    p.add_argument("--stream-order", choices=("snake", "round-robin"), default="snake",
                   help="how bit widths map to streams: snake pairs the smallest width with the largest "
                        "(1+8, 2+7, ...: balanced work per stream), round-robin takes them in order")
    p.add_argument("--plans-out", metavar="FILE", help="write the plans used per bit width (JSON)")
    p.add_argument("--plans-in", metavar="FILE",
                   help="use the plans of a --plans-out file instead of tuning (profiled runs replay the plans "
                        "of an untraced one)")
    p.add_argument("--counters", action="store_true",
                   help="launch each kernel once per bit width, eagerly, then a 1 GiB streaming copy, and exit "
                        "(the program rocprofv3 --pmc passes run)")
    p.add_argument("--vggb", action="store_true",
                   help="instead of the default workload, sweep the ten VGG-B convolution layers (batch 1) over "
                        "N-bit signed activations and weights, N = 8..2 (or --bits), SAMD and int8 baseline")
    p.add_argument("--stack", action="store_true",
                   help="instead of the default workload, time the AlexNet-shaped five-layer stack (b = 2, 4, 8 or "
                        "--bits): SAMD with packed or operand-word activations between layers, and int8")
    p.add_argument("--configs", action="store_true",
                   help="instead of the default workload, time the other workloads: the single small layer, "
                        "the 2^20-value conv1d (b = 1..8, 3 and 5 taps) and the extremes-heavy signed layer")
    p.add_argument("--conv1d", action="store_true",
                   help="instead of the default workload, time the 2^20-value conv1d (b = 1..8, 3 and 5 taps) "
                        "next to a store-only kernel writing the same output bytes")
    p.add_argument("--spacers", action="store_true",
                   help="instead of the default workload, compare temporary and permanent spacer bits per bit width "
                        "on the single, mid-size and extremes-heavy layers: time and HBM bytes of a convolution from "
                        "packed activations (spread + multiply) and from the permanent-spacer layout (multiply)")
    p.add_argument("--lanewise", action="store_true",
                   help="instead of the default workload, time lane-wise add/sub/mul/scale on packed words (GB/s)")
    p.add_argument("--int8-counters", action="store_true",
                   help="launch every int8 baseline candidate once on the --int8-layer layer (b = 4), eagerly, and "
                        "exit (the program rocprofv3 --pmc passes of the int8 kernels run)")
    p.add_argument("--int8-layer", choices=sorted(INT8_LAYERS), default="mid",
                   help="layer of --int8-counters and --int8-summary: the mid-size layer, VGG-B layer 1 or an "
                        "AlexNet-shaped stack layer (batch 16)")
    p.add_argument("--int8-summary", nargs="+", metavar="PMC_DIR",
                   help="print the counter table of --int8-counters runs profiled with rocprofv3 --pmc (one "
                        "folder per pass)")
    p.add_argument("--valu-summary", metavar="PMC_DIR",
                   help="print the VALU / texture-path counter table of a --counters run profiled with "
                        "rocprofv3 --pmc " + VALU_COUNTERS)
    p.add_argument("--trace-summary", metavar="TRACE_DIR",
                   help="print markdown tables of a rocprofv3 --kernel-trace --stats output folder (csv) and exit")
    p.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="print the HBM-traffic summary of two rocprofv3 --pmc output folders of --counters runs "
                        "(FETCH_SIZE, then WRITE_SIZE) and exit")
    return p.parse_args()


HERE = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(HERE, "profiles", "conv2d_samd_mid_sweep_hbm_traffic.md")
COPY_BYTES = 1 << 30                  # the calibration copy reads and writes this many bytes


def kernel_source_sha():
    """Hash of the sources that decide what the SAMD conv kernel reads and writes."""
    import hashlib
    h = hashlib.sha256()
    for f in ("conv2d_samd.hip", "plan.cpp", "samd_internal.hpp"):
        with open(os.path.join(HERE, "paper_1809_10572_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_counter_csv(folder, counter):
    """{dispatch id: (kernel name, value)} of one counter from a rocprofv3 csv output folder."""
    import csv
    import glob
    files = glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one counter_collection.csv under {folder}, found {len(files)}")
    out = {}
    with open(files[0]) as fh:
        for row in csv.DictReader(fh):
            if row["Counter_Name"] == counter:
                d = int(row["Dispatch_Id"])
                name, v = out.get(d, (row["Kernel_Name"], 0.0))
                out[d] = (name, v + float(row["Counter_Value"]))
    return out


VALU_COUNTERS = ("SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_VMEM_RD SQ_INSTS_LDS SQ_INSTS_SALU SQ_WAIT_INST_ANY "
                 "SQ_WAVE_CYCLES SQ_BUSY_CYCLES TA_TA_BUSY_sum TD_TD_BUSY_sum GRBM_GUI_ACTIVE")


def valu_summary(folder, bits_list, plans_file=None):
    """Markdown table of one `rocprofv3 --pmc <VALU_COUNTERS>` pass over `bench.py --counters`:
    per bit width, the SAMD conv kernel's dispatch duration, VALU instructions, VALU issue
    utilisation (4 clocks per wave-wide VALU instruction on a SIMD16, over 1024 SIMDs and
    the dispatch's duration at 2.4 GHz), the share of multiply-adds among them, the
    method's efficiency (direct MACs per VALU lane-operation, every VALU instruction
    counted), and the texture-path (TA/TD) busy fractions over the 256 compute units."""
    import csv
    import glob

    import paper_1809_10572_amd as samd
    import samd_workloads as wl

    files = glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one counter_collection.csv under {folder}, found {len(files)}")
    disp = {}
    for row in csv.DictReader(open(files[0])):
        d = disp.setdefault(int(row["Dispatch_Id"]), {"name": row["Kernel_Name"], "c": {}})
        d["c"][row["Counter_Name"]] = d["c"].get(row["Counter_Name"], 0.0) + float(row["Counter_Value"])
        d["dur"] = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-9
    conv = [disp[k] for k in sorted(disp) if "conv2d_samd_kernel" in disp[k]["name"]]
    if len(conv) != len(bits_list):
        raise SystemExit(f"{len(conv)} conv dispatches for bits {bits_list}")
    plans = json.load(open(plans_file)) if plans_file else None
    shape = wl.MID
    out = ["| b | dispatch µs | VALU wave-instructions | VALU issue % | multiply-adds % of VALU | "
           "multiply-adds % of VALU peak | MACs per VALU lane-op | VMEM reads | LDS instructions | TA busy % | "
           "TD busy % |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    for b, d in zip(bits_list, conv):
        xf, wf = samd.Fmt(b, False), samd.Fmt(b, True)
        if plans:
            samd.conv2d_use_plan(shape, xf, wf, plans[str(b)])
        p = samd.conv2d_plan(shape, xf, wf)
        Ho, _ = samd.out_hw(shape)
        mads = shape.N * shape.M * Ho * p.words_per_row * shape.C * shape.KH * p.tap_words
        macs = shape.N * shape.M * Ho * samd.out_hw(shape)[1] * shape.C * shape.KH * shape.KW
        c, dur = d["c"], d["dur"]
        cycles = dur * 2.4e9
        valu = c["SQ_INSTS_VALU"]
        out.append(f"| {b} | {dur * 1e6:.1f} | {valu:.4g} | {100 * valu * 4 / (1024 * cycles):.0f} | "
                   f"{100 * mads / 64 / valu:.0f} | {100 * mads / dur / PEAK_VALU_OPS:.0f} | {macs / (64 * valu):.2f} | "
                   f"{c['SQ_INSTS_VMEM_RD']:.4g} | {c['SQ_INSTS_LDS']:.4g} | "
                   f"{100 * c['TA_TA_BUSY_sum'] / (256 * cycles):.0f} | {100 * c['TD_TD_BUSY_sum'] / (256 * cycles):.0f} |")
    return "\n".join(out)


def traffic_summary(fetch_dir, write_dir, bits_list):
    """HBM bytes per launch of the SAMD conv kernel at each bit width, from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) scaled by what the counters read for a copy of known size."""
    per = {}
    for key, folder, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = read_counter_csv(folder, counter)
        order = sorted(rows)
        conv = [rows[d][1] for d in order if "conv2d_samd_kernel" in rows[d][0]]
        copy = [rows[d][1] for d in order if "bitwise_not" in rows[d][0]]
        if len(conv) != len(bits_list) or len(copy) < 1:
            raise SystemExit(f"{folder}: {len(conv)} conv dispatches for bits {bits_list}, {len(copy)} copies")
        factor = COPY_BYTES / (copy[-1] * 1024.0)
        per[key] = (conv, copy[-1], factor)
    res = {"kernel": "conv2d_samd_kernel", "source_sha256": kernel_source_sha(),
           "copy": {"bytes_each_way": COPY_BYTES, "fetch_kib": per["fetch"][1], "write_kib": per["write"][1],
                    "fetch_factor": round(per["fetch"][2], 4), "write_factor": round(per["write"][2], 4)},
           "per_bits": {}}
    tot = 0.0
    for i, b in enumerate(bits_list):
        fk, wk = per["fetch"][0][i], per["write"][0][i]
        fb, wb = fk * 1024 * per["fetch"][2], wk * 1024 * per["write"][2]
        res["per_bits"][str(b)] = {"fetch_kib": fk, "write_kib": wk, "fetch_bytes": round(fb), "write_bytes": round(wb)}
        tot += fb + wb
    res["bytes_per_launch"] = round(tot / len(bits_list))
    return res


def trace_summary(folder):
    """Markdown tables of a rocprofv3 --kernel-trace --stats csv folder: the stats of every
    kernel called at least 5 times, then per kernel and launch shape the dispatch count,
    resources and durations (End - Start), including the mean of its last 20 dispatches."""
    import csv
    import glob

    def one(pattern):
        files = glob.glob(os.path.join(folder, "**", pattern), recursive=True)
        if len(files) != 1:
            raise SystemExit(f"expected one {pattern} under {folder}, found {len(files)}")
        return list(csv.DictReader(open(files[0])))

    def short(name):
        name = name.replace("samd::(anonymous namespace)::", "")
        return name[5:] if name.startswith("void ") else name

    out = ["| kernel | calls | avg us | min us | max us | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in one("*kernel_stats.csv"):
        if int(r["Calls"]) < 5:
            continue
        out.append(f"| {short(r['Name']).split('(')[0]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    def size(r, what):   # Workgroup_Size / Grid_Size, or the product of their _X, _Y, _Z columns
        if what in r:
            return r[what]
        return str(int(r[what + "_X"]) * int(r[what + "_Y"]) * int(r[what + "_Z"]))

    shapes = {}
    for r in one("*kernel_trace.csv"):
        key = (short(r["Kernel_Name"]).split("(")[0], size(r, "Workgroup_Size"), size(r, "Grid_Size"),
               r.get("VGPR_Count", ""), r.get("SGPR_Count", ""))
        shapes.setdefault(key, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    out += ["", "| kernel | workgroup | grid (threads) | VGPR | SGPR | dispatches | avg us | min us | avg of the last 20 us |",
            "|---|---|---|---|---|---|---|---|---|"]
    for (name, wg, grid, vg, sg), d in shapes.items():
        if len(d) < 5:
            continue
        out.append(f"| {name} | {wg} | {grid} | {vg} | {sg} | {len(d)} | {sum(d) / len(d) / 1e3:.2f} | "
                   f"{min(d) / 1e3:.2f} | {sum(d[-20:]) / len(d[-20:]) / 1e3:.2f} |")
    return "\n".join(out)


def stored_traffic():
    """The traffic summary committed under profiles/, or None when the kernel's sources have
    changed since the counters were taken."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    data = json.loads(text[start + 7:end])
    return data if data.get("source_sha256") == kernel_source_sha() else None


def capture_graph(fn, reps):
    """fn() called reps times, captured once into a HIP graph (replays skip the host)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(reps):
            fn()
    return graph


def timed_graph_stats(fn, reps, warm_s, samples=5):
    """(median, min) seconds per call of fn: HIP events on the launching stream around each
    of `samples` replays of a graph of reps calls (the GPU never waits for the host), after
    warm_s seconds of back-to-back replays (the clocks rise under sustained load)."""
    import torch
    graph = capture_graph(fn, reps)
    graph.replay()
    torch.cuda.synchronize()
    t_end = time.perf_counter() + warm_s
    while time.perf_counter() < t_end:
        graph.replay()
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(samples + 1)]
    ev[0].record(stream)
    for i in range(samples):
        graph.replay()
        ev[i + 1].record(stream)
    ev[-1].synchronize()
    per = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e-3 / reps for i in range(samples))
    return per[len(per) // 2], per[0]


def timed_graph(fn, reps, warm_s, samples=5):
    """Median seconds per call of fn (see timed_graph_stats)."""
    return timed_graph_stats(fn, reps, warm_s, samples)[0]


def host_cpu():
    """The host processor the CPU oracle ran on: model name and logical processors."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "logical_cpus": os.cpu_count()}


def int8_launch_name(plan):
    """A readable name of an int8 launch: kernel, output channels x positions per
    workgroup (weight-resident: the longest run of positions), waves per workgroup."""
    kind = {0: "im2col", 1: "halo", 2: "resident", 3: "packed-row"}[plan.halo]
    return f"{kind} {plan.mtile}x{plan.positions}" + (f" w{plan.waves}" if plan.halo == 2 else "")


def tune_int8(samd, shape, xf, wf, run, warm_s=0.05):
    """Set-up: time every launch the int8 baseline can make for the layer (run() makes one
    call) and install the fastest; returns (the chosen plan as a dict, {launch: us})."""
    times = {}
    best, best_t = None, None
    for plan in samd.conv2d_int8_candidates(shape, xf, wf):
        samd.conv2d_int8_use_plan(shape, xf, wf, plan)
        t = timed_graph(run, 10, warm_s, samples=3)
        times[int8_launch_name(plan)] = round(t * 1e6, 2)
        if best_t is None or t < best_t:
            best, best_t = plan, t
    samd.conv2d_int8_use_plan(shape, xf, wf, best)
    return ({"halo": best.halo, "mtile": best.mtile, "positions": best.positions,
             "row_segments": best.row_segments, "waves": best.waves}, times)


INT8_COUNTERS = ("SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_VALU_MFMA_BUSY_CYCLES "
                 "SQ_INSTS_VALU_MFMA_MOPS_I8 SQ_WAIT_INST_LDS SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE TA_TA_BUSY_sum "
                 "TD_TD_BUSY_sum",
                 "TCP_TCC_READ_REQ_sum TCP_TCC_WRITE_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCP_PENDING_STALL_CYCLES_sum "
                 "TCC_HIT_sum TCC_MISS_sum TCC_EA0_RDREQ_sum TCC_EA0_WRREQ_sum GRBM_GUI_ACTIVE SQ_INSTS_VMEM_RD "
                 "SQ_INSTS_VMEM_WR SQ_INSTS_LDS")


# Layers of the int8 counter runs: name -> (index into VGGB_LAYERS / ALEXNET_LAYERS, or
# None for the mid-size layer)
INT8_LAYERS = {"mid": None, "vggb1": ("VGGB_LAYERS", 0),
               **{f"alexnet{i + 1}": ("ALEXNET_LAYERS", i) for i in range(5)}}


def int8_layer(name):
    """The shape of an --int8-layer choice."""
    import samd_workloads as wl
    ref = INT8_LAYERS[name]
    return wl.MID if ref is None else getattr(wl, ref[0])[ref[1]]


def run_int8_counters(args):
    """One eager launch of every int8 baseline candidate on the chosen layer (4-bit
    unsigned activations, 4-bit signed weights), each after an untimed launch of the
    same candidate; prints the launch order."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl

    dev = torch.device("cuda:0")
    shape, b = int8_layer(args.int8_layer), 4
    if args.int8_layer == "mid":
        case = wl.conv2d_case(3, b)
        xv, wv = case.x, case.w
    else:
        rng = np.random.default_rng(wl.seed_for(6, b))
        xv = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), b, False)
        wv = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), b, True)
    xf, wf = samd.Fmt(b, False), samd.Fmt(b, True)
    x_nhwc = torch.from_numpy(np.ascontiguousarray(np.transpose(xv, (0, 2, 3, 1))).astype(np.uint8)).to(dev)
    w8 = torch.from_numpy(wv.astype(np.int8)).to(dev)
    ws8 = samd.conv2d_int8_prepare(w8, wf, shape, xf)
    Ho, Wo = samd.out_hw(shape)
    y = torch.empty((shape.N, shape.M, Ho, Wo), dtype=torch.int32, device=dev)
    for plan in samd.conv2d_int8_candidates(shape, xf, wf):
        samd.conv2d_int8_use_plan(shape, xf, wf, plan)
        for _ in range(2):
            samd.conv2d_int8_prepared(x_nhwc, xf, wf, shape, ws8, out=y)
        torch.cuda.synchronize()
        print(f"int8-counters: {int8_launch_name(plan)} launched twice",
              flush=True)
    samd.conv2d_int8_use_plan(shape, xf, wf, None)


def int8_summary(folders, layer="mid"):
    """Markdown table of rocprofv3 --pmc passes over --int8-counters: per int8 launch (the
    second of each candidate's two dispatches), its duration and counters."""
    import csv
    import glob

    import paper_1809_10572_amd as samd
    import samd_workloads as wl

    disp = {}
    for folder in folders:
        files = glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True)
        if len(files) != 1:
            raise SystemExit(f"expected one counter_collection.csv under {folder}, found {len(files)}")
        rows = list(csv.DictReader(open(files[0])))
        ids = sorted({int(r["Dispatch_Id"]) for r in rows if "conv2d_i8" in r["Kernel_Name"]})
        for k, d in enumerate(ids):
            e = disp.setdefault(k, {"c": {}, "dur": []})
            for r in rows:
                if int(r["Dispatch_Id"]) == d:
                    e["name"] = r["Kernel_Name"].replace("samd::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
                    e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                    e["dur"].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    shape = int8_layer(layer)
    cands = samd.conv2d_int8_candidates(shape, samd.Fmt(4, False), samd.Fmt(4, True))
    Ho, Wo = samd.out_hw(shape)
    macs = shape.N * shape.M * Ho * Wo * shape.C * shape.KH * shape.KW
    # Busy and issue cycles are not divided by GRBM_GUI_ACTIVE: under --pmc that counter
    # spans the profiler's per-dispatch overhead as well, so the table keeps raw counts
    # and the quantities that need no clock (requests, hit rates, latencies per request).
    out = ["| launch | kernel | dispatch us | MAC/s % of int8 peak | waves | wait % of wave cycles | "
           "LDS bank conflict cycles | LDS wait cycles | L1->L2 read requests | L2 hit % | L2->HBM read requests | "
           "L1->L2 read latency (cycles per request) | L1->L2 write requests | VMEM reads | LDS instructions |",
           "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for k in sorted(disp):
        if k % 2 == 0:
            continue   # the first launch of each candidate warms it
        e, c = disp[k], disp[k]["c"]
        plan = cands[k // 2]
        dur = min(e["dur"])

        def g(name):
            return c.get(name, float("nan"))
        hit, miss = g("TCC_HIT_sum"), g("TCC_MISS_sum")
        out.append(f"| {int8_launch_name(plan)} | {e['name']} | "
                   f"{dur * 1e6:.2f} | {100 * macs / dur / PEAK_I8_MACS:.1f} | {g('SQ_WAVES'):.0f} | "
                   f"{100 * g('SQ_WAIT_INST_ANY') / max(g('SQ_WAVE_CYCLES'), 1):.0f} | "
                   f"{g('SQ_LDS_BANK_CONFLICT'):.3g} | {g('SQ_WAIT_INST_LDS'):.3g} | "
                   f"{g('TCP_TCC_READ_REQ_sum'):.4g} | {100 * hit / max(hit + miss, 1):.1f} | "
                   f"{g('TCC_EA0_RDREQ_sum'):.4g} | "
                   f"{g('TCP_TCC_READ_REQ_LATENCY_sum') / max(g('TCP_TCC_READ_REQ_sum'), 1):.0f} | "
                   f"{g('TCP_TCC_WRITE_REQ_sum'):.4g} | {g('SQ_INSTS_VMEM_RD'):.4g} | {g('SQ_INSTS_LDS'):.4g} |")
    return "\n".join(out)


SPEC = {"mad": (PEAK_VALU_OPS, "T lane-ops/s", "alu"), "valu": (PEAK_VALU_OPS, "T lane-ops/s", "alu"),
        "mfma_i8": (PEAK_I8_MACS, "T MAC/s", "mfma"), "copy": (PEAK_HBM, "TB/s", "hbm"),
        "read": (PEAK_HBM, "TB/s", "hbm"), "write": (PEAK_HBM, "TB/s", "hbm"), "lds": (PEAK_LDS, "TB/s", "lds")}


def measure_peak(samd, kind, seconds=0.3, waves_per_simd=8):
    """Rate of one ceiling microbenchmark (include/samd_peaks.h) in work units per second:
    the median of 5 HIP-event-timed launches after `seconds` of back-to-back launches."""
    import torch
    code = {"mad": samd.PEAK_MAD_I64_I32, "valu": samd.PEAK_VALU_I32, "mfma_i8": samd.PEAK_MFMA_I8,
            "copy": samd.PEAK_COPY, "read": samd.PEAK_READ, "write": samd.PEAK_WRITE, "lds": samd.PEAK_LDS}[kind]
    dev = torch.device("cuda:0")
    nbytes = 1 << 30
    if kind in ("copy", "read", "write"):
        blocks, iters = 256 * 8 * 4, 1
        src = torch.empty(nbytes if kind != "write" else 16, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty(4 * blocks if kind == "read" else nbytes, dtype=torch.uint8, device=dev)
    else:
        # waves_per_simd workgroups of 4 waves per compute unit
        blocks, iters, src = 256 * waves_per_simd, (1 << 12) if kind in ("mfma_i8", "lds") else (1 << 14), None
        dst = torch.empty(4 * 256 * blocks, dtype=torch.uint8, device=dev)
    fn = lambda: samd.peak_launch(code, iters, blocks, dst, src, nbytes if src is not None else 0)
    fn()
    torch.cuda.synchronize()
    t_end = time.perf_counter() + seconds
    while time.perf_counter() < t_end:
        fn()
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    ev[0].record(stream)
    for i in range(5):
        fn()
        ev[i + 1].record(stream)
    ev[-1].synchronize()
    t = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e-3 for i in range(5))[2]
    work = samd.peak_work(code, iters, blocks, nbytes if src is not None else 0)
    return work / t


def device_info(torch):
    """GPU name, compute units, ROCm / HIP and torch versions of the run."""
    prop = torch.cuda.get_device_properties(0)
    info = {"name": prop.name, "gcn_arch": getattr(prop, "gcnArchName", None),
            "compute_units": prop.multi_processor_count, "hip": torch.version.hip, "torch": torch.__version__}
    try:
        info["rocm"] = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        info["rocm"] = None
    return info


def run_peaks(args):
    """The ceilings the roofline fractions divide by, measured on this GPU next to the
    published / unit-count figures.  Prints one JSON line."""
    import torch

    import paper_1809_10572_amd as samd

    rows = {}
    for kind in ("mad", "valu", "mfma_i8", "copy", "read", "write", "lds"):
        rate = measure_peak(samd, kind, seconds=0.5)
        spec, unit, bound = SPEC[kind]
        rows[kind] = {"measured": round(rate / 1e12, 3), "spec": round(spec / 1e12, 3), "unit": unit,
                      "frac_of_spec": round(rate / spec, 4)}
        print(f"peaks: {kind} {rate / 1e12:.3f} {unit} ({rate / spec:.3f} of {spec / 1e12:.2f})", file=sys.stderr,
              flush=True)
    # one wave per SIMD: what a kernel with a single wave per SIMD can issue
    for kind in ("mad", "mfma_i8"):
        rate = measure_peak(samd, kind, seconds=0.3, waves_per_simd=1)
        spec, unit, bound = SPEC[kind]
        rows[kind + "_1wave"] = {"measured": round(rate / 1e12, 3), "spec": round(spec / 1e12, 3), "unit": unit,
                                 "frac_of_spec": round(rate / spec, 4)}
        print(f"peaks: {kind} with one wave per SIMD {rate / 1e12:.3f} {unit} ({rate / spec:.3f} of {spec / 1e12:.2f})",
              file=sys.stderr, flush=True)
    print(json.dumps({"metric": "MI355X ceilings, measured", "n_gpus": 1, "device": device_info(torch),
                      "notes": {"mad": "v_mad_i64_i32 (exact signed 32x32->64 multiply-add), 8 independent chains "
                                       "per lane, uniform multiplier; spec = 256 CUs x 64 lanes x 2.4 GHz",
                                "valu": "v_add_u32, 8 independent chains per lane; same spec",
                                "mfma_i8": "v_mfma_i32_16x16x64_i8, 4 independent accumulators per wave; "
                                           "spec = 5.0 POP/s dense = 2.5 P MAC/s",
                                "copy": "16-byte loads and stores, 1 GiB each way, bytes read + written",
                                "read": "16-byte loads of 1 GiB",
                                "write": "16-byte stores of 1 GiB",
                                "lds": "ds_read_b128, conflict-free, 8 per trip; spec = 256 CUs x 256 B/clk x 2.4 GHz",
                                "*_1wave": "the same loop with one wave per SIMD (256 workgroups of 4 waves)"},
                      "peaks": rows}), flush=True)


def run_configs(args):
    """Workloads 1, 2 and 4 next to the default one: per (workload, b[, K]) GMAC/s, the
    roofline fraction of the bound that applies (VALU multiply-adds for conv2d, HBM bytes
    for conv1d), the int8 baseline where it applies, and a parity check against the
    oracle on the same inputs.  Prints one JSON line."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl
    from oracle import reference as ref

    dev = torch.device("cuda:0")
    out = {"single": [], "conv1d": [], "stress": []}

    def conv2d_row(cfg, b, shape, case):
        xf, wf = samd.Fmt(b, case.x_signed), samd.Fmt(b, case.w_signed)
        x = torch.from_numpy(case.x.astype(np.int8 if case.x_signed else np.uint8)).to(dev)
        x_nhwc = torch.from_numpy(np.ascontiguousarray(np.transpose(case.x, (0, 2, 3, 1))).astype(
            np.int8 if case.x_signed else np.uint8)).to(dev)
        w8 = torch.from_numpy(case.w.astype(np.int8)).to(dev)
        wp = samd.pack(w8, b, True)
        xp = samd.pack(x, b, case.x_signed)
        if not args.no_tune:
            samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=args.tune_candidates, reps=10)
        ws = samd.conv2d_prepare(wp, wf, shape, xf)
        ws8 = samd.conv2d_int8_prepare(w8, wf, shape, xf)
        Ho, Wo = samd.out_hw(shape)
        y = torch.empty((shape.N, shape.M, Ho, Wo), dtype=torch.int32, device=dev)
        y8 = torch.empty_like(y)
        if not args.no_tune_int8:
            tune_int8(samd, shape, xf, wf, lambda: samd.conv2d_int8_prepared(x_nhwc, xf, wf, shape, ws8, out=y8))
        t = timed_graph(lambda: samd.conv2d_prepared(xp, xf, wf, shape, ws, out=y), args.reps, args.kernel_warm_s)
        ta = timed_graph(lambda: samd.conv2d_accumulate(xf, wf, shape, ws, out=y), args.reps, args.kernel_warm_s)
        t8 = timed_graph(lambda: samd.conv2d_int8_prepared(x_nhwc, xf, wf, shape, ws8, out=y8), args.reps,
                         args.kernel_warm_s)
        samd.conv2d_prepared(xp, xf, wf, shape, ws, out=y)
        torch.cuda.synchronize()
        rng = np.random.default_rng(cfg * 100 + b)
        idx = np.stack([rng.integers(0, n, 512) for n in (shape.N, shape.M, Ho, Wo)], axis=1)
        want = ref.conv2d_points(case.x, case.w, shape.as_tuple(), idx)
        ok = bool(np.array_equal(y.cpu().numpy()[tuple(idx.T)], want) and
                  np.array_equal(y8.cpu().numpy()[tuple(idx.T)], want))
        p = samd.conv2d_plan(shape, xf, wf)
        macs = shape.N * shape.M * Ho * Wo * shape.C * shape.KH * shape.KW
        mads = shape.N * shape.M * Ho * p.words_per_row * shape.C * shape.KH * p.tap_words
        return {"bits": b, "us": round(t * 1e6, 2), "accumulate_us": round(ta * 1e6, 2),
                "gmacs": round(macs / t / 1e9, 1), "valu_frac": round(mads / ta / PEAK_VALU_OPS, 4),
                "int8_us": round(t8 * 1e6, 2), "speedup_vs_int8": round(t8 / t, 3),
                "lane_bits": p.lane_bits, "lanes": p.lanes, "flush_channels": p.flush_channels, "parity": ok}

    for b in (4,):
        out["single"].append(conv2d_row(1, b, wl.SINGLE, wl.conv2d_case(1, b)))
    out["conv1d"] = conv1d_rows(args)
    for b in wl.BITS_SWEEP[4]:
        out["stress"].append(conv2d_row(4, b, wl.STRESS, wl.conv2d_case(4, b)))
    print(json.dumps({"metric": "SAMD workloads 1, 2 and 4: GMAC/s and roofline fractions", "n_gpus": 1,
                      "data": "synthetic", "dtype": "int64",
                      "config": {"single": "1x16x16x16 -> 16, 3x3, u4 x s4",
                                 "conv1d": "2^20 unsigned b-bit values, 3 and 5 unsigned taps, valid mode",
                                 "stress": "4x256x28x28 -> 256, 3x3, signed x signed, half the values at the range ends",
                                 "timing": "stage + accumulate (kernel words prepared once); conv1d whole call",
                                 "plans": "model" if args.no_tune else "tuned at set-up"},
                      **out}), flush=True)


def conv1d_rows(args):
    """Workload 2 (2^20 unsigned b-bit values, 3 and 5 unsigned taps, valid mode) per
    (b, K): the whole call's time, its algorithmic bytes (packed input + 4 B per output)
    as a fraction of HBM peak, two floors timed the same way (a kernel that only stores
    the output's bytes, and one that copies a buffer of that size: a load, then a store)
    and a full-output parity check against the oracle."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl
    from oracle import reference as ref

    dev = torch.device("cuda:0")
    rows, floors = [], {}
    for b in range(1, 9):
        for K in (3, 5):
            case = wl.conv1d_case(b, K)
            n = case.x.size
            xp = samd.pack(torch.from_numpy(case.x.astype(np.uint8)).to(dev).view(1, n), b, False).view(-1)
            y = samd.conv1d(xp, n, b, case.k.tolist(), b)
            t = timed_graph(lambda: samd.conv1d(xp, n, b, case.k.tolist(), b, out=y), args.reps, args.kernel_warm_s)
            torch.cuda.synchronize()
            ok = bool(np.array_equal(y.cpu().numpy(), ref.conv1d(case.x, case.k)))
            out_bytes = (n - K + 1) * 4
            if out_bytes not in floors:
                # the output's bytes stored by the plain grid-stride store kernel (16 B per
                # lane), and copied from a buffer of the same size (read + write)
                n16 = out_bytes // 16
                src = torch.ones(n16 * 16, dtype=torch.uint8, device=dev)
                dst = torch.empty(n16 * 16, dtype=torch.uint8, device=dev)
                blocks = (n16 + 255) // 256
                floors[out_bytes] = (
                    timed_graph(lambda: samd.peak_launch(samd.PEAK_WRITE, 1, blocks, dst, None, n16 * 16),
                                args.reps, args.kernel_warm_s),
                    timed_graph(lambda: samd.peak_launch(samd.PEAK_COPY, 1, blocks, dst, src, n16 * 16),
                                args.reps, args.kernel_warm_s))
            nbytes = samd.row_words(n, b) * 4 + out_bytes
            p = samd.conv1d_plan(n, b, case.k.tolist(), b)
            rows.append({"bits": b, "taps": K, "us": round(t * 1e6, 2),
                         "gmacs": round((n - K + 1) * K / t / 1e9, 1),
                         "gbps": round(nbytes / t / 1e9, 1), "hbm_frac": round(nbytes / t / PEAK_HBM, 4),
                         "store_floor_us": round(floors[out_bytes][0] * 1e6, 2),
                         "copy_floor_us": round(floors[out_bytes][1] * 1e6, 2),
                         "vs_store_floor": round(t / floors[out_bytes][0], 3),
                         "vs_copy_floor": round(t / floors[out_bytes][1], 3),
                         "lane_bits": p.lane_bits, "lanes": p.lanes, "groups": p.groups, "extra": p.extra,
                         "parity": ok})
            print(f"conv1d: b={b} K={K} {t * 1e6:.2f} us (store floor {floors[out_bytes][0] * 1e6:.2f} us, "
                  f"copy floor {floors[out_bytes][1] * 1e6:.2f} us) parity {ok}", file=sys.stderr, flush=True)
    return rows


def run_conv1d(args):
    """Workload 2 alone (see conv1d_rows).  Prints one JSON line."""
    import torch
    print(json.dumps({"metric": "SAMD conv1d: time per call, HBM fraction and store-only floor", "n_gpus": 1,
                      "device": device_info(torch), "data": "synthetic", "dtype": "int64",
                      "config": {"conv1d": "2^20 unsigned b-bit values, 3 and 5 unsigned taps, valid mode",
                                 "timing": "whole call (one kernel), median of graph-replay samples",
                                 "floors": "grid-stride store (and copy) kernels over the output's bytes, 16 B per "
                                           "lane"},
                      "conv1d": conv1d_rows(args)}), flush=True)


def run_spacers(args):
    """Temporary against permanent spacer bits (Sec. 2.2, Sec. 6.1, the two result sets of
    Sec. 7): per workload and bit width, the convolution from packed activations (the
    spread pass that inserts the spacer bits, then the multiply) and from activations
    stored in the permanent-spacer layout (the multiply alone, whose decode also leaves
    out the fix-up's xor), with the bytes each stores and moves, both checked against the
    oracle.  Prints one JSON line."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl
    from oracle import reference as ref

    dev = torch.device("cuda:0")
    out = {}
    for name, cfg, shape, bits_list in (("single", 1, wl.SINGLE, range(1, 9)), ("mid", 3, wl.MID, range(1, 9)),
                                        ("stress", 4, wl.STRESS, wl.BITS_SWEEP[4])):
        rows = []
        Ho, Wo = samd.out_hw(shape)
        macs = shape.N * shape.M * Ho * Wo * shape.C * shape.KH * shape.KW
        for b in bits_list:
            case = wl.conv2d_case(cfg, b, shape)
            xf, wf = samd.Fmt(b, case.x_signed), samd.Fmt(b, case.w_signed)
            x = torch.from_numpy(case.x.astype(np.int8 if case.x_signed else np.uint8)).to(dev)
            wp = samd.pack(torch.from_numpy(case.w.astype(np.int8)).to(dev), b, case.w_signed)
            xp = samd.pack(x, b, case.x_signed)
            if not args.no_tune:
                samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=args.tune_candidates, reps=10)
                samd.conv2d_spaced_tune(xp, xf, wp, wf, shape, candidates=args.tune_candidates, reps=10)
            ws = samd.conv2d_prepare(wp, wf, shape, xf)
            ws_s = samd.conv2d_spaced_prepare(wp, wf, shape, xf)
            spaced = samd.conv2d_spaced_pack(x, xf, wf, shape)
            y = torch.empty((shape.N, shape.M, Ho, Wo), dtype=torch.int32, device=dev)
            y_s = torch.empty_like(y)
            t_temp, t_temp_min = timed_graph_stats(lambda: samd.conv2d_prepared(xp, xf, wf, shape, ws, out=y),
                                                   args.reps, args.kernel_warm_s, args.samples)
            t_perm, t_perm_min = timed_graph_stats(lambda: samd.conv2d_spaced(spaced, xf, wf, shape, ws_s, out=y_s),
                                                   args.reps, args.kernel_warm_s, args.samples)
            t_spread, _ = timed_graph_stats(lambda: samd.conv2d_stage(xp, xf, wf, shape, ws), args.reps,
                                            args.kernel_warm_s, args.samples)
            samd.conv2d_prepared(xp, xf, wf, shape, ws, out=y)
            samd.conv2d_spaced(spaced, xf, wf, shape, ws_s, out=y_s)
            torch.cuda.synchronize()
            rng = np.random.default_rng(cfg * 100 + b)
            idx = np.stack([rng.integers(0, n, 512) for n in (shape.N, shape.M, Ho, Wo)], axis=1)
            want = ref.conv2d_points(case.x, case.w, shape.as_tuple(), idx)
            ok_t = bool(np.array_equal(y.cpu().numpy()[tuple(idx.T)], want))
            ok_p = bool(np.array_equal(y_s.cpu().numpy()[tuple(idx.T)], want))
            pt, pp = samd.conv2d_plan(shape, xf, wf), samd.conv2d_spaced_plan(shape, xf, wf)
            lay = samd.conv2d_spaced_layout(shape, xf, wf)
            packed_bytes = shape.N * shape.C * shape.H * samd.row_words(shape.W, b) * 4
            words_t = shape.N * shape.C * (shape.H + 2 * shape.pad_h) * pt.tap_words * pt.words_per_row * 4
            spaced_bytes = (lay.words - lay.padded_rows * lay.tap_words * lay.words_per_row) * 4
            kw_t = shape.M * shape.C * shape.KH * pt.tap_words * 4
            kw_p = shape.M * shape.C * shape.KH * pp.tap_words * 4
            y_bytes = shape.N * shape.M * Ho * Wo * 4
            rows.append({
                "bits": b,
                "temporary_us": round(t_temp * 1e6, 2), "temporary_us_min": round(t_temp_min * 1e6, 2),
                "spread_us": round(t_spread * 1e6, 2),
                "permanent_us": round(t_perm * 1e6, 2), "permanent_us_min": round(t_perm_min * 1e6, 2),
                "temporary_gmacs": round(macs / t_temp / 1e9, 1), "permanent_gmacs": round(macs / t_perm / 1e9, 1),
                "permanent_speedup": round(t_temp / t_perm, 3),
                # bytes the activations occupy, and the bytes one call moves at best
                "stored_bytes_temporary": packed_bytes, "stored_bytes_permanent": spaced_bytes,
                "moved_bytes_temporary": packed_bytes + 2 * words_t + kw_t + y_bytes,
                "moved_bytes_permanent": spaced_bytes + kw_p + y_bytes,
                "lanes_temporary": f"L={pt.lane_bits} I={pt.lanes} G={pt.flush_channels}",
                "lanes_permanent": f"L={pp.lane_bits} I={pp.lanes} G={pp.flush_channels} msb_spacer={pp.spacer_msb}",
                "parity_temporary": ok_t, "parity_permanent": ok_p})
            print(f"spacers: {name} b={b} temporary {t_temp * 1e6:.2f} us permanent {t_perm * 1e6:.2f} us "
                  f"parity {ok_t} {ok_p}", file=sys.stderr, flush=True)
        out[name] = rows
    print(json.dumps({"metric": "temporary vs permanent spacer bits: conv2d time and bytes per bit width",
                      "unit": "us", "n_gpus": 1, "data": "synthetic", "dtype": "int64",
                      "config": {"single": "1x16x16x16 -> 16, 3x3, u_b x s_b",
                                 "mid": "8x128x56x56 -> 128, 3x3, u_b x s_b",
                                 "stress": "4x256x28x28 -> 256, 3x3, s_b x s_b, half the values at the range ends",
                                 "temporary": "conv2d_prepared: spread of the packed activations + multiply",
                                 "permanent": "conv2d_spaced: multiply from the permanent-spacer layout",
                                 "plans": "model" if args.no_tune else "each layout's plan tuned at set-up"},
                      **out}), flush=True)


def run_vggb(args):
    """The paper's own experiment (Sec. 7): every VGG-B convolution layer at batch 1 with
    N-bit signed activations and weights, N = 8 down to 2, next to the native-int8
    baseline on the same layer.  Prints one JSON line."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl
    from oracle import reference as ref

    dev = torch.device("cuda:0")
    bits_list = [int(b) for b in args.bits.split(",")] if args.bits_given else wl.BITS_SWEEP[6]
    rows, tot_macs, tot_s, tot_int8_s, tot_perm_s = [], 0, 0.0, 0.0, 0.0
    for li, shape in enumerate(wl.VGGB_LAYERS):
        Ho, Wo = samd.out_hw(shape)
        macs = shape.N * shape.M * Ho * Wo * shape.C * shape.KH * shape.KW
        for b in bits_list:
            case = wl.vggb_case(li, b)
            f = samd.Fmt(b, True)
            x = torch.from_numpy(case.x.astype(np.int8)).to(dev)
            x_nhwc = torch.from_numpy(np.ascontiguousarray(np.transpose(case.x, (0, 2, 3, 1))).astype(np.int8)).to(dev)
            w8 = torch.from_numpy(case.w.astype(np.int8)).to(dev)
            wp = samd.pack(w8, b, True)
            xp = samd.pack(x, b, True)
            if not args.no_tune:
                # set-up: the layer's plan chosen by timing the model's top candidates
                samd.conv2d_tune(xp, f, wp, f, shape, candidates=args.tune_candidates, reps=10)
            ws = samd.conv2d_prepare(wp, f, shape, f)
            ws8 = samd.conv2d_int8_prepare(w8, f, shape, f)
            y = torch.empty((shape.N, shape.M, Ho, Wo), dtype=torch.int32, device=dev)
            y8 = torch.empty_like(y)
            if not args.no_tune_int8:
                tune_int8(samd, shape, f, f, lambda: samd.conv2d_int8_prepared(x_nhwc, f, f, shape, ws8, out=y8))
            t_pack = timed_graph(lambda: samd.pack(x, b, True, out=xp), args.reps, args.kernel_warm_s)
            t_samd = timed_graph(lambda: samd.conv2d_prepared(xp, f, f, shape, ws, out=y), args.reps,
                                 args.kernel_warm_s)
            t_int8 = timed_graph(lambda: samd.conv2d_int8_prepared(x_nhwc, f, f, shape, ws8, out=y8), args.reps,
                                 args.kernel_warm_s)
            # permanent spacer bits: the activations stored in the layer's spaced layout
            if not args.no_tune:
                samd.conv2d_spaced_tune(xp, f, wp, f, shape, candidates=args.tune_candidates, reps=10)
            ws_s = samd.conv2d_spaced_prepare(wp, f, shape, f)
            spaced = samd.conv2d_spaced_pack(x, f, f, shape)
            y_s = torch.empty_like(y)
            t_perm = timed_graph(lambda: samd.conv2d_spaced(spaced, f, f, shape, ws_s, out=y_s), args.reps,
                                 args.kernel_warm_s)
            samd.conv2d_spaced(spaced, f, f, shape, ws_s, out=y_s)
            torch.cuda.synchronize()
            rng = np.random.default_rng(li * 10 + b)
            idx = np.stack([rng.integers(0, n, 256) for n in (shape.N, shape.M, Ho, Wo)], axis=1)
            want = ref.conv2d_points(case.x, case.w, shape.as_tuple(), idx)
            ok = bool(np.array_equal(y.cpu().numpy()[tuple(idx.T)], want) and
                      np.array_equal(y8.cpu().numpy()[tuple(idx.T)], want) and
                      np.array_equal(y_s.cpu().numpy()[tuple(idx.T)], want))
            p = samd.conv2d_plan(shape, f, f)
            rows.append({"layer": li + 1, "C": shape.C, "M": shape.M, "HW": shape.H, "bits": b,
                         "samd_us": round(t_samd * 1e6, 2), "pack_us": round(t_pack * 1e6, 2),
                         "permanent_us": round(t_perm * 1e6, 2),
                         "permanent_speedup_vs_int8": round(t_int8 / t_perm, 3),
                         "int8_us": round(t_int8 * 1e6, 2), "samd_gmacs": round(macs / t_samd / 1e9, 1),
                         "int8_gmacs": round(macs / t_int8 / 1e9, 1), "speedup_vs_int8": round(t_int8 / t_samd, 3),
                         "lane_bits": p.lane_bits, "lanes": p.lanes, "tap_words": p.tap_words,
                         "flush_channels": p.flush_channels, "tile": f"{p.rows_per_block}x{p.mblock}",
                         "rows_per_thread": p.rows_per_thread, "shared_rows": bool(p.shared_rows),
                         "split_waves": p.split_waves, "parity": ok})
            tot_macs += macs
            tot_s += t_samd
            tot_int8_s += t_int8
            tot_perm_s += t_perm
            print(f"vggb: layer {li + 1} b={b} samd {t_samd * 1e6:.1f} us permanent {t_perm * 1e6:.1f} us "
                  f"int8 {t_int8 * 1e6:.1f} us parity {ok}", file=sys.stderr, flush=True)
    line = {"metric": "VGG-B conv layers, N-bit signed activations and weights (N = 8..2), GMAC/s",
            "value": round(tot_macs / tot_s / 1e9, 1), "unit": "GMAC/s", "n_gpus": 1,
            "higher_is_better": True, "dtype": "int64", "data": "synthetic",
            "config": {"workload": "VGG-B's ten 3x3 convolution layers, batch 1, each layer on its own; "
                                   "one call = stage + accumulate with prepared kernel words (temporary spacer bits) "
                                   "or the multiply from the permanent-spacer layout (permanent spacer bits)",
                       "bits": bits_list,
                       "plans": "model" if args.no_tune else f"tuned at set-up ({args.tune_candidates} candidates timed)"},
            "int8_gmacs": round(tot_macs / tot_int8_s / 1e9, 1),
            "permanent_gmacs": round(tot_macs / tot_perm_s / 1e9, 1),
            "per_layer": rows}
    print(json.dumps(line), flush=True)


def run_stack(args):
    """The AlexNet-shaped stack (five conv layers, ReLU + requantisation between them,
    batch 16): one forward pass per step, kernel words prepared once.  Three chains:
    SAMD with packed activations between layers (max, relu_requant_pack, pack-format
    stage), SAMD with the epilogue writing the next layer's operand words directly
    (max, relu_requant_stage), and the int8 baseline (max, NHWC uint8 requantisation).
    Prints one JSON line."""
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl

    dev = torch.device("cuda:0")
    bits_list = [int(b) for b in args.bits.split(",")] if args.bits_given else wl.BITS_SWEEP[5]
    rows = []
    for bits in bits_list:
        case = wl.stack_case(bits)
        xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
        lys = case.layers
        macs = 0
        for l in lys:
            Ho, Wo = samd.out_hw(l)
            macs += l.N * l.M * Ho * Wo * l.C * l.KH * l.KW
        wps = [samd.pack(torch.from_numpy(w.astype(np.int8)).to(dev), bits, True) for w in case.ws]
        wss = [samd.conv2d_prepare(wp, wf, l, xf) for wp, l in zip(wps, lys)]
        ws8 = [samd.conv2d_int8_prepare(torch.from_numpy(w.astype(np.int8)).to(dev), wf, l, xf)
               for w, l in zip(case.ws, lys)]
        x8 = torch.from_numpy(case.x.astype(np.uint8)).to(dev)
        xn = torch.from_numpy(np.ascontiguousarray(np.transpose(case.x, (0, 2, 3, 1))).astype(np.uint8)).to(dev)
        ys = [torch.empty((l.N, l.M) + samd.out_hw(l), dtype=torch.int32, device=dev) for l in lys]
        mx = torch.empty(1, dtype=torch.int32, device=dev)
        xps = [torch.empty((l.N, l.C, l.H, samd.row_words(l.W, bits)), dtype=torch.int32, device=dev) for l in lys]
        x8s = [xn] + [torch.empty((l.N, l.H, l.W, l.C), dtype=torch.uint8, device=dev) for l in lys[1:]]

        def chain_packed():
            samd.pack(x8, bits, False, out=xps[0])
            for li, l in enumerate(lys):
                samd.conv2d_prepared(xps[li], xf, wf, l, wss[li], out=ys[li])
                if li + 1 < len(lys):
                    samd.max_i32(ys[li], out=mx)
                    samd.relu_requant_pack(ys[li], mx, bits, out=xps[li + 1])

        def chain_fused():
            samd.pack(x8, bits, False, out=xps[0])
            samd.conv2d_stage(xps[0], xf, wf, lys[0], wss[0])
            for li, l in enumerate(lys):
                samd.conv2d_accumulate(xf, wf, l, wss[li], out=ys[li])
                if li + 1 < len(lys):
                    samd.max_i32(ys[li], out=mx)
                    samd.relu_requant_stage(ys[li], mx, bits, wf, lys[li + 1], wss[li + 1])

        if not args.no_tune:
            # set-up: each layer's plan tuned on its own input (one pass of the packed chain
            # gives every layer's activations), then the kernel words prepared again
            chain_packed()
            for li, l in enumerate(lys):
                samd.conv2d_tune(xps[li], xf, wps[li], wf, l, candidates=args.tune_candidates, reps=3)
                wss[li] = samd.conv2d_prepare(wps[li], wf, l, xf)
            torch.cuda.synchronize()

        if not args.no_tune_int8:
            chain_packed()   # activations of every layer for the int8 chain's inputs
            for li, l in enumerate(lys):
                if li > 0:
                    samd.max_i32(ys[li - 1], out=mx)
                    samd.relu_requant_nhwc_u8(ys[li - 1], mx, bits, out=x8s[li])
                tune_int8(samd, l, xf, wf, lambda: samd.conv2d_int8_prepared(x8s[li], xf, wf, l, ws8[li], out=ys[li]))
            torch.cuda.synchronize()

        def chain_int8():
            for li, l in enumerate(lys):
                samd.conv2d_int8_prepared(x8s[li], xf, wf, l, ws8[li], out=ys[li])
                if li + 1 < len(lys):
                    samd.max_i32(ys[li], out=mx)
                    samd.relu_requant_nhwc_u8(ys[li], mx, bits, out=x8s[li + 1])

        t = {name: timed_graph(fn, 3, args.kernel_warm_s) for name, fn in
             (("samd_packed", chain_packed), ("samd_fused", chain_fused), ("int8", chain_int8))}

        # per layer: each chain's convolution and the epilogue that follows it
        layer_rows = []
        for li, l in enumerate(lys):
            Ho, Wo = samd.out_hw(l)
            lmacs = l.N * l.M * Ho * Wo * l.C * l.KH * l.KW
            r = {"layer": li + 1, "gmac": round(lmacs / 1e9, 2),
                 "samd_conv_ms": timed_graph(lambda: samd.conv2d_prepared(xps[li], xf, wf, l, wss[li], out=ys[li]),
                                             3, args.kernel_warm_s) * 1e3,
                 "samd_accumulate_ms": timed_graph(lambda: samd.conv2d_accumulate(xf, wf, l, wss[li], out=ys[li]),
                                                   3, args.kernel_warm_s) * 1e3,
                 "int8_conv_ms": timed_graph(lambda: samd.conv2d_int8_prepared(x8s[li], xf, wf, l, ws8[li],
                                                                               out=ys[li]), 3, args.kernel_warm_s) * 1e3}
            if li + 1 < len(lys):
                nxt = lys[li + 1]
                r["epilogue_packed_ms"] = timed_graph(lambda: (samd.max_i32(ys[li], out=mx),
                                                               samd.relu_requant_pack(ys[li], mx, bits,
                                                                                      out=xps[li + 1])),
                                                      3, args.kernel_warm_s) * 1e3
                r["epilogue_fused_ms"] = timed_graph(lambda: (samd.max_i32(ys[li], out=mx),
                                                              samd.relu_requant_stage(ys[li], mx, bits, wf, nxt,
                                                                                      wss[li + 1])),
                                                     3, args.kernel_warm_s) * 1e3
                r["epilogue_int8_ms"] = timed_graph(lambda: (samd.max_i32(ys[li], out=mx),
                                                             samd.relu_requant_nhwc_u8(ys[li], mx, bits,
                                                                                       out=x8s[li + 1])),
                                                    3, args.kernel_warm_s) * 1e3
            r["samd_conv_gmacs"] = round(lmacs / r["samd_conv_ms"] / 1e6, 1)
            r["int8_conv_gmacs"] = round(lmacs / r["int8_conv_ms"] / 1e6, 1)
            layer_rows.append({k: (round(v, 4) if isinstance(v, float) and k.endswith("_ms") else v)
                               for k, v in r.items()})

        # parity: every layer's int32 output of each chain, at full batch, against the oracle
        parity = None
        if not args.no_check:
            from oracle import reference as ref
            accs, _, _ = ref.stack(case.x, case.ws, [l.as_tuple() for l in lys], bits)
            parity = {}
            for name, fn in (("samd_packed", chain_packed), ("samd_fused", chain_fused), ("int8", chain_int8)):
                fn()
                torch.cuda.synchronize()
                parity[name] = all(np.array_equal(ys[li].cpu().numpy(), accs[li]) for li in range(len(lys)))
            print(f"stack: b={bits} parity {parity}", file=sys.stderr, flush=True)

        rows.append({"bits": bits, **{f"{k}_ms": round(v * 1e3, 3) for k, v in t.items()},
                     **{f"{k}_gmacs": round(macs / v / 1e9, 1) for k, v in t.items()},
                     "fused_saving": round(1 - t["samd_fused"] / t["samd_packed"], 3),
                     "parity": parity, "per_layer": layer_rows})
        print(f"stack: b={bits} " + " ".join(f"{k} {v * 1e3:.3f} ms" for k, v in t.items()), file=sys.stderr,
              flush=True)
    print(json.dumps({"metric": "AlexNet-shaped conv stack forward, GMAC/s", "unit": "GMAC/s",
                      "value": round(sum(r["samd_fused_gmacs"] for r in rows) / len(rows), 1), "n_gpus": 1,
                      "data": "synthetic",
                      "config": {"workload": "five conv layers (11x11/4 96, 5x5 256, 3x3 384, 3x3 384, 3x3 256) on "
                                             "16x3x224x224, no pooling, ReLU + requantisation between layers",
                                 "bits": bits_list, "macs": macs,
                                 "plans": "model" if args.no_tune else
                                 f"tuned per layer at set-up ({args.tune_candidates} candidates timed)"},
                      "per_bits": rows}), flush=True)


def run_lanewise(args):
    """Lane-wise SAMD arithmetic on packed words (add, subtract, multiply, vector scale):
    HBM-bound elementwise kernels over 64 Mi words per operand.  Prints one JSON line of
    achieved GB/s per (operation, bit width) against the 8 TB/s HBM peak."""
    import torch

    import paper_1809_10572_amd as samd

    nwords = 64 << 20
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(1809105720)
    a = torch.randint(-(1 << 31), (1 << 31) - 1, (nwords,), dtype=torch.int32, device=dev, generator=gen)
    b = torch.randint(-(1 << 31), (1 << 31) - 1, (nwords,), dtype=torch.int32, device=dev, generator=gen)
    out = torch.empty_like(a)
    rows = []
    bits_list = [int(v) for v in args.bits.split(",")]
    for bits in bits_list:
        # clear the bits above each word's last lane (the packed format keeps them zero)
        P = 32 // bits
        valid = (1 << (P * bits)) - 1 if P * bits < 32 else -1
        av, bv = a & valid if valid != -1 else a, b & valid if valid != -1 else b
        for name, fn, nbytes in (("add", lambda: samd.lanewise(samd.LANE_ADD, av, bv, bits, False, out=out), 12),
                                 ("sub", lambda: samd.lanewise(samd.LANE_SUB, av, bv, bits, False, out=out), 12),
                                 ("mul", lambda: samd.lanewise(samd.LANE_MUL, av, bv, bits, False, out=out), 12),
                                 ("scale", lambda: samd.scale(av, 5, bits, False, out=out), 8)):
            t = timed_graph(fn, 5, args.kernel_warm_s)
            gbs = nwords * nbytes / t / 1e9
            rows.append({"op": name, "bits": bits, "us": round(t * 1e6, 1), "GB_s": round(gbs, 1),
                         "hbm_frac": round(gbs * 1e9 / PEAK_HBM, 3),
                         "G_lanes_s": round(nwords * P / t / 1e9, 1)})
    print(json.dumps({"metric": "lane-wise SAMD arithmetic on packed words, GB/s", "unit": "GB/s",
                      "value": round(sum(r["GB_s"] for r in rows) / len(rows), 1), "n_gpus": 1,
                      "config": {"workload": f"{nwords} packed uint32 words per operand (inputs 2x256 MiB)",
                                 "bits": bits_list},
                      "per_op": rows}), flush=True)


def main():
    args = parse()
    args.bits_given = "--bits" in sys.argv
    if args.peaks:
        run_peaks(args)
        return
    if args.int8_counters:
        run_int8_counters(args)
        return
    if args.int8_summary:
        print(int8_summary(args.int8_summary, args.int8_layer))
        return
    if args.vggb:
        run_vggb(args)
        return
    if args.configs:
        run_configs(args)
        return
    if args.conv1d:
        run_conv1d(args)
        return
    if args.lanewise:
        run_lanewise(args)
        return
    if args.spacers:
        run_spacers(args)
        return
    if args.stack:
        run_stack(args)
        return
    if args.trace_summary:
        print(trace_summary(args.trace_summary))
        return
    if args.valu_summary:
        print(valu_summary(args.valu_summary, [int(b) for b in args.bits.split(",")], args.plans_in))
        return
    if args.traffic_summary:
        print(json.dumps(traffic_summary(*args.traffic_summary, [int(b) for b in args.bits.split(",")]), indent=1))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the SAMD library runs on a single MI355X and has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1809_10572_amd as samd
    import samd_workloads as wl

    bits_list = [int(b) for b in args.bits.split(",")]
    dev = torch.device("cuda:0")
    shape = wl.MID
    N, C, H, W, M, KH, KW = shape.N, shape.C, shape.H, shape.W, shape.M, shape.KH, shape.KW
    Ho, Wo = samd.out_hw(shape)
    macs = N * M * Ho * Wo * C * KH * KW
    samd_hp = H + 2 * shape.pad_h

    layers = []
    for b in bits_list:
        case = wl.conv2d_case(3, b)
        xf, wf = samd.Fmt(b, case.x_signed), samd.Fmt(b, case.w_signed)
        x = torch.from_numpy(case.x.astype(np.uint8)).to(dev)
        x_nhwc = torch.from_numpy(np.ascontiguousarray(np.transpose(case.x, (0, 2, 3, 1))).astype(np.uint8)).to(dev)
        w8 = torch.from_numpy(case.w.astype(np.int8)).to(dev)
        wp = samd.pack(w8, b, True)
        xp = torch.empty((N, C, H, samd.row_words(W, b)), dtype=torch.int32, device=dev)
        ws = torch.empty(max(samd.conv2d_workspace(shape, xf, wf), 256), dtype=torch.uint8, device=dev)
        ws8 = samd.conv2d_int8_prepare(w8, wf, shape, xf)
        plan = samd.conv2d_plan(shape, xf, wf)
        layers.append(dict(b=b, case=case, xf=xf, wf=wf, x=x, x_nhwc=x_nhwc, wp=wp, xp=xp, ws=ws, ws8=ws8, plan=plan,
                           y=torch.empty((N, M, Ho, Wo), dtype=torch.int32, device=dev),
                           y8=torch.empty((N, M, Ho, Wo), dtype=torch.int32, device=dev)))
    torch.cuda.synchronize()

    # set-up: each bit width's plan chosen by timing the planner's top candidates on the
    # layer's own inputs (outside every timed region); the workspace is then sized again
    plans_in = json.load(open(args.plans_in)) if args.plans_in else None
    if plans_in or not args.no_tune:
        for L in layers:
            if plans_in:
                samd.conv2d_use_plan(shape, L["xf"], L["wf"], plans_in[str(L["b"])])
            else:
                samd.pack(L["x"], L["b"], False, out=L["xp"])
                samd.conv2d_tune(L["xp"], L["xf"], L["wp"], L["wf"], shape, candidates=args.tune_candidates, reps=10)
            L["ws"] = torch.empty(max(samd.conv2d_workspace(shape, L["xf"], L["wf"]), 256), dtype=torch.uint8,
                                  device=dev)
            L["plan"] = samd.conv2d_plan(shape, L["xf"], L["wf"])
        torch.cuda.synchronize()
    if args.plans_out:
        with open(args.plans_out, "w") as fh:
            json.dump({str(L["b"]): samd.plan_key(L["plan"]) for L in layers}, fh, indent=1)

    # the layer's kernel words are prepared once per layer (weights are constant)
    for L in layers:
        samd.conv2d_prepare(L["wp"], L["wf"], shape, L["xf"], ws=L["ws"])
    # the int8 baseline's launch, chosen by timing its candidates on the same layer
    for L in layers:
        if args.no_tune_int8:
            p8 = samd.conv2d_int8_plan(shape, L["xf"], L["wf"])
            L["int8_plan"], L["int8_cands"] = {"halo": p8.halo, "mtile": p8.mtile, "positions": p8.positions,
                                               "row_segments": p8.row_segments, "waves": p8.waves}, None
        else:
            L["int8_plan"], L["int8_cands"] = tune_int8(
                samd, shape, L["xf"], L["wf"],
                lambda: samd.conv2d_int8_prepared(L["x_nhwc"], L["xf"], L["wf"], shape, L["ws8"], out=L["y8"]))
    torch.cuda.synchronize()

    if args.counters:
        # one eager launch of each kernel per bit width, in step order, then the calibration
        # copy (twice; the second is the one read)
        for L in layers:
            samd.pack(L["x"], L["b"], False, out=L["xp"])
            samd.conv2d_stage(L["xp"], L["xf"], L["wf"], shape, L["ws"])
            samd.conv2d_accumulate(L["xf"], L["wf"], shape, L["ws"], out=L["y"])
            samd.conv2d_int8_prepared(L["x_nhwc"], L["xf"], L["wf"], shape, L["ws8"], out=L["y8"])
            torch.cuda.synchronize()
            print(f"counters: b={L['b']} launched", flush=True)
        src = torch.empty(COPY_BYTES // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        print(f"counters: copy of {COPY_BYTES} bytes done; kernel sources {kernel_source_sha()}", flush=True)
        return

    # The bit widths are independent layers (own inputs, workspaces and outputs): with
    # --streams S > 1 they run round-robin on S side streams that fork from and join the
    # launching stream, so one width's pack and stage and the ramp and drain of its
    # accumulate overlap another's.  Every kernel still runs once per step.
    side = [torch.cuda.Stream() for _ in range(args.streams)] if args.streams > 1 else []
    # layer i's stream: in order of bit width, 0, 1, .., S-1, then S-1, .., 0 (snake) or
    # 0, 1, .., S-1 again (round-robin)
    S = max(1, args.streams)
    by_bits = sorted(range(len(layers)), key=lambda i: layers[i]["b"])
    stream_of = [0] * len(layers)
    for r, i in enumerate(by_bits):
        k, lap = r % S, r // S
        stream_of[i] = (S - 1 - k) if (args.stream_order == "snake" and lap % 2 == 1) else k

    def step():
        if not side:
            for L in layers:
                samd.pack(L["x"], L["b"], False, out=L["xp"])
                samd.conv2d_prepared(L["xp"], L["xf"], L["wf"], shape, L["ws"], out=L["y"])
            return
        main = torch.cuda.current_stream()
        for st in side:
            st.wait_stream(main)
        for i, L in enumerate(layers):
            with torch.cuda.stream(side[stream_of[i]]):
                samd.pack(L["x"], L["b"], False, out=L["xp"])
                samd.conv2d_prepared(L["xp"], L["xf"], L["wf"], shape, L["ws"], out=L["y"])
        for st in side:
            main.wait_stream(st)

    # eager steps: every kernel launched from the host (context only)
    for _ in range(min(args.warmup, 20)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t0) * 1e3 / args.steps

    # The timed steps: the step captured once into a HIP graph and replayed.  Warm-up is
    # `warmup` replays and at least `step_warm_s` seconds of them (the GPU's clocks rise
    # under sustained load; a short warm-up would time the ramp), then exactly `steps`
    # replays between two synchronisations, timed with HIP events on the launching stream
    # (the side streams fork from and join it inside the graph).
    step_graph = capture_graph(step, 1)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        step_graph.replay()
    torch.cuda.synchronize()
    t_end = time.perf_counter() + args.step_warm_s
    while time.perf_counter() < t_end:
        for _ in range(10):
            step_graph.replay()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step_graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ms_per_step = e0.elapsed_time(e1) / args.steps
    # the outputs of the timed steps themselves, for the parity check below
    for L in layers:
        L["y_step"] = L["y"].clone()

    def timed(fn, reps):
        return timed_graph_stats(fn, reps, args.kernel_warm_s, args.samples)

    for L in layers:
        samd.conv2d_stage(L["xp"], L["xf"], L["wf"], shape, L["ws"])
        L["t_conv"], L["t_conv_min"] = timed(lambda: samd.conv2d_accumulate(L["xf"], L["wf"], shape, L["ws"],
                                                                             out=L["y"]), args.reps)
        L["t_stage"], _ = timed(lambda: samd.conv2d_stage(L["xp"], L["xf"], L["wf"], shape, L["ws"]), args.reps)
        L["t_pack"], _ = timed(lambda: samd.pack(L["x"], L["b"], False, out=L["xp"]), args.reps)
        L["t_int8"], L["t_int8_min"] = timed(lambda: samd.conv2d_int8_prepared(L["x_nhwc"], L["xf"], L["wf"], shape,
                                                                                L["ws8"], out=L["y8"]), args.reps)
    torch.cuda.synchronize()
    peak_mad = round(measure_peak(samd, "mad") / 1e12, 3) if not args.no_peak_check else None

    # sampled parity against the oracle, same inputs, both paths
    parity = {}
    if not args.no_check:
        from oracle import reference as ref
        rng = np.random.default_rng(0)
        idx = np.stack([rng.integers(0, s, 256) for s in (N, M, Ho, Wo)], axis=1)
        for L in layers:
            want = ref.conv2d_points(L["case"].x, L["case"].w, shape.as_tuple(), idx)
            got = L["y"].cpu().numpy()[tuple(idx.T)]
            got_step = L["y_step"].cpu().numpy()[tuple(idx.T)]
            got8 = L["y8"].cpu().numpy()[tuple(idx.T)]
            parity[L["b"]] = bool(np.array_equal(got, want) and np.array_equal(got_step, want) and
                                  np.array_equal(got8, want))

    traffic = stored_traffic()
    per_bits, tot_mads, tot_conv_s, tot_alg_bytes, tot_word_bytes = {}, 0.0, 0.0, 0.0, 0.0
    for L in layers:
        t, t8 = L["t_conv"], L["t_int8"]
        p = L["plan"]
        mads = N * M * Ho * p.words_per_row * C * KH * p.tap_words
        b = L["b"]
        packed_bytes = N * C * H * samd.row_words(W, b) * 4
        # what the method must move: packed activations at b bits, packed weights at b bits,
        # int32 outputs
        alg_bytes = packed_bytes + M * C * KH * samd.row_words(KW, b) * 4 + N * M * Ho * Wo * 4
        # what this kernel reads and writes at best: the spread operand words and the kernel
        # words once each, the int32 outputs
        word_bytes = (N * C * samd_hp * p.tap_words * p.words_per_row * 4 + M * C * KH * p.tap_words * 4
                      + N * M * Ho * Wo * 4)
        tot_mads += mads
        tot_conv_s += t
        tot_alg_bytes += alg_bytes
        tot_word_bytes += word_bytes
        per_bits[str(b)] = {
            "conv_us": round(t * 1e6, 2), "conv_us_min": round(L["t_conv_min"] * 1e6, 2),
            "stage_us": round(L["t_stage"] * 1e6, 2),
            "pack_us": round(L["t_pack"] * 1e6, 2),
            # packed data: pack reads 1 B per value and writes the packed words; the stage
            # reads the packed words and writes the operand words
            "pack_gbps": round((N * C * H * W + packed_bytes) / L["t_pack"] / 1e9, 1),
            "stage_gbps": round((packed_bytes + N * C * samd_hp * p.tap_words * p.words_per_row * 4) / L["t_stage"]
                                / 1e9, 1),
            "gmacs": round(macs / t / 1e9, 1),
            "gmacs_with_stage": round(macs / (t + L["t_stage"]) / 1e9, 1),
            "int8_us": round(t8 * 1e6, 2), "int8_us_min": round(L["t_int8_min"] * 1e6, 2),
            "int8_gmacs": round(macs / t8 / 1e9, 1),
            "speedup_vs_int8": round(t8 / (t + L["t_stage"]), 3),
            "valu_frac": round(mads / t / PEAK_VALU_OPS, 4),
            "hbm_frac": round(alg_bytes / t / PEAK_HBM, 4),
            "hbm_bytes_alg": alg_bytes,
            "operand_word_bytes": word_bytes,
            "hbm_bytes_counted": (traffic["per_bits"][str(b)]["fetch_bytes"] + traffic["per_bits"][str(b)]["write_bytes"]
                                  if traffic and str(b) in traffic["per_bits"] else None),
            "int8_mfma_frac": round(macs / t8 / PEAK_I8_MACS, 4),
            "int8_launch": L["int8_plan"], "int8_candidates_us": L["int8_cands"],
            "lane_bits": p.lane_bits, "lanes": p.lanes, "tap_words": p.tap_words,
            "flush_channels": p.flush_channels, "macs_per_mad": round(p.macs_per_mad, 2),
            "tile": f"{p.rows_per_block}x{p.mblock}", "split_waves": p.split_waves,
            "rows_per_thread": p.rows_per_thread, "shared_rows": bool(p.shared_rows),
            "chunk_channels": p.chunk_channels,
            "parity": parity.get(b),
        }

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import reference as ref
        # the layers in step order, repeated until the time budget is spent
        done, spent, nlayers = 0, 0.0, 0
        while spent < args.cpu_seconds:
            L = layers[nlayers % len(layers)]
            c0 = time.perf_counter()
            ref.conv2d(L["case"].x, L["case"].w, shape.as_tuple())
            spent += time.perf_counter() - c0
            done += macs
            nlayers += 1
        cpu = {"value": round(done / spent / 1e9, 2), "unit": "GMAC/s", "cores": ref.threads(), "kind": "oracle",
               "sample": f"int64 direct conv2d of the same layer, the step's bit widths {bits_list} in turn "
                         f"({nlayers} layers, {done / 1e9:.1f} GMAC, {spent:.1f} s)",
               "host": host_cpu()}

    achieved = tot_mads / tot_conv_s
    line = {
        "metric": "b-bit quantized conv2d GMAC/s (b=1..8) vs native-int8; % of VALU-int peak",
        "value": round(macs * len(layers) / (ms_per_step * 1e-3) / 1e9, 1),
        "unit": "GMAC/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "wall_ms_per_step": round(wall_ms, 4), "step_warm_s": args.step_warm_s,
        "eager_ms_per_step": round(eager_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int64", "data": "synthetic",
        "config": {"workload": "conv2d 8x128x56x56 -> 128, 3x3, stride 1, pad 1; unsigned b-bit activations x "
                               "signed b-bit weights; one step = pack + stage + accumulate at each b (kernel words prepared once per layer; the 8 independent layers spread over side streams)",
                   "plans": (f"from {os.path.basename(args.plans_in)}" if args.plans_in else "model" if args.no_tune
                             else f"tuned at set-up ({args.tune_candidates} candidates timed)"),
                   "streams": args.streams, "stream_order": args.stream_order,
                   "bits": bits_list, "global_batch": N, "macs_per_layer": macs},
        "device": device_info(torch),
        "roofline": {"bound": "alu", "achieved": round(achieved / 1e12, 3), "peak": round(PEAK_VALU_OPS / 1e12, 2),
                     "unit": "TOP/s", "frac": round(achieved / PEAK_VALU_OPS, 4),
                     # HBM bytes per launch counted by FETCH_SIZE + WRITE_SIZE (mean over the bit
                     # widths), next to the algorithmic bytes the method must move (packed x and w
                     # at b bits, int32 y) and the operand-word bytes this kernel moves at best
                     "traffic": (round(sum(v["hbm_bytes_counted"] for v in per_bits.values()) / len(layers))
                                 if all(v["hbm_bytes_counted"] is not None for v in per_bits.values()) else None),
                     "alg_bytes_per_launch": round(tot_alg_bytes / len(layers)),
                     "operand_word_bytes_per_launch": round(tot_word_bytes / len(layers)),
                     "measured_mad_peak": peak_mad,
                     "kernel": "conv2d_samd_kernel", "op": "32x32->64-bit multiply-accumulate (v_mad_i64_i32)",
                     "timing": f"median of {args.samples} HIP-event-timed replays of a graph of {args.reps} launches"},
        "cpu_baseline": cpu,
        "per_bits": per_bits,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
