#!/usr/bin/env python3
"""Benchmark of the W4A16 GEMM on one MI355X.

One step = the whole hot path over the workload: every decoder-linear GEMM of
the Llama-2-7B set (4 shapes x M in {1,4,16,64,128,256}) and of the
Llama-2-70B set (4 shapes x M in {1,16,128,512,1024}), 44 GEMMs, each with
its own device copy of the packed weights (2.7 GB in all, far beyond the
256 MB Infinity Cache, so every launch streams its weights from HBM).  Inputs
are seeded synthetic tensors from workloads.py, resident in HBM before the
timed region.  The offline pack runs once, untimed, before it.

Timing: the step is captured once as a HIP graph (after eager warm-up on the
capture stream, and checked bit for bit against the eager outputs); the timed
region is K graph replays between device synchronizations, so the host's
per-launch overhead (larger than many small-M kernels) stays out of it.
Per-GEMM times come from HIP events around every GEMM on the launch stream in
separate eager steps, each preceded by a GPU-side wait so the host has
enqueued the whole step before the GPU reaches it.

Printed: one JSON line with the aggregate TFLOP/s (value), the HBM GB/s,
the roofline of the dominant kernel (a graph of just its launches, timed with
HIP events around replays on the launch stream), the same for the
bandwidth-bound small-M points, and the CPU oracle's rate on a bounded sample
(cpu_baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix peak, TFLOP/s
METRIC = "W4A16 GEMM TFLOPS + HBM GB/s vs roofline, M=1..1024, Llama-7B/70B shapes"
ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(ROOT, "paper_2402_10076_amd", "csrc", "quick_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_bench_llama2_7b_70b.json")
COPY_CAL_BYTES = 256 << 20   # plain device copy used to scale the HBM byte counters


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_name(sel: dict) -> str:
    if sel["variant"] == 1:
        return "stream_kernel<MT,%d,%d>" % (sel["tile_n"], sel["split_k"])
    if sel["variant"] == 5:
        return "kstream_kernel<%d>(S=%d)" % (sel["tile_n"], sel["split_k"])
    name = "tiled%s_kernel<%d,%d>" % ("32" if sel["variant"] in (6, 7) else "", sel["tile_m"], sel["tile_n"])
    if sel["variant"] in (3, 7):
        name += "+streamK(G=%d)" % sel["split_k"]
    elif sel["split_k"] > 1:
        name += "+splitk_reduce(S=%d)" % sel["split_k"]
    return name


def kernel_source_digest() -> str:
    """Identifies the kernel code a stored counter measurement belongs to."""
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def launch_sequence(points):
    """Kernel launches of one step, in order: (bench kernel name, symbol prefix)."""
    seq = []
    for p in points:
        sel = p["sel"]
        if sel["variant"] == 1:
            seq.append((p["kernel"], "stream_kernel<"))
        elif sel["variant"] == 5:
            seq.append((p["kernel"], "kstream_kernel<%d>" % sel["tile_n"]))
        elif sel["variant"] in (6, 7):
            seq.append((p["kernel"], "tiled32_kernel<%d, %d, false>" % (sel["tile_m"], sel["tile_n"])))
            if sel["variant"] == 6 and sel["split_k"] > 1:
                seq.append((None, "splitk_reduce_kernel"))
        else:
            seq.append((p["kernel"], "tiled_kernel<%d, %d, 0, false, false>" % (sel["tile_m"], sel["tile_n"])))
            if sel["variant"] == 2 and sel["split_k"] > 1:
                seq.append((None, "splitk_reduce_kernel"))
    return seq


def read_counter_csv(path: str, counter: str):
    """[(dispatch id, kernel symbol, value)] of one rocprofv3 counter CSV, in dispatch order."""
    import csv
    rows = []
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] == counter:
            rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    rows.sort()
    return rows


def dominant_kernel(points_json: str, default: str) -> str:
    """The kernel with the most per-GEMM event time in a bench run's
    --points-out file (how the bench itself picks its dominant kernel);
    `default` when there is no such file."""
    if not points_json or not os.path.exists(points_json):
        return default
    tot = {}
    for p in json.load(open(points_json)):
        tot[p["kernel"]] = tot.get(p["kernel"], 0.0) + p["ms"]
    return max(tot, key=tot.get)


def whole_repetitions(names, seq):
    """How many times the launch sequence `seq` repeats at the start of the
    dispatched kernel `names`."""
    reps = 0
    while (reps + 1) * len(seq) <= len(names) and all(
            prefix in names[reps * len(seq) + i] for i, (_, prefix) in enumerate(seq)):
        reps += 1
    return reps


def launch_points(points):
    """Index of the point each launch of launch_sequence(points) belongs to."""
    idx = []
    for i, p in enumerate(points):
        idx.append(i)
        if p["sel"]["variant"] in (2, 6) and p["sel"]["split_k"] > 1:
            idx.append(i)   # its split-K reduction pass
    return idx


TRAFFIC_MD = os.path.join(ROOT, "profiles", "traffic_per_gemm_llama2_7b_70b.md")
PMC_COMMANDS = "\n".join(
    "timeout -s KILL 300 rocprofv3 --pmc %s --output-format csv -d <dir> -o %s -- python3 <repo>/bench.py %s" % (
        c, o, a) for c, o, a in (("FETCH_SIZE", "f", "--steps 1 --warmup 0 --no-cpu-baseline"),
                                ("WRITE_SIZE", "w", "--steps 1 --warmup 0 --no-cpu-baseline"),
                                ("FETCH_SIZE", "cf", "--copy-calibration"),
                                ("WRITE_SIZE", "cw", "--copy-calibration")))


def ingest_pmc(fetch_csv, write_csv, cal_fetch_csv, cal_write_csv, points, dominant, out_md=TRAFFIC_MD,
               command=""):
    """HBM bytes from FETCH_SIZE / WRITE_SIZE runs of one bench step, each
    scaled by what the counter reads for a plain device-to-device copy of
    COPY_CAL_BYTES: per launch of the dominant kernel (returned, for the
    stored roofline traffic) and per GEMM of the step (split-K reduction
    included), written as a markdown table against the algorithmic bytes."""
    seq = launch_sequence(points)
    lp = launch_points(points)
    per = {}
    per_point = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        ours = [r for r in read_counter_csv(path, name)
                if "anonymous namespace)::" in r[1] and "at::" not in r[1]]
        # whole repetitions of the step's launch sequence from the start
        # (eager warm-up, graph replays, eager timing steps); the subset-graph
        # replays that follow are not used
        reps = whole_repetitions([r[1] for r in ours], seq)
        if reps == 0:
            raise SystemExit("%s: the library dispatches do not start with the step's launch sequence" % path)
        full = seq * reps
        vals = [r[2] for (bname, _), r in zip(full, ours) if bname == dominant]
        if not vals:
            raise SystemExit("no launch of %s in the step" % dominant)
        per[name] = float(np.mean(vals))
        acc = np.zeros(len(points))
        for k in range(reps * len(seq)):
            acc[lp[k % len(seq)]] += ours[k][2]
        per_point[name] = acc / reps
    cal = {}
    for name, path in (("FETCH_SIZE", cal_fetch_csv), ("WRITE_SIZE", cal_write_csv)):
        # the device-to-device copies of the calibration run (HIP runtime copy kernel)
        v = [r[2] for r in read_counter_csv(path, name) if "copyBuffer" in r[1]]
        top = max(v)
        cal[name] = (COPY_CAL_BYTES / 1024.0) / float(np.median([x for x in v if x >= 0.9 * top]))
    fetch_b = per["FETCH_SIZE"] * cal["FETCH_SIZE"] * 1024.0
    write_b = per["WRITE_SIZE"] * cal["WRITE_SIZE"] * 1024.0
    if out_md:
        lines = ["| cfg | shape | K | N | M | kernel | fetched MB | written MB | alg. read MB | alg. write MB | "
                 "fetched / alg. read | written / alg. write |", "|---|---|---|---|---|---|---|---|---|---|---|---|"]
        for i, p in enumerate(points):
            fb = per_point["FETCH_SIZE"][i] * cal["FETCH_SIZE"] * 1024.0
            wb = per_point["WRITE_SIZE"][i] * cal["WRITE_SIZE"] * 1024.0
            aw = 2 * p["M"] * p["N"]
            ar = p["bytes"] - aw
            lines.append("| C%d | %s | %d | %d | %d | %s | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f |" % (
                p["cid"], p["shape"], p["K"], p["N"], p["M"], p["kernel"], fb / 1e6, wb / 1e6, ar / 1e6, aw / 1e6,
                fb / ar, wb / aw))
        with open(out_md, "w") as f:
            f.write("# HBM traffic per GEMM of the bench step (rocprofv3 FETCH_SIZE / WRITE_SIZE)\n\n")
            f.write("Commands (from the repository root on an MI355X, after `cd /tmp && export TMPDIR=/tmp`), "
                    "each counter in a run of its own:\n\n```\n%s\n```\n\n" % command)
            f.write("Then `python bench.py --ingest-pmc <fetch.csv> <write.csv> <cal_fetch.csv> <cal_write.csv>` "
                    "(CPU).  Means over %d repetitions of the step's launch sequence; a split GEMM includes its "
                    "reduction pass.  Counter readings are scaled by a plain %d MiB device-to-device copy of the same "
                    "run type: FETCH_SIZE x %.3f, WRITE_SIZE x %.3f.  Algorithmic read bytes = packed weights, scales, "
                    "zeros and x (each once); algorithmic write bytes = y.  FETCH_SIZE counts L2 misses, which "
                    "include reads served by the Infinity Cache.\n\n" % (
                        reps, COPY_CAL_BYTES >> 20, cal["FETCH_SIZE"], cal["WRITE_SIZE"]))
            f.write("\n".join(lines) + "\n")
    return {
        "kernel": dominant,
        "kernel_source_sha256_16": kernel_source_digest(),
        "launches": int(sum(1 for b, _ in seq if b == dominant)),
        "fetch_kib_per_dispatch": round(per["FETCH_SIZE"], 1),
        "write_kib_per_dispatch": round(per["WRITE_SIZE"], 1),
        "fetch_scale": round(cal["FETCH_SIZE"], 4),
        "write_scale": round(cal["WRITE_SIZE"], 4),
        "hbm_bytes_per_launch": int(round(fetch_b + write_b)),
        "alg_bytes_per_launch": int(round(np.mean([p["bytes"] for p in points if p["kernel"] == dominant]))),
    }


def ingest_trace(trace_csv, points, dominant, out_md, command, run_log=""):
    """Kernel durations per GEMM of the step from a rocprofv3 kernel trace of
    a bench run (the run issues the step's launch sequence a whole number of
    times), written as a markdown table; returns the dominant kernel's mean
    duration in microseconds."""
    import csv
    seq = launch_sequence(points)
    rows = []
    for r in csv.DictReader(open(trace_csv)):
        if "anonymous namespace)::" in r["Kernel_Name"] and "at::" not in r["Kernel_Name"]:
            rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"],
                         (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3))
    rows.sort()
    # whole repetitions of the step from the start (eager warm-up, graph
    # replays, eager event steps); the subset-graph replays that follow are
    # not used
    reps = whole_repetitions([r[1] for r in rows], seq)
    if reps == 0:
        raise SystemExit("%s: the library dispatches do not start with the step's launch sequence" % trace_csv)
    # per point: its kernels' durations (tiled kernel + reduction when split), per repetition
    per_point = [[0.0] * reps for _ in points]
    dom_launch = []
    j = 0
    for rep in range(reps):
        for i, p in enumerate(points):
            n = 2 if (p["sel"]["variant"] in (2, 6) and p["sel"]["split_k"] > 1) else 1
            for t in range(n):
                per_point[i][rep] += rows[j + t][2]
            if p["kernel"] == dominant:
                dom_launch.append(rows[j][2])
            j += n
    def roof_us(p):
        # the GEMM's time at its binding roofline (HBM bytes or matrix flops at peak)
        return max(p["bytes"] / HBM_PEAK_GBS / 1e3, p["flops"] / MFMA_F16_PEAK_TFLOPS / 1e6)

    lines = ["| cfg | shape | K | N | M | kernel | mean us | min us | GB/s | TFLOP/s | bound | fraction of roofline |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    tot = 0.0
    for i, p in enumerate(points):
        mu = float(np.mean(per_point[i]))
        tot += mu
        hbm = p["bytes"] / HBM_PEAK_GBS / 1e3 >= p["flops"] / MFMA_F16_PEAK_TFLOPS / 1e6
        lines.append("| C%d | %s | %d | %d | %d | %s | %.2f | %.2f | %.0f | %.1f | %s | %.3f |" % (
            p["cid"], p["shape"], p["K"], p["N"], p["M"], p["kernel"], mu, min(per_point[i]),
            p["bytes"] / mu / 1e3, p["flops"] / mu / 1e6, "hbm" if hbm else "mfma", roof_us(p) / mu))
    dom_us = float(np.mean(dom_launch))
    # the replays of the graph of the dominant kernel's launches alone, which
    # follow the step repetitions: the launches bench.py's roofline times
    n_dom = sum(1 for p in points if p["kernel"] == dominant)
    dom_prefix = next(pre for b, pre in seq if b == dominant)
    k = j
    while k < len(rows) and dom_prefix in rows[k][1]:
        k += 1
    sub = [r[2] for r in rows[j:j + (k - j) // n_dom * n_dom]]
    small = [i for i, p in enumerate(points) if p["M"] <= 16]
    s_us = sum(float(np.mean(per_point[i])) for i in small)
    s_gbs = sum(points[i]["bytes"] for i in small) / s_us / 1e3
    big = [i for i, p in enumerate(points) if p["M"] >= 256]
    b_tf = sum(points[i]["flops"] for i in big) / sum(float(np.mean(per_point[i])) for i in big) / 1e6 if big else 0
    band = [i for i, p in enumerate(points) if 64 <= p["M"] <= 256]
    band_frac = (sum(roof_us(points[i]) for i in band) / sum(float(np.mean(per_point[i])) for i in band)
                 if band else 0)
    with open(out_md, "w") as f:
        f.write("# Kernel durations of the bench step (rocprofv3 kernel trace)\n\n")
        f.write("Command (from the repository root on an MI355X, after `cd /tmp && export TMPDIR=/tmp`):\n\n")
        f.write("```\n%s\n```\n\n" % command)
        f.write("Then `python bench.py --ingest-trace <kernel_trace.csv> --trace-out <this file>` (CPU).\n\n")
        f.write("%d library dispatches = %d repetitions of the step's %d launches (eager warm-up, "
                "graph replays, eager event steps); each row averages the point's kernel time "
                "(tiled kernel + split-K reduction where split) over the repetitions.\n\n" % (
                    len(rows), reps, len(seq)))
        f.write("* Dominant kernel `%s`: %d launches per step, mean kernel duration **%.2f us**.\n" % (
            dominant, n_dom, dom_us))
        if sub:
            f.write("* The same launches in the %d replays of the graph of the dominant kernel's launches alone "
                    "(what the bench's `roofline.avg_launch_us` times): mean kernel duration **%.2f us**.\n" % (
                        len(sub) // n_dom, float(np.mean(sub))))
        roof = None
        if run_log and os.path.exists(run_log):
            for line in open(run_log, errors="replace"):
                if line.startswith("{") and '"roofline"' in line:
                    roof = json.loads(line)["roofline"]
        if roof:
            f.write("* bench.py's own JSON line from the profiled run: `roofline.avg_launch_us` = %.2f us "
                    "(replay time of that graph / launches, so it also holds the gaps between launches), "
                    "`frac` = %.4f.\n" % (roof["avg_launch_us"], roof["frac"]))
        f.write("* Sum of kernel time per step: %.1f us.\n" % tot)
        f.write("* GEMMs with M <= 16: %.1f us of kernels, %.0f GB/s of algorithmic bytes (%.3f of %d GB/s).\n" % (
            s_us, s_gbs, s_gbs / HBM_PEAK_GBS, HBM_PEAK_GBS))
        if big:
            f.write("* GEMMs with M >= 256: %.1f TFLOP/s of kernel time (%.3f of %d TFLOP/s).\n" % (
                b_tf, b_tf / MFMA_F16_PEAK_TFLOPS, MFMA_F16_PEAK_TFLOPS))
        if band:
            f.write("* GEMMs with 64 <= M <= 256 (%d): %.3f of their binding rooflines together (sum of the "
                    "roofline times over the sum of the kernel times).\n" % (len(band), band_frac))
        f.write("\n")
        f.write("\n".join(lines) + "\n")
        stats = trace_csv.replace("_kernel_trace.csv", "_kernel_stats.csv")
        if stats != trace_csv and os.path.exists(stats):
            # the profiler's own --stats summary of the same run, per kernel symbol
            # (every launch of the run: warm-up, eager steps, graph replays)
            f.write("\nrocprofv3 `--stats` summary of the same run (%s), all launches of each "
                    "kernel symbol:\n\n" % os.path.basename(stats))
            f.write("| kernel | calls | average us | min us | max us | % of time |\n|---|---|---|---|---|---|\n")
            for r in csv.DictReader(open(stats)):
                name = r["Name"].replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0]
                f.write("| `%s` | %s | %.2f | %.2f | %.2f | %.2f |\n" % (
                    name, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                    float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    return dom_us


MFMA_COUNTERS = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_F16", "SQ_BUSY_CU_CYCLES", "SQ_INSTS_LDS",
                 "SQ_LDS_BANK_CONFLICT", "SQ_INSTS_VALU", "SQ_WAVE_CYCLES", "GRBM_GUI_ACTIVE")
MI355X_XCDS = 8
MI355X_SIMDS = 256 * 4
MI355X_PEAK_GHZ = 2.4


def gemm_counters(csv_path, points, counters):
    """Counter values of each GEMM kernel launch of the step from a rocprofv3
    --pmc CSV: (whole repetitions of the launch sequence, per point a dict
    counter -> list over repetitions (plus "dur", ns), and (duration ns,
    GRBM_GUI_ACTIVE) of the runtime's copy kernels)."""
    import csv
    seq = launch_sequence(points)
    disp = {}
    copies = []
    for r in csv.DictReader(open(csv_path)):
        name = r["Kernel_Name"]
        dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        if "copyBuffer" in name and r["Counter_Name"] == "GRBM_GUI_ACTIVE":
            copies.append((dur, float(r["Counter_Value"])))
        if "anonymous namespace)::" not in name or "at::" in name:
            continue
        d = disp.setdefault(int(r["Dispatch_Id"]), {"name": name, "dur": dur})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    ids = sorted(disp)
    names = [disp[i]["name"] for i in ids]
    reps = whole_repetitions(names, seq)
    if reps == 0:
        raise SystemExit("%s: the library dispatches do not start with the step's launch sequence" % csv_path)
    acc = [dict() for _ in points]
    j = 0
    for _ in range(reps):
        for i, p in enumerate(points):
            d = disp[ids[j]]   # the GEMM kernel itself (a split-K reduction follows it)
            for c in tuple(counters) + ("dur",):
                acc[i].setdefault(c, []).append(d.get(c, 0.0))
            j += 2 if (p["sel"]["variant"] in (2, 6) and p["sel"]["split_k"] > 1) else 1
    return reps, acc, copies


WAIT_COUNTERS = ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU",
                 "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_VMEM")
WAITS_MD = os.path.join(ROOT, "profiles", "wave_states_bench_llama2_7b_70b.md")


def ingest_waits(csv_path, points, out_md, command):
    """Where the waves of each GEMM launch spend their time, from one
    rocprofv3 --pmc run of WAIT_COUNTERS: each counter over SQ_WAVE_CYCLES
    (all accumulate per wave, in the same units)."""
    reps, acc, _ = gemm_counters(csv_path, points, WAIT_COUNTERS)
    lines = ["| cfg | shape | K | N | M | kernel | us | waiting on a dependency | ready, not issued | issuing | "
             "VALU | LDS | VMEM |", "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for i, p in enumerate(points):
        a = {c: float(np.mean(v)) for c, v in acc[i].items()}
        wc = a["SQ_WAVE_CYCLES"] or 1.0
        lines.append("| C%d | %s | %d | %d | %d | %s | %.1f | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f |" % (
            p["cid"], p["shape"], p["K"], p["N"], p["M"], p["kernel"], a["dur"] / 1000.0,
            a["SQ_WAIT_ANY"] / wc, a["SQ_WAIT_INST_ANY"] / wc, a["SQ_ACTIVE_INST_ANY"] / wc,
            a["SQ_ACTIVE_INST_VALU"] / wc, a["SQ_ACTIVE_INST_LDS"] / wc, a["SQ_ACTIVE_INST_VMEM"] / wc))
    with open(out_md, "w") as f:
        f.write("# Wave states per GEMM of the bench step (rocprofv3 counters)\n\n")
        f.write("Command (from the repository root on an MI355X, after `cd /tmp && export TMPDIR=/tmp`):\n\n")
        f.write("```\n%s\n```\n\n" % command)
        f.write("Then `python bench.py --ingest-waits <counter_collection.csv>` (CPU). %d repetitions of the step's "
                "launch sequence; means per GEMM kernel launch (the split-K reduction pass is not included). Every "
                "column after the duration is a counter over SQ_WAVE_CYCLES, the summed lifetime of the launch's "
                "waves:\n\n"
                "* waiting on a dependency = SQ_WAIT_ANY (a wait count or a barrier: memory latency, LDS, or other "
                "waves);\n"
                "* ready, not issued = SQ_WAIT_INST_ANY (an instruction is ready but its unit or the issue port is "
                "busy, e.g. the matrix unit running the other wave's instructions);\n"
                "* issuing = SQ_ACTIVE_INST_ANY, split into VALU (matrix instructions included), LDS and "
                "VMEM.\n\n" % reps)
        f.write("\n".join(lines) + "\n")
    return reps


def ingest_mfma(csv_path, points, out_md, command):
    """Matrix-core utilisation per GEMM of the step from one rocprofv3 --pmc
    run of MFMA_COUNTERS over this script (--steps 1 --warmup 0): busy cycles
    of the matrix units over the GPU's active cycles times the SIMDs (the
    profiler's MfmaUtil), the matrix operations issued against the GEMM's
    algorithmic flops, the vector-ALU instructions against those of one
    dequantization of every weight, the LDS instruction and bank-conflict
    counts, and the achieved clock of the longer launches."""
    reps, acc, copies = gemm_counters(csv_path, points, MFMA_COUNTERS)
    # GRBM_GUI_ACTIVE covers a window a fixed number of cycles longer than the
    # dispatch: fit cycles per XCD = clock x duration + window over the copy
    # kernels of the run (lightly loaded, so one clock) and take the window out
    window = 0.0
    if len(copies) >= 3:
        cd = np.array(copies, dtype=np.float64)
        _, window = np.polyfit(cd[:, 0], cd[:, 1] / MI355X_XCDS, 1)
    lines = ["| cfg | shape | K | N | M | kernel | matrix busy % | matrix flops / algorithmic | VALU / one dequant | "
             "clock GHz | LDS instr | LDS bank conflicts |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for i, p in enumerate(points):
        a = {c: float(np.mean(v)) for c, v in acc[i].items()}
        active = a["GRBM_GUI_ACTIVE"] / MI355X_XCDS
        util = 100.0 * a["SQ_VALU_MFMA_BUSY_CYCLES"] / (active * MI355X_SIMDS) if active else 0.0
        mflops = a["SQ_INSTS_VALU_MFMA_MOPS_F16"] * 512
        # one dequantization of every weight: 13 wave instructions per 64 lanes x 8 weights
        deq = 13.0 * p["K"] * p["N"] / 512.0
        # SQ_INSTS_VALU counts the matrix instructions too (16384 flops each,
        # 32768 for the 32x32x16 form)
        mfma_insts = mflops / (32768.0 if p["kernel"].startswith("tiled32") else 16384.0)
        clock = (active - window) / a["dur"] if a["dur"] >= 20000 else float("nan")
        if clock > MI355X_PEAK_GHZ:
            # more than the kernel fell into the counter window: the clock
            # (and the busy fraction over that window) is not the kernel's
            clock, util = float("nan"), float("nan")
        lines.append("| C%d | %s | %d | %d | %d | %s | %s | %.2f | %.2f | %s | %.3g | %.3g |" % (
            p["cid"], p["shape"], p["K"], p["N"], p["M"], p["kernel"], "%.1f" % util if util == util else "-",
            mflops / p["flops"],
            (a["SQ_INSTS_VALU"] - mfma_insts) / deq, "%.2f" % clock if clock == clock else "-", a["SQ_INSTS_LDS"],
            a["SQ_LDS_BANK_CONFLICT"]))
    with open(out_md, "w") as f:
        f.write("# Matrix-core utilisation per GEMM of the bench step (rocprofv3 counters)\n\n")
        f.write("Command (from the repository root on an MI355X, after `cd /tmp && export TMPDIR=/tmp`):\n\n")
        f.write("```\n%s\n```\n\n" % command)
        f.write("Then `python bench.py --ingest-mfma <counter_collection.csv>` (CPU). %d repetitions of the step's "
                "launch sequence; values are means per GEMM kernel launch (the split-K reduction pass is not "
                "included).\n\n"
                "* matrix busy %% = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / %d XCDs x %d SIMDs), the "
                "profiler's MfmaUtil.\n"
                "* matrix flops = SQ_INSTS_VALU_MFMA_MOPS_F16 x 512 against 2MNK (above 1 where M is padded to "
                "16-row blocks).\n"
                "* VALU / one dequant = the launch's vector-ALU wave instructions other than matrix instructions "
                "(SQ_INSTS_VALU, which counts those too, less the matrix instructions from the MOPS count; address "
                "arithmetic and epilogue included) over 13 K N / 512, the instructions of dequantizing every weight "
                "once (13 per 8 weights of 64 lanes); a tiled launch dequantizes each weight once per row tile, so "
                "the ideal is the number of row tiles, ceil(M / BM).\n"
                "* clock = (GRBM_GUI_ACTIVE / %d XCDs - window) / kernel duration (counter-run timestamps), for "
                "launches of at least 20 us; window = %.0f cycles, the fixed excess of the counter window over the "
                "dispatch, fitted over the run's runtime copy kernels. Where this comes out above the chip's "
                "%.1f GHz peak clock, more than the kernel fell into the counter window: that row's clock and "
                "matrix busy %% are shown as -.\n\n" % (
                    reps, MI355X_XCDS, MI355X_SIMDS, MI355X_XCDS, window, MI355X_PEAK_GHZ))
        f.write("\n".join(lines) + "\n")
    return reps


def stored_traffic(dominant: str):
    """HBM bytes per launch from the stored counter measurement, or None when
    there is none for this kernel or the kernel source changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel") != dominant or t.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return t.get("hbm_bytes_per_launch")


def copy_calibration():
    import torch
    n = COPY_CAL_BYTES // 4
    src = torch.arange(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    assert bool((dst == src).all())
    log("copy calibration: 5 x %d MiB device copies" % (COPY_CAL_BYTES >> 20))


READ_CEILING_MB = (4.4, 8.7, 17.4, 23.4, 26.2, 34.9, 43.6, 46.9, 65.9, 122.0, 244.0)


def read_ceiling(sizes_mb=READ_CEILING_MB, reps=40):
    """The practical ceiling of short HBM transfers: device-to-device copies
    (torch, the HIP runtime's copy kernel) of the packed-weight sizes of the
    benchmark GEMMs, each copy rotating through sources and destinations
    spanning >= 1 GiB (so every copy streams from HBM, not the Infinity
    Cache), `reps` copies captured in a graph and timed with HIP events
    around replays.  Returns per size the copy time and the read rate (bytes
    read / time) and read + write rate."""
    import torch
    rows = []
    st = torch.cuda.Stream()
    for mb in sizes_mb:
        n = int(mb * 1e6) // 16 * 16
        k = max(2, -(-(1 << 30) // n))
        src = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(k)]
        dst = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(k)]
        for t in src:
            t.fill_(1)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=st):
            for r in range(reps):
                dst[r % k].copy_(src[(r + 1) % k])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        best = None
        with torch.cuda.stream(st):
            g.replay()
            for _ in range(5):
                e0.record()
                g.replay()
                e1.record()
                e1.synchronize()
                us = e0.elapsed_time(e1) / reps * 1e3
                best = us if best is None else min(best, us)
        rows.append(dict(mb=mb, bytes=n, copies_rotated=k, us=round(best, 2),
                         read_gbs=round(n / best / 1e3, 1), read_write_gbs=round(2 * n / best / 1e3, 1)))
        log("read ceiling %7.1f MB: %8.2f us, read %7.1f GB/s, read+write %7.1f GB/s" % (
            mb, best, n / best / 1e3, 2 * n / best / 1e3))
        del g, src, dst
        torch.cuda.empty_cache()
    return rows


def compare_fp16(K, N, Ms, reps=20):
    """Context only: the W4A16 GEMM beside an fp16 GEMM of the same shape
    through torch (hipBLASLt) on the dequantized weights, each timed with HIP
    events over `reps` back-to-back launches that rotate through enough
    weight copies to stream from HBM."""
    import torch
    import paper_2402_10076_amd as Q
    import workloads as W
    q, z, s = W.draw_weights(5, 1, K, N)
    pw, ps, pz = Q.pack_weights(q, z, s)
    wq = Q.to_device(pw, ps, pz)
    # fp16 weights for the reference GEMM, dequantized on the device by the
    # library itself (one-hot activations select the rows of W)
    eye = torch.eye(K, dtype=torch.float16, device="cuda")
    w16 = Q.w4a16_gemm(eye, *wq, N)
    del eye
    wbytes = K * N // 2
    nq = max(2, -(-(1 << 30) // wbytes))
    n16 = max(2, -(-(1 << 30) // (2 * K * N)))
    qcopies = [tuple(t.clone() for t in wq) for _ in range(nq)]
    hcopies = [w16.clone() for _ in range(n16)]
    rows = []
    for M in Ms:
        x = torch.randn(M, K, device="cuda").half()
        y = torch.empty(M, N, device="cuda", dtype=torch.float16)

        def timed(fn):
            for i in range(3):
                fn(i)
            torch.cuda.synchronize()
            torch.cuda._sleep(5_000_000)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(reps):
                fn(i)
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps * 1e3
        t_q = timed(lambda i: Q.w4a16_gemm(x, *qcopies[i % nq], N, y=y))
        t_h = timed(lambda i: torch.matmul(x, hcopies[i % n16], out=y))
        rows.append(dict(M=M, w4a16_us=round(t_q, 2), fp16_us=round(t_h, 2), speedup=round(t_h / t_q, 3)))
        log("K=%d N=%d M=%5d  W4A16 %9.2f us  fp16 hipBLASLt %9.2f us  speedup %.2fx" % (K, N, M, t_q, t_h, t_h / t_q))
    return rows


def ablation(shapes, reps=20):
    """The method's central choice measured: the same 64 x 256 tiled kernel
    with the dequantized weights going straight to the fragment registers
    (mode 0) or through an LDS tile and back (mode 1 padded rows, mode 2
    unpadded rows); HIP events over `reps` back-to-back launches rotating
    through >= 1 GiB of weight copies."""
    import torch
    import paper_2402_10076_amd as Q
    import workloads as W
    rows = []
    for K, N, Ms in shapes:
        q, z, s = W.draw_weights(5, 2, K, N)
        wq = Q.to_device(*Q.pack_weights(q, z, s))
        nq = max(2, -(-(1 << 30) // (K * N // 2)))
        copies = [tuple(t.clone() for t in wq) for _ in range(nq)]
        for M in Ms:
            x = torch.randn(M, K, device="cuda").half()
            y = torch.empty(M, N, device="cuda", dtype=torch.float16)
            t = []
            for mode in (0, 1, 2):
                for i in range(3):
                    Q.ablation_gemm(x, *copies[i % nq], N, mode, y=y)
                torch.cuda.synchronize()
                torch.cuda._sleep(5_000_000)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for i in range(reps):
                    Q.ablation_gemm(x, *copies[i % nq], N, mode, y=y)
                e1.record()
                torch.cuda.synchronize()
                t.append(e0.elapsed_time(e1) / reps * 1e3)
            rows.append(dict(K=K, N=N, M=M, direct_us=round(t[0], 2), writeback_padded_us=round(t[1], 2),
                             writeback_unpadded_us=round(t[2], 2)))
            log("K=%5d N=%5d M=%5d  direct %8.2f us  write-back padded %8.2f us (%.2fx)  unpadded %8.2f us (%.2fx)"
                % (K, N, M, t[0], t[1], t[1] / t[0], t[2], t[2] / t[0]))
        del copies
    return rows


def moe(reps=20, sweep=True):
    """Mixtral-8x7B expert FFN on one GPU (512 tokens, top-2 routing over 8
    experts, about 128 rows per expert): the 24 expert GEMMs (w1, w3 over the
    routed tokens, w2 over fresh [M_e][14336] inputs) as 24 dense GEMMs on
    pre-gathered activations, against 3 grouped GEMMs that gather the
    token rows inside the kernel.  Each form is one HIP graph, checked against
    its eager run and timed with HIP events over `reps` replays (the faster
    of two such timings)."""
    import torch
    import paper_2402_10076_amd as Q
    import workloads as W
    routes = W.mixtral_routing()
    counts = [len(r) for r in routes]
    R = sum(counts)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    od = torch.from_numpy(offsets).cuda()
    rd = torch.from_numpy(np.concatenate(routes).astype(np.int32)).cuda()
    xt = torch.from_numpy(W.mixtral_tokens().view(np.int16)).cuda().view(torch.float16)
    xg = [xt[torch.from_numpy(r).cuda()].contiguous() for r in routes]   # gathered outside the GEMMs
    h = torch.from_numpy(np.concatenate([W.mixtral_w2_input(e, counts[e]) for e in range(8)]).view(np.int16))
    h = h.cuda().view(torch.float16)
    mats = []
    flops = 0
    for which in range(3):
        experts = [W.mixtral_expert_weights(e, which) for e in range(8)]
        K, N = experts[0][0].shape
        dw, ds, dz = Q.to_device(*Q.pack_experts(experts))
        wb, zb, sb = Q.packed_sizes(K, N)
        views = [(dw[e * wb // 4:(e + 1) * wb // 4], ds[e * sb // 2:(e + 1) * sb // 2],
                  dz[e * zb // 4:(e + 1) * zb // 4]) for e in range(8)]
        mats.append(dict(K=K, N=N, w=(dw, ds, dz), views=views,
                         y_dense=torch.empty(R, N, dtype=torch.float16, device="cuda"),
                         y_grp=torch.empty(R, N, dtype=torch.float16, device="cuda")))
        flops += 2 * R * N * K
    stream = torch.cuda.Stream()

    def dense():
        for which, m in enumerate(mats):
            for e in range(8):
                lo, hi = int(offsets[e]), int(offsets[e + 1])
                x = xg[e] if which < 2 else h[lo:hi]
                Q.w4a16_gemm(x, *m["views"][e], m["N"], y=m["y_dense"][lo:hi])

    def grouped(cfg):
        for which, m in enumerate(mats):
            if which < 2:
                Q.grouped_gemm(xt, od, *m["w"], m["N"], rows=rd, y=m["y_grp"], cfg=cfg)
            else:
                Q.grouped_gemm(h, od, *m["w"], m["N"], y=m["y_grp"], cfg=cfg)

    def timed(fn, outs):
        with torch.cuda.stream(stream):
            fn()
        stream.synchronize()
        ref = [o.clone() for o in outs]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            fn()
        for o in outs:
            o.zero_()
        # the faster of two timings of `reps` replays, after 10 warm-up
        # replays: the form timed first after another one otherwise reads a
        # few percent slow
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2)]
        with torch.cuda.stream(stream):
            for _ in range(10):
                g.replay()
            for e0, e1 in evs:
                e0.record()
                for _ in range(reps):
                    g.replay()
                e1.record()
        torch.cuda.synchronize()
        if not all(torch.equal(a, b) for a, b in zip(outs, ref)):
            raise SystemExit("graph replay differs from the eager run")
        return min(e0.elapsed_time(e1) for e0, e1 in evs) / reps * 1e3

    t_dense = timed(dense, [m["y_dense"] for m in mats])
    rows = [dict(form="24 dense GEMMs (pre-gathered rows)", us=round(t_dense, 2),
                 tflops=round(flops / t_dense / 1e6, 1))]
    log("Mixtral 8x7B experts, R=%d routed rows (per expert %s), %.1f GFLOP" % (R, counts, flops / 1e9))
    log("  24 dense GEMMs           %9.2f us  %7.1f TFLOP/s" % (t_dense, flops / t_dense / 1e6))
    cfgs = [None]
    if sweep:
        for bm, wn in ((64, 32), (128, 32)):
            cfgs += [Q.make_config(variant=3, tile_m=bm, tile_n=wn)]
            cfgs += [Q.make_config(variant=2, split_k=s, tile_m=bm, tile_n=wn) for s in (1, 2, 4)]
    outs = [m["y_grp"] for m in mats]
    for cfg in cfgs:
        t = timed(lambda: grouped(cfg), outs)
        if cfg is None:
            sel = Q.grouped_select_config(R, 8, mats[0]["N"], mats[0]["K"])
            name = "auto %s" % (sel,)
            if sel["tile_m"] == 128:
                name += " + remainders < 64 rows in 32x32 tiles"
        else:
            name = "v%d split %d tile %dx%d" % (cfg.variant, cfg.split_k, cfg.tile_m, cfg.tile_n)
        diff = max(float((a.float() - b.float()).abs().max() / b.float().abs().max())
                   for a, b in zip(outs, [m["y_dense"] for m in mats]))
        rows.append(dict(form="3 grouped GEMMs, " + name, us=round(t, 2), tflops=round(flops / t / 1e6, 1),
                         speedup=round(t_dense / t, 3), max_rel_diff_vs_dense=round(diff, 6)))
        log("  3 grouped GEMMs %-42s %9.2f us  %7.1f TFLOP/s  %.2fx  (max rel diff vs dense %.2g)" % (
            name, t, flops / t / 1e6, t_dense / t, diff))
    # the layer as it runs: w1 and w3 as one grouped launch over their
    # interleaved columns with the gated SiLU fused into the epilogue, then
    # w2 over that output (the SiLU-gated product never leaves registers in
    # f32 and is rounded once)
    q13 = []
    for e in range(8):
        g1 = W.mixtral_expert_weights(e, 0)
        g3 = W.mixtral_expert_weights(e, 1)
        q13.append(Q.interleave_gate_up(g1, g3))
    w13 = Q.to_device(*Q.pack_experts(q13))
    h13 = torch.empty(R, 14336, dtype=torch.float16, device="cuda")
    y2 = torch.empty(R, 4096, dtype=torch.float16, device="cuda")

    def chain():
        Q.grouped_gemm_fused(xt, od, *w13, 2 * 14336, rows=rd, activation=Q.ACT_SILU_GATE, y=h13)
        Q.grouped_gemm(h13, od, *mats[2]["w"], 4096, y=y2)

    t = timed(chain, [h13, y2])
    rows.append(dict(form="2 grouped GEMMs: w1|w3 with the fused gated SiLU, then w2 on its output",
                     us=round(t, 2), tflops=round(flops / t / 1e6, 1), speedup=round(t_dense / t, 3)))
    log("  2 grouped GEMMs, fused SiLU gate       %9.2f us  %7.1f TFLOP/s  %.2fx" % (t, flops / t / 1e6, t_dense / t))
    return dict(routed_rows=R, rows_per_expert=counts, gflop=round(flops / 1e9, 2), rows=rows)


def build_points(configs):
    import workloads as W
    pts = []
    for cid in configs:
        cfg = W.CONFIGS[cid]
        for si, sh in enumerate(cfg.shapes):
            for M in sh.Ms:
                pts.append(dict(cid=cid, si=si, shape=sh.name, K=sh.K, N=sh.N, M=M))
    return pts


def cpu_baseline(points, threads: int, col_fraction: float):
    """The oracle (as it stands) on a bounded sample: every (shape, M) point,
    all rows, a seeded sample of ceil(N * col_fraction) columns."""
    import oracle
    import workloads as W
    t_total = 0.0
    t_extra = 0.0   # each point's time scaled to all N columns
    fl_total = 0
    cache = {}
    for p in points:
        key = (p["cid"], p["si"])
        if key not in cache:
            cache.clear()
            cfg = W.CONFIGS[p["cid"]]
            sh = cfg.shapes[p["si"]]
            x = W.draw_x(p["cid"], p["si"], max(sh.Ms), sh.K, cfg.outliers)
            cache[key] = (x,) + W.draw_weights(p["cid"], p["si"], sh.K, sh.N)
        x, q, z, s = cache[key]
        ncols = max(1, int(np.ceil(p["N"] * col_fraction)))
        cols = W.sample_columns(p["N"], ncols, seed=1)
        t0 = time.perf_counter()
        oracle.gemm(x[:p["M"]], q, z, s, cols=cols, threads=threads)
        dt = time.perf_counter() - t0
        t_total += dt
        t_extra += dt * p["N"] / len(cols)
        fl_total += 2 * p["M"] * len(cols) * p["K"]
    return fl_total, t_total, t_extra


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_c1_one_thread():
    """The oracle on the 16 x 512 x 512 configuration, all columns, one thread."""
    import oracle
    import workloads as W
    x, q, z, s = W.shape_inputs(W.C1, 0, 16)
    t0 = time.perf_counter()
    oracle.gemm(x, q, z, s, threads=1)
    return time.perf_counter() - t0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--configs", default="2,5", help="workload configs (2 = Llama-2-7B, 5 = Llama-2-70B)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--moe", action="store_true",
                    help="time the Mixtral-8x7B expert GEMMs: 24 dense GEMMs vs 3 grouped GEMMs")
    ap.add_argument("--moe-auto-only", action="store_true", help="with --moe: only the automatic grouped config")
    ap.add_argument("--cpu-col-fraction", type=float, default=1.0 / 8)
    ap.add_argument("--points-out", default="", help="optional path for the per-GEMM table (JSON)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain %d MiB device copy (scales rocprofv3 byte counters)" % (COPY_CAL_BYTES >> 20))
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH_CSV", "CAL_WRITE_CSV"),
                    help="turn rocprofv3 FETCH_SIZE / WRITE_SIZE runs of one step (--steps 1 --warmup 0) and "
                         "of --copy-calibration into the stored HBM traffic of the dominant kernel")
    ap.add_argument("--dominant", default="",
                    help="kernel name for --ingest-pmc/--ingest-trace (default: the dominant kernel of the "
                         "--points-out file of the profiled bench run)")
    ap.add_argument("--read-ceiling", action="store_true",
                    help="only time device-to-device copies of the benchmark's weight sizes (HBM ceiling of "
                         "short transfers, context for the M <= 16 roofline)")
    ap.add_argument("--compare-fp16", action="store_true",
                    help="only compare the W4A16 GEMM with an fp16 GEMM through torch (hipBLASLt) on the "
                         "8192x8192 Llama-2-70B o_proj shape over M (context, not the metric)")
    ap.add_argument("--compare-shape", default="8192,8192", metavar="K,N",
                    help="with --compare-fp16: the weight shape")
    ap.add_argument("--compare-m", default="1,4,16,32,64,128,256,512,1024,2048",
                    help="with --compare-fp16: the batch sizes")
    ap.add_argument("--tune", action="store_true",
                    help="autotune every GEMM shape of the step during setup (untimed) before timing")
    ap.add_argument("--tune-save", default="", help="with --tune: write the tune table here")
    ap.add_argument("--tune-table", default=os.path.join(ROOT, "paper_2402_10076_amd", "tune_mi355x.txt"),
                    help="tune table loaded before planning (default: the library's MI355X table for the "
                         "bench shapes, written by --tune --tune-save)")
    ap.add_argument("--no-tune-table", action="store_true", help="plan with the built-in rules only")
    ap.add_argument("--ablation", action="store_true",
                    help="only measure direct-to-register vs LDS write-back of the dequantized weights")
    ap.add_argument("--ablation-only", default="", metavar="K,N,M",
                    help="with --ablation: one shape, 5 launches per mode (for counter runs)")
    ap.add_argument("--ingest-waits", metavar="COUNTER_CSV",
                    help="write the wave-state table (profiles/wave_states_*.md) from a rocprofv3 --pmc CSV of "
                         "WAIT_COUNTERS over --steps 1 --warmup 0")
    ap.add_argument("--ingest-mfma", metavar="COUNTER_CSV",
                    help="per-GEMM matrix-core utilisation from a rocprofv3 --pmc run of MFMA_COUNTERS")
    ap.add_argument("--mfma-out", default=os.path.join(ROOT, "profiles", "mfma_util_bench_llama2_7b_70b.md"))
    ap.add_argument("--trace-log", default="", help="with --ingest-trace: stdout of the profiled bench run")
    ap.add_argument("--ingest-trace", metavar="KERNEL_TRACE_CSV",
                    help="per-GEMM kernel durations from a rocprofv3 --kernel-trace run of this script")
    ap.add_argument("--trace-out", default=os.path.join(ROOT, "profiles", "bench_llama2_7b_70b_kernel_trace.md"))
    ap.add_argument("--trace-command", default="rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o kt "
                    "-- python3 <repo>/bench.py --steps 5 --warmup 2 --no-cpu-baseline")
    args = ap.parse_args()

    if args.tune_table and not args.no_tune_table and not args.tune:
        import paper_2402_10076_amd as Q
        Q.tune_table_load(args.tune_table)

    if args.ingest_trace or args.ingest_pmc:
        args.dominant = args.dominant or dominant_kernel(args.points_out, "tiled_kernel<128,32>")
    if args.ingest_trace:
        import paper_2402_10076_amd as Q
        import workloads as W
        points = build_points([int(c) for c in args.configs.split(",") if c])
        for p in points:
            p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
            p["kernel"] = kernel_name(p["sel"])
            p["bytes"] = W.alg_bytes(p["M"], p["N"], p["K"])
            p["flops"] = W.flops(p["M"], p["N"], p["K"])
        print("dominant %s mean kernel duration %.2f us" % (
            args.dominant, ingest_trace(args.ingest_trace, points, args.dominant, args.trace_out, args.trace_command,
                                        args.trace_log)))
        return

    if args.ingest_waits:
        import paper_2402_10076_amd as Q
        points = build_points([int(c) for c in args.configs.split(",") if c])
        for p in points:
            p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
            p["kernel"] = kernel_name(p["sel"])
        cmd = ("rocprofv3 --pmc " + " ".join(WAIT_COUNTERS) + " --output-format csv -d <dir> -o sq "
               "-- python3 <repo>/bench.py --steps 1 --warmup 0 --no-cpu-baseline")
        print("%d repetitions ingested into %s" % (ingest_waits(args.ingest_waits, points, WAITS_MD, cmd), WAITS_MD))
        return

    if args.ingest_mfma:
        import paper_2402_10076_amd as Q
        import workloads as W
        points = build_points([int(c) for c in args.configs.split(",") if c])
        for p in points:
            p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
            p["kernel"] = kernel_name(p["sel"])
            p["flops"] = W.flops(p["M"], p["N"], p["K"])
        cmd = ("rocprofv3 --pmc " + " ".join(MFMA_COUNTERS) + " --output-format csv -d <dir> -o m "
               "-- python3 <repo>/bench.py --steps 1 --warmup 0 --no-cpu-baseline")
        print("%d repetitions ingested into %s" % (ingest_mfma(args.ingest_mfma, points, args.mfma_out, cmd),
                                                   args.mfma_out))
        return

    if args.ingest_pmc:
        import paper_2402_10076_amd as Q
        points = build_points([int(c) for c in args.configs.split(",") if c])
        import workloads as W
        for p in points:
            p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
            p["kernel"] = kernel_name(p["sel"])
            p["bytes"] = W.alg_bytes(p["M"], p["N"], p["K"])
        t = ingest_pmc(*args.ingest_pmc, points, args.dominant, command=PMC_COMMANDS)
        os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(t, f, indent=1)
        print(json.dumps(t))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU path only: the library runs on one MI355X "
              "(--gpus 1); multi-GPU runs are not implemented.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2402_10076_amd as Q
    import workloads as W

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.ablation:
        if args.ablation_only:
            K, N, M = (int(v) for v in args.ablation_only.split(","))
            rows = ablation([(K, N, [M])], reps=5)
        else:
            rows = ablation([(8192, 8192, [16, 64, 256, 1024]), (8192, 57344, [256, 1024]),
                             (28672, 8192, [256, 1024]), (4096, 4096, [256])])
        print(json.dumps({"ablation": "direct-to-register vs LDS write-back (64x256 tiles)", "rows": rows}))
        return
    if args.moe:
        print(json.dumps({"moe": "Mixtral-8x7B expert FFN, dense per expert vs grouped", **moe(sweep=not args.moe_auto_only)}))
        return
    if args.read_ceiling:
        print(json.dumps({"read_ceiling": "device-to-device copies rotating >= 1 GiB, graph of 40",
                          "rows": read_ceiling()}))
        return
    if args.compare_fp16:
        ck, cn = (int(v) for v in args.compare_shape.split(","))
        rows = compare_fp16(ck, cn, [int(m) for m in args.compare_m.split(",") if m])
        print(json.dumps({"compare": "w4a16 vs fp16 hipBLASLt", "K": ck, "N": cn, "rows": rows}))
        return
    Q.lib()  # raises if the HIP library is not built

    configs = [int(c) for c in args.configs.split(",") if c]
    points = build_points(configs)
    dev = torch.device("cuda:0")

    # ---- inputs: generate, pack (untimed, host), upload one weight copy per point
    t_setup = time.perf_counter()
    xs = {}
    for p in points:
        key = (p["cid"], p["si"])
        if key not in xs:
            cfg = W.CONFIGS[p["cid"]]
            sh = cfg.shapes[p["si"]]
            log("setup C%d %s K=%d N=%d" % (p["cid"], sh.name, sh.K, sh.N))
            q, z, s = W.draw_weights(p["cid"], p["si"], sh.K, sh.N)
            pw, ps, pz = Q.pack_weights(q, z, s)
            del q, z, s
            base = Q.to_device(pw, ps, pz, dev)
            del pw, ps, pz
            x = W.draw_x(p["cid"], p["si"], max(sh.Ms), sh.K, cfg.outliers)
            xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.float16)
            xs[key] = (xd, base)
        xd, base = xs[key]
        p["w"] = tuple(t.clone() for t in base)
        p["x"] = xd[:p["M"]]
        p["y"] = torch.empty((p["M"], p["N"]), dtype=torch.float16, device=dev)
        if args.tune:
            Q.tune(p["x"], *p["w"], p["N"], y=p["y"])
        p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
        p["kernel"] = kernel_name(p["sel"])
        p["flops"] = W.flops(p["M"], p["N"], p["K"])
        p["bytes"] = W.alg_bytes(p["M"], p["N"], p["K"])
    xs.clear()
    torch.cuda.synchronize()
    if args.tune and args.tune_save:
        Q.tune_table_save(args.tune_save)
    log("setup %.1f s, %d GEMMs per step, %.2f GB of packed weights on device" % (
        time.perf_counter() - t_setup, len(points),
        sum(sum(t.numel() * t.element_size() for t in p["w"]) for p in points) / 1e9))

    def step(evs=None):
        for i, p in enumerate(points):
            if evs is not None:
                evs[i][0].record()
            Q.w4a16_gemm(p["x"], *p["w"], p["N"], y=p["y"])
            if evs is not None:
                evs[i][1].record()

    # Warm up eagerly on the stream the step is captured on: the library's
    # per-stream split-K / stream-K workspace then exists before capture, so
    # the captured step allocates nothing.
    cap_stream = torch.cuda.Stream()
    with torch.cuda.stream(cap_stream):
        for _ in range(max(1, args.warmup)):
            step()
    cap_stream.synchronize()
    eager_y = [p["y"].clone() for p in points]

    # One step as a HIP graph: replaying it issues the 44 GEMMs without the
    # host's per-launch overhead (the decode-style small-M GEMMs are shorter
    # than a Python-level launch).  The replay must reproduce the eager
    # outputs bit for bit (every kernel is deterministic).
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap_stream):
        step()
    for p in points:
        p["y"].zero_()
    graph.replay()
    torch.cuda.synchronize()
    bad = [i for i, p in enumerate(points) if not torch.equal(p["y"], eager_y[i])]
    if bad:
        raise SystemExit("graph replay differs from the eager step for GEMMs %s" % bad)
    del eager_y
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()

    # ---- timed region: K steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # ---- per-GEMM times: eager steps with HIP events around every GEMM on
    # the warmed-up launch stream (its split-K / stream-K workspace already
    # exists, so no interval holds an allocation); a GPU-side wait at the
    # start of each step lets the host enqueue the whole step first, so the
    # intervals hold GPU time only
    psteps = max(3, min(args.steps, 10))
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in points] for _ in range(psteps)]
    with torch.cuda.stream(cap_stream):
        for s_ in range(psteps):
            torch.cuda._sleep(40_000_000)  # ~20 ms: the host enqueues all 44 GEMMs with their events first
            step(evs[s_])
    torch.cuda.synchronize()

    for i, p in enumerate(points):
        p["ms"] = float(np.mean([evs[s_][i][0].elapsed_time(evs[s_][i][1]) for s_ in range(psteps)]))
        p["tflops"] = p["flops"] / (p["ms"] * 1e-3) / 1e12
        p["gbs"] = p["bytes"] / (p["ms"] * 1e-3) / 1e9
        p["frac_hbm"] = p["gbs"] / HBM_PEAK_GBS
        p["frac_mfma"] = p["tflops"] / MFMA_F16_PEAK_TFLOPS
        p["bound"] = "hbm" if p["bytes"] / HBM_PEAK_GBS >= p["flops"] / 1e3 / MFMA_F16_PEAK_TFLOPS else "mfma"
        p["frac_roof"] = p["frac_hbm"] if p["bound"] == "hbm" else p["frac_mfma"]

    log("%-4s %-8s %6s %6s %6s %-34s %9s %8s %8s %6s %6s" % (
        "cfg", "shape", "K", "N", "M", "kernel", "us", "TFLOP/s", "GB/s", "fHBM", "fMFMA"))
    for p in points:
        log("C%-3d %-8s %6d %6d %6d %-34s %9.2f %8.1f %8.0f %6.3f %6.3f" % (
            p["cid"], p["shape"], p["K"], p["N"], p["M"], p["kernel"], p["ms"] * 1e3, p["tflops"],
            p["gbs"], p["frac_hbm"], p["frac_mfma"]))

    tot_flops = sum(p["flops"] for p in points)
    tot_bytes = sum(p["bytes"] for p in points)
    ms_per_step = elapsed / args.steps * 1e3

    def graph_time_ms(pts, reps):
        """Per-replay time of a HIP graph holding the given GEMMs of the step
        (each with its own weight copy), from HIP events around `reps`
        replays on the launch stream: kernel time plus the graph's own
        back-to-back launch gaps, with no per-GEMM event packets."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap_stream):
            for p in pts:
                Q.w4a16_gemm(p["x"], *p["w"], p["N"], y=p["y"])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(cap_stream):
            g.replay()
            e0.record()
            for _ in range(reps):
                g.replay()
            e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    # dominant kernel: the kernel (by name) with the most event time per step;
    # its roofline is timed on a graph of just its launches
    by_k = {}
    for p in points:
        by_k.setdefault(p["kernel"], []).append(p)
    dom = max(by_k, key=lambda k: sum(p["ms"] for p in by_k[k]))
    dpts = by_k[dom]
    reps = max(3, args.steps)
    d_ms = graph_time_ms(dpts, reps)
    d_bound = "mfma" if all(p["bound"] == "mfma" for p in dpts) else "hbm"
    if d_bound == "mfma":
        ach = sum(p["flops"] for p in dpts) / (d_ms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(ach, 2), peak=MFMA_F16_PEAK_TFLOPS, unit="TFLOP/s",
                    frac=round(ach / MFMA_F16_PEAK_TFLOPS, 4), traffic=None)
    else:
        ach = sum(p["bytes"] for p in dpts) / (d_ms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(ach, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(ach / HBM_PEAK_GBS, 4), traffic=None)
    roof["traffic"] = stored_traffic(dom)
    # the counters cannot run inside the timed bench: the figure is the stored
    # rocprofv3 FETCH_SIZE + WRITE_SIZE measurement of this kernel source
    roof["traffic_source"] = ("stored rocprofv3 FETCH_SIZE+WRITE_SIZE per launch, copy-calibrated, "
                              "profiles/traffic_bench_llama2_7b_70b.json (same kernel source hash)"
                              if roof["traffic"] is not None else "no counter run for this kernel source")
    roof["kernel"] = dom
    roof["launches_per_step"] = len(dpts)
    roof["avg_launch_us"] = round(d_ms * 1e3 / len(dpts), 2)
    roof["alg_bytes_per_launch"] = int(round(np.mean([p["bytes"] for p in dpts])))
    roof["alg_flops_per_launch"] = int(round(np.mean([p["flops"] for p in dpts])))

    small = [p for p in points if p["M"] <= 16]
    s_ms = graph_time_ms(small, reps) if small else 0.0
    s_gbs = sum(p["bytes"] for p in small) / (s_ms * 1e-3) / 1e9 if small else 0.0
    big = [p for p in points if p["M"] >= 256]
    b_ms = graph_time_ms(big, reps) if big else 0.0
    b_tf = sum(p["flops"] for p in big) / (b_ms * 1e-3) / 1e12 if big else 0.0

    out = {
        "metric": METRIC,
        "value": round(tot_flops * args.steps / elapsed / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "W4A16 g128 decoder-linear GEMMs: Llama-2-7B (K,N) in {(4096,12288),(4096,4096),"
                        "(4096,22016),(11008,4096)} x M in {1,4,16,64,128,256} and Llama-2-70B "
                        "{(8192,10240),(8192,8192),(8192,57344),(28672,8192)} x M in {1,16,128,512,1024}",
            "gemms_per_step": len(points),
            "group": 128,
            "weights": "uint4 q, uint4 zero, fp16 scale per 128 input channels; one packed copy per GEMM",
        },
        "hbm_gbps": round(tot_bytes * args.steps / elapsed / 1e9, 1),
        "timing": "K replays of a HIP graph of the step; per-GEMM times from HIP events in eager steps",
        "plan": ("autotuned at setup" if args.tune else
                 "built-in rules" if args.no_tune_table or not args.tune_table else
                 "tune table " + os.path.basename(args.tune_table)),
        "events_ms_per_step": round(sum(p["ms"] for p in points), 4),
        "roofline": roof,
        "roofline_small_m": dict(bound="hbm", achieved=round(s_gbs, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                                 frac=round(s_gbs / HBM_PEAK_GBS, 4), points=len(small),
                                 scope="all GEMMs with M<=16, replayed as one graph"),
        "mfma_large_m": dict(achieved=round(b_tf, 2), peak=MFMA_F16_PEAK_TFLOPS, unit="TFLOP/s",
                             frac=round(b_tf / MFMA_F16_PEAK_TFLOPS, 4), points=len(big),
                             scope="all GEMMs with M>=256, replayed as one graph"),
    }

    if not args.no_cpu_baseline:
        # every core this process may run on, unless the host sets a smaller
        # CPU share for it (OMP_NUM_THREADS)
        affinity = len(os.sched_getaffinity(0))
        share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
        threads = min(affinity, share) if share > 0 else affinity
        log("cpu baseline: oracle on %d threads, %.4f of the columns of every GEMM" % (
            threads, args.cpu_col_fraction))
        fl, t, t_full = cpu_baseline(points, threads, args.cpu_col_fraction)
        out["cpu_baseline"] = {
            "value": round(fl / t / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "affinity_cores": affinity,
            "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS", ""),
            "sample": "every GEMM of the step, all rows, a seeded sample of ceil(N/%d) columns "
                      "(%.1f GFLOP in %.1f s)" % (round(1 / args.cpu_col_fraction), fl / 1e9, t),
            "step_s_extrapolated": round(t_full, 1),
            "c1_16x512x512_one_thread_s": round(cpu_c1_one_thread(), 4),
        }

    if args.points_out:
        with open(args.points_out, "w") as f:
            json.dump([{k: v for k, v in p.items() if k not in ("w", "x", "y")} for p in points], f, indent=1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
