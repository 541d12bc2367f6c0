"""CPU checks of the profile ingestion in bench.py: synthetic rocprofv3 CSVs
laid out like the profiler's (a kernel trace; one counter pass) are mapped
back onto the bench step's launch sequence, and every GEMM gets exactly the
values planted for it, including split-K launches with their reduction pass
and the runtime's and torch's kernels interleaved."""
import csv
import os
import re

import numpy as np
import pytest

import bench
import paper_2402_10076_amd as Q
import workloads as W

TRACE_FIELDS = ["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id", "Kernel_Id", "Kernel_Name",
                "Correlation_Id", "Start_Timestamp", "End_Timestamp", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
                "Accum_VGPR_Count", "SGPR_Count", "Workgroup_Size_X", "Workgroup_Size_Y", "Workgroup_Size_Z",
                "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z"]
PMC_FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
              "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
              "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


@pytest.fixture(scope="module")
def points():
    Q.tune_table_load(os.path.join(os.path.dirname(Q.LIB_PATH), "tune_mi355x.txt"))
    try:
        pts = bench.build_points([2, 5])
        for p in pts:
            p["sel"] = Q.select_config(p["M"], p["N"], p["K"])
            p["kernel"] = bench.kernel_name(p["sel"])
            p["bytes"] = W.alg_bytes(p["M"], p["N"], p["K"])
            p["flops"] = W.flops(p["M"], p["N"], p["K"])
        yield pts
    finally:
        Q.tune_table_clear()


def _symbol(prefix):
    """A full kernel name as the profiler prints it, from a launch prefix."""
    if prefix == "splitk_reduce_kernel":
        return "(anonymous namespace)::splitk_reduce_kernel(float const*, unsigned short*, long, int, int, quick::Epi)"
    return "void (anonymous namespace)::%s(unsigned short const*, unsigned int __vector(4) const*)" % (
        prefix if prefix.endswith(">") else prefix + "1, 1, 4, 8, true>")


def _dispatches(points, reps):
    """(kernel name, point index or None, planted value) per dispatch: the
    step's launches `reps` times, with runtime copies and torch kernels in
    between, as a bench run dispatches them."""
    seq = bench.launch_sequence(points)
    owner = bench.launch_points(points)
    out = [("__amd_rocclr_copyBuffer", None, 3.0)]
    for rep in range(reps):
        out.append(("void at::native::vectorized_elementwise_kernel<8, at::native::FillFunctor<c10::Half>>", None, 1.0))
        for j, (_, prefix) in enumerate(seq):
            i = owner[j]
            # value: point index + 10, reduction passes 0.5, repetition offset
            v = 0.5 if prefix == "splitk_reduce_kernel" else i + 10.0 + 0.25 * rep
            out.append((_symbol(prefix), i, v))
    return out


def test_trace_ingest_maps_every_gemm(points, tmp_path):
    reps = 3
    rows = []
    t = 1000
    for d, (name, _, v) in enumerate(_dispatches(points, reps), start=1):
        dur = int(round(v * 1000))
        rows.append({"Kind": "KERNEL_DISPATCH", "Dispatch_Id": d, "Kernel_Name": name, "Start_Timestamp": t,
                     "End_Timestamp": t + dur})
        t += dur + 100
    path = tmp_path / "kt_kernel_trace.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=TRACE_FIELDS, restval="0")
        w.writeheader()
        w.writerows(rows)
    out = tmp_path / "trace.md"
    dominant = "tiled_kernel<128,32>"
    dom_us = bench.ingest_trace(str(path), points, dominant, str(out), "cmd")
    text = out.read_text()
    assert "%d repetitions" % reps in text
    table = [l for l in text.splitlines() if l.startswith("| C")]
    assert len(table) == len(points)
    for i, (p, line) in enumerate(zip(points, table)):
        cells = [c.strip() for c in line.strip("|").split("|")]
        assert cells[5] == p["kernel"]
        red = 0.5 if (p["sel"]["variant"] in (2, 6) and p["sel"]["split_k"] > 1) else 0.0
        mean = np.mean([i + 10.0 + 0.25 * r for r in range(reps)]) + red
        assert abs(float(cells[6]) - mean) < 0.006, (p["kernel"], cells[6], mean)
        assert abs(float(cells[7]) - (i + 10.0 + red)) < 0.006
    dom = [i for i, p in enumerate(points) if p["kernel"] == dominant]
    assert dom and abs(dom_us - np.mean([i + 10.0 + 0.25 * r for i in dom for r in range(reps)])) < 1e-6


def test_counter_ingest_maps_every_gemm(points, tmp_path):
    reps = 2
    rows = []
    for d, (name, i, v) in enumerate(_dispatches(points, reps), start=1):
        for c in ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY"):
            rows.append({"Dispatch_Id": d, "Kernel_Name": name, "Counter_Name": c,
                         "Counter_Value": 1000.0 if c == "SQ_WAVE_CYCLES" else 10.0 * v,
                         "Start_Timestamp": 0, "End_Timestamp": 1000})
    path = tmp_path / "c_counter_collection.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=PMC_FIELDS, restval="0")
        w.writeheader()
        w.writerows(rows)
    got_reps, acc, _ = bench.gemm_counters(str(path), points, ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY"))
    assert got_reps == reps
    for i, p in enumerate(points):
        # the GEMM kernel's own dispatch, never its reduction pass
        assert acc[i]["SQ_WAIT_ANY"] == [10.0 * (i + 10.0 + 0.25 * r) for r in range(reps)], p["kernel"]


def test_launch_sequence_names_and_reduction_passes(points):
    seq = bench.launch_sequence(points)
    owner = bench.launch_points(points)
    assert len(seq) == len(owner)
    split = [i for i, p in enumerate(points) if p["sel"]["variant"] in (2, 6) and p["sel"]["split_k"] > 1]
    assert len(seq) == len(points) + len(split)
    assert sum(1 for _, pre in seq if pre == "splitk_reduce_kernel") == len(split)
    for (name, pre), i in zip(seq, owner):
        if name is not None:
            assert name == points[i]["kernel"]
            assert re.match(r"(stream_kernel<|kstream_kernel<\d>|tiled(32)?_kernel<\d+, \d+)", pre)
