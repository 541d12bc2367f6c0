"""GEMMs captured in a HIP graph replay the eager results bit for bit.

Every kernel path (stream kernel, tiled data-parallel, split-K with its
reduction kernel, stream-K and the sliced stream kernel with their arrival
counters; the grouped GEMM's
two-launch plan and a fused epilogue) is captured after an
eager warm-up on the capture stream (so the library's per-stream workspace
exists and the capture allocates nothing).  The graph is replayed several
times with unrelated eager work and synchronizations in between, and every
replay is compared with the eager outputs.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, to_dev_x

pytestmark = pytest.mark.gpu

CASES = [  # (M, K, N, cfg)
    (1, 1024, 272, None),                                               # stream kernel
    (48, 1024, 528, dict(variant=2, tile_m=32, tile_n=16, split_k=2)),  # split-K + reduction
    (300, 2304, 528, dict(variant=3, tile_m=64, tile_n=32, split_k=24)),  # stream-K
    (256, 1024, 512, dict(variant=2, tile_m=128, tile_n=32, split_k=1)),  # data-parallel
    (16, 6144, 528, dict(variant=5, split_k=3, tile_n=1)),              # sliced stream, last-arriver sum
]


def test_graph_replay_matches_eager():
    side = torch.cuda.Stream()
    jobs = []
    for i, (M, K, N, cfg) in enumerate(CASES):
        x, q, z, s = rand_case(300 + i, M, K, N)
        p = Packed(q, z, s)
        xd = to_dev_x(x)
        y = torch.empty((M, N), dtype=torch.float16, device="cuda")
        jobs.append((p, xd, y, Q.make_config(**cfg) if cfg else None))

    def run_all():
        for p, xd, y, cfg in jobs:
            p.gemm(xd, cfg=cfg, y=y)

    with torch.cuda.stream(side):
        run_all()
    side.synchronize()
    eager = [y.clone() for _, _, y, _ in jobs]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        run_all()

    other_x, oq, oz, os_ = rand_case(999, 64, 1024, 256)
    other = Packed(oq, oz, os_)
    for rep in range(4):
        for _, _, y, _ in jobs:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (_, _, y, _) in enumerate(jobs):
            assert torch.equal(y, eager[i]), "replay %d differs from eager for case %d" % (rep, i)
        # unrelated eager work between replays (same library, default stream)
        other.gemm(to_dev_x(other_x), cfg=Q.make_config(variant=2, tile_m=32, tile_n=16, split_k=4))
        torch.cuda.synchronize()


def test_graph_replay_grouped_and_fused():
    """The grouped GEMM's automatic two-launch plan (128-row tiles, then
    32-row tiles over short remainders, both stream-K) and a fused gated
    epilogue, captured together after an eager warm-up and replayed with
    eager work in between: every replay equals the eager outputs."""
    side = torch.cuda.Stream()
    g_np = np.random.Generator(np.random.PCG64(41))
    T, K, N, E = 300, 512, 256, 4
    experts = []
    for _ in range(E):
        experts.append((g_np.integers(0, 16, (K, N), dtype=np.uint8),
                        g_np.integers(0, 16, (K // 128, N), dtype=np.uint8),
                        g_np.uniform(0.002, 0.02, (K // 128, N)).astype(np.float16).view(np.uint16)))
    counts = [131, 149, 100, 128]
    rows = torch.from_numpy(np.concatenate([np.sort(g_np.integers(0, T, c)) for c in counts]).astype(np.int32)).cuda()
    offsets = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)).cuda()
    R = int(sum(counts))
    assert Q.grouped_select_config(R, E, N, K)["tile_m"] == 128
    dw, ds, dz = Q.to_device(*Q.pack_experts(experts))
    x = to_dev_x(rand_case(42, T, K, 16)[0])
    yg = torch.empty((R, N), dtype=torch.float16, device="cuda")
    xf, qf, zf, sf = rand_case(43, 40, 640, 96)
    pf = Packed(qf, zf, sf)
    xfd = to_dev_x(xf)
    yf = torch.empty((40, 48), dtype=torch.float16, device="cuda")

    def run_all():
        Q.grouped_gemm(x, offsets, dw, ds, dz, N, rows=rows, y=yg)
        Q.gemm_fused(xfd, pf.dw, pf.ds, pf.dz, 96, activation=Q.ACT_SILU_GATE, y=yf)

    with torch.cuda.stream(side):
        run_all()
    side.synchronize()
    eager = [yg.clone(), yf.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        run_all()
    for rep in range(3):
        yg.fill_(float("nan"))
        yf.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(yg, eager[0]) and torch.equal(yf, eager[1]), "replay %d differs" % rep
        Q.grouped_gemm(x, offsets, dw, ds, dz, N, rows=rows, cfg=Q.make_config(variant=2, split_k=2, tile_m=32,
                                                                               tile_n=16))
        torch.cuda.synchronize()


def test_capture_without_workspace_returns_status():
    """A first call on a fresh stream under capture, whose plan needs the
    internal workspace, returns QUICK_ERR_CAPTURE and enqueues nothing (no
    allocation, clear or synchronization on the capturing stream); after
    an eager warm-up the same call captures and replays.  A graph captured
    earlier keeps working after a larger plan grows the stream's buffer
    (the old buffer is retired, not freed)."""
    side = torch.cuda.Stream()
    M, K, N = 48, 1024, 2048
    x, q, z, s = rand_case(500, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=2, tile_m=32, tile_n=16, split_k=2)   # split-K: workspace needed
    assert Q.workspace_bytes(M, N, K, cfg) > 0
    y = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda")
    marker = torch.zeros(4, device="cuda")
    torch.cuda.synchronize()
    g0 = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g0, stream=side):
        marker.fill_(1.0)
        try:
            p.gemm(xd, cfg=cfg, y=y)
        except Q.QuickError as e:
            status = e.status
    assert status == Q.QUICK_ERR_CAPTURE
    g0.replay()
    torch.cuda.synchronize()
    assert bool((marker == 1.0).all()) and bool((y == 7.0).all()), "the refused call left work in the graph"

    with torch.cuda.stream(side):
        p.gemm(xd, cfg=cfg, y=y)
    side.synchronize()
    eager = y.clone()
    g1 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g1, stream=side):
        p.gemm(xd, cfg=cfg, y=y)
    y.fill_(float("nan"))
    torch.cuda.synchronize()
    g1.replay()
    torch.cuda.synchronize()
    assert torch.equal(y, eager)

    # a larger plan on the same stream: refused under capture, grows the
    # buffer eagerly; the graph captured with the old buffer still replays
    big = Q.make_config(variant=2, tile_m=32, tile_n=16, split_k=8)
    # more than the first allocation (at least 1 MiB) holds
    assert Q.workspace_bytes(M, N, K, big) > max(Q.workspace_bytes(M, N, K, cfg), 1 << 20)
    yb = torch.empty_like(y)
    g2 = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g2, stream=side):
        marker.fill_(2.0)
        try:
            p.gemm(xd, cfg=big, y=yb)
        except Q.QuickError as e:
            status = e.status
    assert status == Q.QUICK_ERR_CAPTURE
    with torch.cuda.stream(side):
        p.gemm(xd, cfg=big, y=yb)
    side.synchronize()
    assert rel_err(from_dev_y(yb), oracle.gemm(x, q, z, s)) <= TOL
    for _ in range(3):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g1.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, eager)
