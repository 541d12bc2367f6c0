"""GEMMs captured in a HIP graph replay the eager results bit for bit.

Every kernel path (stream kernel, tiled data-parallel, split-K with its
reduction kernel, stream-K with its arrival counters) is captured after an
eager warm-up on the capture stream (so the library's per-stream workspace
exists and the capture allocates nothing).  The graph is replayed several
times with unrelated eager work and synchronizations in between, and every
replay is compared with the eager outputs.
"""
import numpy as np
import pytest
import torch

import paper_2402_10076_amd as Q
from gpu_util import Packed, rand_case, to_dev_x

pytestmark = pytest.mark.gpu

CASES = [  # (M, K, N, cfg)
    (1, 1024, 272, None),                                               # stream kernel
    (48, 1024, 528, dict(variant=2, tile_m=32, tile_n=16, split_k=2)),  # split-K + reduction
    (300, 2304, 528, dict(variant=3, tile_m=64, tile_n=32, split_k=24)),  # stream-K
    (256, 1024, 512, dict(variant=2, tile_m=128, tile_n=32, split_k=1)),  # data-parallel
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
