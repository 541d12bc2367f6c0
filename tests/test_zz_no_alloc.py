"""The allocation-free entry point (quick_w4a16_gemm_noalloc) through the C
ABI against quick_w4a16_gemm_ex with the same automatic plan: bit-identical
outputs, and within tolerance of the oracle, on two calls in a row (the
second with a smaller input) for every kind of plan that uses a workspace
(split-K partial sums, stream-K partial tiles, the sliced kernel's partial
columns) and one that uses none."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu

# (K, N, M first call, M second call): the automatic plan of each shape
CASES = [
    (4096, 4096, 64, 40),      # tiled split-K: fp32 partials + reduction
    (6144, 16384, 256, 200),   # tiled stream-K: arrival counters + partial tiles
    (4096, 8192, 16, 12),      # sliced stream kernel, several K slices
    (1024, 272, 3, 1),         # stream kernel: no workspace
]


def _kind(sel):
    return {1: "stream", 2: "tiled", 3: "stream-K", 5: "sliced"}[sel["variant"]]


@pytest.mark.parametrize("K,N,M1,M2", CASES)
def test_noalloc_matches_ex_on_consecutive_calls(K, N, M1, M2):
    x, q, z, s = rand_case(K + N + M1, M1, K, N)
    p = Packed(q, z, s)
    for M in (M1, M2):
        sel = Q.select_config(M, N, K)
        need = Q.workspace_bytes(M, N, K)
        say("noalloc K=%d N=%d M=%d plan=%s (%s) workspace=%d" % (K, N, M, sel, _kind(sel), need))
        assert need <= Q.SCRATCH_BYTES
        xd = to_dev_x(x[:M])
        y_ex = torch.empty((M, N), dtype=torch.float16, device="cuda")
        ws = torch.zeros(max(need, 16) // 4 + 4, dtype=torch.int32, device="cuda")
        Q.w4a16_gemm(xd, p.dw, p.ds, p.dz, N, y=y_ex, cfg=Q.make_config(), workspace=ws)
        y_na = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
        Q.w4a16_gemm_noalloc(xd, p.dw, p.ds, p.dz, N, y_na)
        torch.cuda.synchronize()
        a, b = from_dev_y(y_na), from_dev_y(y_ex)
        assert np.array_equal(a, b), "noalloc differs from the _ex call at %d entries" % int((a != b).sum())
        # the oracle on every row and one column of every n-tile (rotating position)
        t = np.arange(N // 16)
        cols = 16 * t + (t % 16)
        assert rel_err(a[:, cols], oracle.gemm(x[:M], q, z, s, cols=cols)) <= TOL


def test_noalloc_repeated_calls_and_capture():
    """The scratch counters are left zero: ten calls in a row give the same
    bits, also when the calls are captured in a graph and replayed."""
    K, N, M = 6144, 16384, 256         # stream-K: counters and partial tiles in the scratch array
    x, q, z, s = rand_case(91, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    Q.w4a16_gemm_noalloc(xd, p.dw, p.ds, p.dz, N, y)
    torch.cuda.synchronize()
    first = y.clone()
    for _ in range(10):
        Q.w4a16_gemm_noalloc(xd, p.dw, p.ds, p.dz, N, y)
    torch.cuda.synchronize()
    assert torch.equal(y, first)
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):          # nothing to allocate: captures on a fresh stream
        Q.w4a16_gemm_noalloc(xd, p.dw, p.ds, p.dz, N, y)
    for _ in range(3):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, first)
        Q.w4a16_gemm_noalloc(xd[:7], p.dw, p.ds, p.dz, N, torch.empty((7, N), dtype=torch.float16, device="cuda"))
        torch.cuda.synchronize()
