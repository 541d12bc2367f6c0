"""quick_tune: times the configurations of a shape (rotating through copies of
the caller's weights), records the fastest, and the automatic path then uses it."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, to_dev_x

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,N", [(1, 2048, 272), (48, 1024, 528), (300, 2304, 528)])
def test_tune_records_fastest_and_auto_uses_it(M, K, N):
    Q.tune_table_clear()
    try:
        x, q, z, s = rand_case(700 + M, M, K, N)
        p = Packed(q, z, s)
        xd = to_dev_x(x)
        y = torch.empty((M, N), dtype=torch.float16, device="cuda")
        best = Q.tune(xd, p.dw, p.ds, p.dz, N, y=y)
        torch.cuda.synchronize()
        ref = oracle.gemm(x, q, z, s)
        assert rel_err(from_dev_y(y), ref) <= TOL          # y holds the chosen config's result
        assert Q.tune_table_size() == 1
        sel = Q.select_config(M, N, K)
        assert sel["variant"] == best["variant"] and sel["tile_n"] == best["tile_n"]
        y_auto = from_dev_y(p.gemm(xd))                     # automatic path -> tuned config
        y_cfg = from_dev_y(p.gemm(xd, cfg=Q.make_config(**best)))
        assert np.array_equal(y_auto, y_cfg)
        assert rel_err(y_auto, ref) <= TOL
    finally:
        Q.tune_table_clear()


def test_tune_refused_under_capture():
    """quick_tune allocates and synchronizes: on a capturing stream it
    returns QUICK_ERR_CAPTURE and records nothing."""
    Q.tune_table_clear()
    M, K, N = 16, 1024, 272
    x, q, z, s = rand_case(801, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    marker = torch.zeros(4, device="cuda")
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g, stream=side):
        marker.fill_(1.0)
        try:
            Q.tune(xd, p.dw, p.ds, p.dz, N, y=y)
        except Q.QuickError as e:
            status = e.status
    assert status == Q.QUICK_ERR_CAPTURE
    assert Q.tune_table_size() == 0
    g.replay()
    torch.cuda.synchronize()
    assert bool((marker == 1.0).all())
