"""The write-back ablation (quick_ablation_gemm): the dequantized weights
taken through an LDS tile (padded or unpadded rows) give exactly the results
of the direct-to-register path, which matches the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, to_dev_x

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,N", [(65, 640, 528), (1, 384, 80), (130, 1152, 256)])
def test_write_back_modes_match_direct_path(M, K, N):
    x, q, z, s = rand_case(800 + M, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    ys = [from_dev_y(Q.ablation_gemm(xd, p.dw, p.ds, p.dz, N, mode)) for mode in (0, 1, 2)]
    torch.cuda.synchronize()
    assert rel_err(ys[0], oracle.gemm(x, q, z, s)) <= TOL
    assert np.array_equal(ys[1], ys[0]) and np.array_equal(ys[2], ys[0])
    # mode 0 is the library's 64 x 32 tiled kernel
    y_lib = from_dev_y(p.gemm(xd, cfg=Q.make_config(variant=2, tile_m=64, tile_n=32, split_k=1)))
    assert np.array_equal(y_lib, ys[0])


def test_bad_mode_rejected():
    x, q, z, s = rand_case(1, 16, 256, 32)
    p = Packed(q, z, s)
    with pytest.raises(Q.QuickError):
        Q.ablation_gemm(to_dev_x(x), p.dw, p.ds, p.dz, 32, 3)
