"""The five workload configurations at full size, on the launch
configuration the benchmark times (automatic kernel choice), against the
oracle on sampled outputs: all rows up to 64 (else 64 sampled rows) and 256
sampled columns (the first 64, the last 64 and 128 random ones), every
(shape, M) point.  Inputs come from workloads.py with the configurations'
seeds and distributions."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import TOL, Packed, from_dev_y, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu


def _check_point(tag, p, x, q, z, s, M):
    xd = to_dev_x(x)
    y = from_dev_y(p.gemm(xd))
    rows = W.sample_rows(M)
    cols = W.sample_columns(p.N, 256)
    ref = oracle.gemm(x[rows], q, z, s, cols=cols)
    err = rel_err(y[np.ix_(rows, cols)], ref)
    say("%s M=%d rel_err=%.3g" % (tag, M, err))
    assert err <= TOL, "%s M=%d: rel err %.3g" % (tag, M, err)


@pytest.mark.parametrize("cid", [2, 3, 5])
def test_llama_config(cid):
    cfg = W.CONFIGS[cid]
    for si, sh in enumerate(cfg.shapes):
        say("C%d %s K=%d N=%d: generating" % (cid, sh.name, sh.K, sh.N))
        x_all = W.draw_x(cid, si, max(sh.Ms), sh.K, cfg.outliers)
        q, z, s = W.draw_weights(cid, si, sh.K, sh.N)
        p = Packed(q, z, s)
        for M in sh.Ms:
            _check_point("C%d %s" % (cid, sh.name), p, x_all[:M], q, z, s, M)
        del p
        torch.cuda.empty_cache()


def test_mixtral_experts():
    routes = W.mixtral_routing()
    assert sum(len(r) for r in routes) == W.MIXTRAL_TOKENS * W.MIXTRAL_TOPK
    xt = W.mixtral_tokens()
    for e in range(W.MIXTRAL_EXPERTS):
        Me = len(routes[e])
        for which, name in enumerate(("w1", "w3", "w2")):
            q, z, s = W.mixtral_expert_weights(e, which)
            x = xt[routes[e]] if which < 2 else W.mixtral_w2_input(e, Me)
            _check_point("C4 expert%d %s" % (e, name), Packed(q, z, s), x, q, z, s, Me)
