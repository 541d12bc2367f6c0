"""Host threads calling the library at once, each on its own stream: the
per-(device, stream) workspaces (split-K partials, stream-K and sliced-kernel
counters and partial tiles) are created and grown concurrently, and every
result is checked against the oracle afterwards."""
import threading

import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu

PLANS = [None, dict(variant=2, split_k=4, tile_m=32, tile_n=16), dict(variant=3, split_k=0, tile_m=64, tile_n=32),
         dict(variant=5, split_k=4, tile_n=1), dict(variant=7, split_k=16, tile_m=64, tile_n=32),
         dict(variant=1, split_k=8, tile_n=2)]


def test_concurrent_threads_own_streams():
    cases = []
    for i, (M, K, N) in enumerate([(16, 1024, 272), (48, 2048, 528), (9, 3072, 400), (130, 1536, 640)]):
        x, q, z, s = rand_case(300 + i, M, K, N)
        cases.append((x, Packed(q, z, s), oracle.gemm(x, q, z, s)))
    n_threads, rounds = 4, 3
    results = {}
    errors = []
    barrier = threading.Barrier(n_threads)

    def worker(t):
        try:
            st = torch.cuda.Stream()
            barrier.wait()
            with torch.cuda.stream(st):
                for r in range(rounds):
                    for c, (x, p, _) in enumerate(cases):
                        plan = PLANS[(t + r + c) % len(PLANS)]
                        if plan and plan["variant"] == 5 and x.shape[0] > 16:
                            plan = None
                        if plan and plan["variant"] == 1 and x.shape[0] > 64:
                            plan = None
                        y = p.gemm(to_dev_x(x), cfg=Q.make_config(**plan) if plan else None, stream=st)
                        results[(t, r, c)] = (y, plan)
            st.synchronize()
        except Exception as e:   # reported in the main thread
            errors.append((t, repr(e)))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    say("threads: %d x %d rounds x %d cases" % (n_threads, rounds, len(cases)))
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads), "a worker did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    assert len(results) == n_threads * rounds * len(cases)
    for (t, r, c), (y, plan) in sorted(results.items()):
        err = rel_err(from_dev_y(y), cases[c][2])
        assert err <= TOL, "thread %d round %d case %d plan %s: %.3g" % (t, r, c, plan, err)
