"""The benchmark's algorithmic work model against the oracle's own source
counts: the closed forms bench.py prices the roofline with must equal the
number of query-source pairs the method defines (Sec. 3), rank p included."""
import sys
import os

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402
import fma_inputs  # noqa: E402
import oracle  # noqa: E402


@pytest.mark.parametrize("ndim,causal,size,r,p", [(1, False, 2048, 64, 1), (1, True, 2048, 64, 1),
                                                  (1, True, 4096, 128, 4), (1, False, 1024, 64, 3),
                                                  (2, False, 64, 8, 1), (2, False, 64, 8, 4),
                                                  (2, False, 64, 16, 2)])
def test_pairs_equal_oracle_counts(ndim, causal, size, r, p):
    if ndim == 1:
        w = fma_inputs.custom("m", 1, causal, "bf16", 1, 1, n=size, block=r, seed=1, rank=p)
    else:
        w = fma_inputs.custom("m", 2, False, "bf16", 1, 1, side=size, block=r, seed=1, rank=p)
    q, k, v, wk, wv = [x.double().numpy() for x in fma_inputs.make_inputs(w)]
    if ndim == 1:
        _, c = oracle.forward_1d(q[0, 0], k[0, 0], v[0, 0], r, wk[0], wv[0], causal=causal,
                                 return_counts=True, rank=p)
        R = p * oracle.coarse_rows_1d(size, r)
    else:
        _, c = oracle.forward_2d(q[0, 0], k[0, 0], v[0, 0], size, r, wk[0], wv[0], return_counts=True, rank=p)
        R = p * oracle.coarse_rows_2d(size, r)
    m = bench.work_model(w)
    assert m["pairs"] == int(np.sum(c))
    assert m["R"] == R


def test_rank_workload_names():
    w = bench.workload(fma_inputs, "C4_p4")
    assert w.rank == 4 and w.n == fma_inputs.WORKLOADS["C4"].n
    assert bench.workload(fma_inputs, "C3").rank == 1
