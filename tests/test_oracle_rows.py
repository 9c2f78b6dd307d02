"""Pins of the row/column-sampled oracle functions against the dense oracle
(itself pinned in test_oracle.py) on small heads with pruning active."""
import math

import numpy as np
import pytest

import oracle as orc
from paper_2504_06949_amd import workloads

EPS = math.exp(-10.0)


@pytest.mark.parametrize("seed,mu", [(0, 0.5), (1, 1.5), (2, 6.0)])
def test_rows_and_cols_match_dense(seed, mu):
    rng = np.random.default_rng(seed)
    L, d = 384, 16
    q, k, v, do = (rng.standard_normal((L, d)) for _ in range(4))
    lf = workloads.log_sigmoid_f32(mu + 0.5 * rng.standard_normal(L))
    full = orc.run_head(q, k, v, lf, EPS, do=do)
    rs = full["row_start"]
    rows = [0, 1, 63, 64, 200, 383]
    o, lse = orc.forward_rows(q, k, v, full["c"], rs, rows)
    np.testing.assert_allclose(o, full["o"][rows], atol=1e-12)
    np.testing.assert_allclose(lse, full["lse"][rows], atol=1e-12)
    dq, rsum = orc.backward_rows(q, k, v, full["c"], rs, do, rows)
    np.testing.assert_allclose(dq, full["dq"][rows], atol=1e-11)
    g = orc.backward(q, k, v, full["c"], full["mask"], do)
    np.testing.assert_allclose(rsum, g["ds"].sum(axis=1)[rows], atol=1e-12)
    cols = [0, 5, 64, 130, 383]
    dk, dv, csum = orc.backward_cols(q, k, v, full["c"], rs, do, cols)
    np.testing.assert_allclose(dk, full["dk"][cols], atol=1e-11)
    np.testing.assert_allclose(dv, full["dv"][cols], atol=1e-11)
    np.testing.assert_allclose(csum, g["ds"].sum(axis=0)[cols], atol=1e-12)
