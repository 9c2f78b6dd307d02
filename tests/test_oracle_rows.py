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


@pytest.mark.parametrize("seed,mu,group", [(3, 0.5, 64), (4, 1.5, 100), (5, 6.0, 256)])
def test_row_range_matches_dense(seed, mu, group):
    """backward_row_range over all rows equals the dense oracle entry for entry
    (groups that split pruning blocks and leave a ragged last group); over a
    partial range it holds the complete columns whose keeping rows it covers, and
    the rectangle sums give dlog f."""
    rng = np.random.default_rng(seed)
    L, d = 448, 16
    q, k, v, do = (rng.standard_normal((L, d)) for _ in range(4))
    lf = workloads.log_sigmoid_f32(mu + 0.5 * rng.standard_normal(L))
    full = orc.run_head(q, k, v, lf, EPS, do=do)
    g = orc.backward(q, k, v, full["c"], full["mask"], do)
    rs, ce, c = full["row_start"], full["col_end"], full["c"]
    ls = (1, 64, 200, 447)
    r = orc.backward_row_range(q, k, v, c, rs, do, 0, L, ls=ls, group=group)
    for n, ref in (("o", full["o"]), ("lse", full["lse"]), ("dq", full["dq"]),
                   ("dk", full["dk"]), ("dv", full["dv"]),
                   ("rowsum", g["ds"].sum(axis=1)), ("colsum", g["ds"].sum(axis=0))):
        np.testing.assert_allclose(r[n], ref, atol=1e-11, err_msg=n)
    for l in ls:
        assert abs(r["rect"][l] - full["dlog_f"][l]) <= 1e-11
    # key block 2 (keys 128..191) only: rows 128 .. 64 col_end[2] + 63
    r0, r1 = 128, 64 * int(ce[2]) + 64
    p = orc.backward_row_range(q, k, v, c, rs, do, r0, r1, group=group)
    np.testing.assert_allclose(p["dk"][128:192], full["dk"][128:192], atol=1e-11)
    np.testing.assert_allclose(p["dv"][128:192], full["dv"][128:192], atol=1e-11)
    np.testing.assert_allclose(p["dq"], full["dq"][r0:r1], atol=1e-11)
