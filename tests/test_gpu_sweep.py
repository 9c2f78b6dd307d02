"""The eps sweep and per-head histogram report what the oracle's boundary gives:
per-head kept-block counts equal the oracle's at every eps, and the pruned
fraction never decreases as eps grows (a larger tolerance raises delta)."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, sweep, workloads
from tests._helpers import ensure_built

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def test_sweep_matches_oracle_and_is_monotone():
    w = workloads.custom("sweep", 1, 8, 1024, 64, "bf16", 41,
                         mu=(0.0, 1.0, 2.0, 3.0, 5.0, 8.0, 12.0, 20.0))
    print(f"case: eps sweep {w.describe()}", flush=True)
    eps_list = (math.exp(-1), math.exp(-5), math.exp(-10), math.exp(-20), 0.0)
    res = sweep.eps_sweep(w, eps_list)
    x = workloads.generate(w, with_grad=False)
    fr_prev = -1.0
    for eps, row in zip(sorted(eps_list), sorted(res["rows"], key=lambda r: r["eps"])):
        fr = []
        for h in range(w.H):
            q = workloads.to_f64(x["q"][0, h]); k = workloads.to_f64(x["k"][0, h])
            p = orc.plan_head(q, k, x["log_f"][0, h].numpy(), eps, method="topright")
            fr.append(1.0 - p["kept"] / orc.causal_tiles(w.M))
        fr = np.array(fr)
        assert row["pruned_fraction"] == round(float(fr.mean()), 4), eps
        assert row["head_histogram"] == sweep.head_histogram(fr)
        assert row["heads_fully_kept"] == int(np.sum(fr == 0.0))
        assert sum(row["head_histogram"]) == w.H
        assert fr.mean() >= fr_prev - 1e-12
        fr_prev = fr.mean()
    assert res["rows"][-1]["pruned_fraction"] == 0.0     # eps = 0 prunes nothing
