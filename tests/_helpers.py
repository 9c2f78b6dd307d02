"""Shared pieces of the test suite: building the library, moving seeded inputs
to the GPU, and running the oracle head by head."""
import math
import os

import numpy as np
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads

EPS = math.exp(-10.0)


def ensure_built():
    """Build libacp.so if it is missing (tests load what is built otherwise)."""
    if not os.path.exists(acp.LIB_PATH):
        from paper_2504_06949_amd import build
        build.build()
    acp.lib()


def to_gpu(x: dict) -> dict:
    return {k: (v.cuda() if torch.is_tensor(v) else v) for k, v in x.items()}


def head_inputs(x: dict, b: int, h: int):
    """float64 numpy copies of one head's inputs (exact upcasts)."""
    q = workloads.to_f64(x["q"][b, h])
    k = workloads.to_f64(x["k"][b, h])
    v = workloads.to_f64(x["v"][b, h])
    do = workloads.to_f64(x["do"][b, h]) if "do" in x else None
    lf = x["log_f"][b, h].numpy()
    return q, k, v, do, lf


def oracle_head(x: dict, b: int, h: int, eps: float, grads: bool = True, method="topright"):
    q, k, v, do, lf = head_inputs(x, b, h)
    return orc.run_head(q, k, v, lf, eps, do=do if grads else None, method=method)


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_same_plan(plan: dict, plan2: dict):
    """Two plans of the same inputs: every field bit for bit, except that the
    workgroup schedules (sched_q, sched_k) only fix which items each XCD's range
    of logical ids holds, not their order among items of equal work."""
    nblocks = plan["sched_q"].numel()
    q, r = divmod(nblocks, 8)
    for n in plan:
        if n.startswith("sched"):
            a, b = plan[n].cpu(), plan2[n].cpu()
            for x in range(8):
                lo = x * q + min(x, r)
                hi = lo + q + (1 if x < r else 0)
                assert torch.equal(a[lo:hi].sort().values, b[lo:hi].sort().values), (n, x)
        else:
            assert torch.equal(plan[n], plan2[n]), n
