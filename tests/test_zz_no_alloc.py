"""fox_attn_fwd_noalloc, the forward that allocates nothing (its workspace is
the library's fixed per-GPU array), against fox_attn_fwd with a caller
workspace: O and lse bit for bit, on two calls in a row, the second with a
smaller input (the array keeps the first call's plan, which must not leak into
the second)."""
import numpy as np
import pytest
import torch

from paper_2504_06949_amd import acp, workloads
from tests._helpers import ensure_built, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _noalloc(g, eps):
    q = g["q"]
    B, H, L, d = (int(s) for s in q.shape)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=q.device)
    st = acp.fox_attn_fwd_noalloc(q.data_ptr(), g["k"].data_ptr(), g["v"].data_ptr(),
                                  g["log_f"].data_ptr(), acp._dt(q), B, H, L, d, eps,
                                  o.data_ptr(), lse.data_ptr(),
                                  torch.cuda.current_stream().cuda_stream)
    assert st == acp.ACP_OK, acp.acp_last_error()
    return o, lse


def test_noalloc_forward_matches_workspace_forward_twice():
    cases = [workloads.WORKLOADS["125m"],                                  # 7.9 MB of plan
             workloads.custom("noalloc2", 1, 3, 1344, 128, "bf16", 91, mu=(0.5, 3.0, 9.0)),
             workloads.custom("noalloc3", 1, 2, 320, 64, "f32", 92, mu=(1.0, 6.0))]
    size = acp.acp_noalloc_scratch_bytes()
    for w in cases:
        print(f"case: noalloc forward {w.describe()}", flush=True)
        x = workloads.generate(w, with_grad=False)
        assert acp.acp_workspace_size(w.B, w.H, w.L, w.d, acp._dt(x["q"])) <= size
        g = to_gpu(x)
        o_ref, lse_ref, _ = acp.forward(g["q"], g["k"], g["v"], g["log_f"], w.eps)
        o, lse = _noalloc(g, w.eps)
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref), w.name
        assert torch.equal(lse, lse_ref), w.name
        assert torch.isfinite(o.float()).all()
