"""The autograd wrapper: the gradients autograd delivers are the bits of the
backward entry point (itself checked against the oracle in test_gpu_attn.py),
also for non-contiguous inputs and when O feeds a further computation."""
import pytest
import torch

from paper_2504_06949_amd import acp, workloads
from tests._helpers import ensure_built, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


@pytest.mark.parametrize("d,dtype", [(64, "bf16"), (128, "bf16"), (64, "f32")])
def test_autograd_matches_the_backward_entry_point(d, dtype):
    w = workloads.custom("ag", 2, 3, 704, d, dtype, 51, mu=(0.5, 3.0, 9.0))
    print(f"case: autograd {w.describe()}", flush=True)
    x = to_gpu(workloads.generate(w))
    o_ref, lse_ref, ws = acp.forward(x["q"], x["k"], x["v"], x["log_f"], w.eps)
    want = acp.backward(x["q"], x["k"], x["v"], o_ref, x["do"], ws)
    leaves = {n: x[n].clone().requires_grad_(True) for n in ("q", "k", "v", "log_f")}
    o, lse = acp.fox_attention(leaves["q"], leaves["k"], leaves["v"], leaves["log_f"], w.eps)
    assert not lse.requires_grad
    # d/dO of sum(O * dO) is dO exactly
    (o.double() * x["do"].double()).sum().backward()
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
    for n, g in zip(("q", "k", "v", "log_f"), want):
        assert torch.equal(leaves[n].grad, g), n


def test_autograd_through_strided_inputs():
    """Q, K, V given as [B, L, H, d] transposed views (not contiguous), log f as a
    transposed [B, L, H] view: same values and gradients as contiguous inputs."""
    w = workloads.custom("ags", 1, 4, 512, 64, "bf16", 52)
    print(f"case: autograd strided {w.describe()}", flush=True)
    x = to_gpu(workloads.generate(w))
    blhd = {n: x[n].transpose(1, 2).contiguous().requires_grad_(True) for n in ("q", "k", "v")}
    lf = x["log_f"].transpose(1, 2).contiguous().requires_grad_(True)
    o, _ = acp.fox_attention(blhd["q"].transpose(1, 2), blhd["k"].transpose(1, 2),
                             blhd["v"].transpose(1, 2), lf.transpose(1, 2), w.eps)
    (o.double() * x["do"].double()).sum().backward()
    o_ref, _, ws = acp.forward(x["q"], x["k"], x["v"], x["log_f"], w.eps)
    want = acp.backward(x["q"], x["k"], x["v"], o_ref, x["do"], ws)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref)
    for n, g in zip(("q", "k", "v"), want[:3]):
        assert torch.equal(blhd[n].grad.transpose(1, 2), g), n
    assert torch.equal(lf.grad.transpose(1, 2), want[3])
