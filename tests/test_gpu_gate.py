"""The forget-gate producer with the cumulative gates in its epilogue (Sec. 2,
f = sigmoid(w_f^T x + b_f) per head; Sec. 3, two-stage implementation) against
the oracle: log f bit-identical to gate_log_forget, c bit-identical to
cumsum_log_gates of it (the chained scan across a sequence's blocks included),
and the forward that takes c from it bit-identical to fox_attn_fwd on the same
gates (plan, O, lse, and the backward after it)."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads
from tests._helpers import EPS, assert_same_plan, ensure_built, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _plan(ws, B, H, L, d, dtype):
    return {n: t.clone() for n, t in acp.plan_views(ws, B, H, L, d, dtype).items()}


@pytest.mark.parametrize("B,L,Dm,H,d,seed", [
    (2, 320, 64, 3, 64, 81),        # a partial group of heads, ragged block count
    (4, 1024, 1024, 16, 128, 82),
    (1, 16384, 768, 12, 64, 83),    # 256 blocks chained per head
    (2, 192, 128, 5, 64, 85),       # groups of two heads, the last one partial
    (1, 256, 64, 20, 64, 86),       # more groups than waves
])
def test_gate_projection_and_gated_forward(B, L, Dm, H, d, seed):
    print(f"case: gate projection B={B} L={L} d_model={Dm} H={H} d={d}", flush=True)
    p = workloads.gate_inputs(B, L, Dm, H, seed)
    lf_ref = orc.gate_log_forget(p["x"].float().numpy(), p["w_f"].float().numpy(),
                                 p["b_f"].numpy(), B)
    c_ref = orc.cumsum_log_gates(lf_ref)
    dev = torch.device("cuda:0")
    g = {n: t.to(dev) for n, t in p.items()}
    w = workloads.custom(f"gate{seed}", B, H, L, d, "bf16", seed)
    x = workloads.generate(w)
    a = to_gpu(x)
    lf, ws = acp.gate_project(g["x"], g["w_f"], g["b_f"], B, H, d)
    o_g, lse_g, _ = acp.forward_gated(a["q"], a["k"], a["v"], EPS, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lf.cpu().numpy(), lf_ref)
    plan_g = _plan(ws, B, H, L, d, torch.bfloat16)
    np.testing.assert_array_equal(plan_g["c"].cpu().numpy(), c_ref)
    assert int(plan_g["flags"].max()) == 0
    assert orc.cumsum_span_bits(lf_ref.reshape(-1, L)[0]) <= 52
    grads_g = acp.backward(a["q"], a["k"], a["v"], o_g, a["do"], ws)
    # the same gates through fox_attn_fwd (stage 1 scanning log f itself)
    lf_in = torch.from_numpy(lf_ref).to(dev)
    o, lse, ws2 = acp.forward(a["q"], a["k"], a["v"], lf_in, EPS)
    grads = acp.backward(a["q"], a["k"], a["v"], o, a["do"], ws2)
    torch.cuda.synchronize()
    assert_same_plan(plan_g, _plan(ws2, B, H, L, d, torch.bfloat16))
    assert torch.equal(o_g, o) and torch.equal(lse_g, lse)
    for x1, x2 in zip(grads_g, grads):
        assert torch.equal(x1, x2)


def test_gate_projection_flags_a_nan_input():
    B, L, Dm, H, d = 2, 256, 64, 4, 64
    p = workloads.gate_inputs(B, L, Dm, H, 84)
    x = p["x"].clone()
    x[100, 7] = float("nan")          # sequence 0, token 100
    dev = torch.device("cuda:0")
    print("case: gate projection with a NaN input", flush=True)
    _, ws = acp.gate_project(x.to(dev), p["w_f"].to(dev), p["b_f"].to(dev), B, H, d)
    w = workloads.custom("gatebad", B, H, L, d, "bf16", 84)
    a = to_gpu(workloads.generate(w, with_grad=False))
    acp.forward_gated(a["q"], a["k"], a["v"], EPS, ws)
    torch.cuda.synchronize()
    flags = acp.plan_views(ws, B, H, L, d, torch.bfloat16)["flags"].cpu().numpy()
    assert np.all(flags[0] & acp.FLAG_NONFINITE_GATE)
    assert np.all(flags[1] == 0)


def test_gate_projection_wide_spans():
    """Gate weights scaled up 12-fold spread each head's logits over about N(mu, 8),
    so that the chained scan adds gates 2^60 apart and more: spans of 60 to past
    105 bits.  log f stays bit-identical; flag bit 2 is set exactly from 105 bits
    on; below, c is bit-identical to the rounded exact sum, and the gated plan
    matches stage 1 scanning the same log f (c, flags and boundary)."""
    B, L, Dm, H, d = 2, 4096, 1024, 8, 64
    p = workloads.gate_inputs(B, L, Dm, H, 87, mu=(0.0, 5.0, 10.0, 15.0, 20.0, 25.0, 30.0, 35.0))
    p["w_f"] = (p["w_f"].float() * 12.0).bfloat16()
    lf_ref = orc.gate_log_forget(p["x"].float().numpy(), p["w_f"].float().numpy(),
                                 p["b_f"].numpy(), B)
    c_ref = orc.cumsum_log_gates(lf_ref)
    spans = np.array([[orc.cumsum_span_bits(lf_ref[b, h]) for h in range(H)] for b in range(B)])
    print(f"case: gate projection, wide spans {spans.min()}..{spans.max()}", flush=True)
    dev = torch.device("cuda:0")
    g = {n: t.to(dev) for n, t in p.items()}
    a = to_gpu(workloads.generate(workloads.custom("gatewide", B, H, L, d, "bf16", 87),
                                  with_grad=False))
    lf, ws = acp.gate_project(g["x"], g["w_f"], g["b_f"], B, H, d)
    acp.forward_gated(a["q"], a["k"], a["v"], EPS, ws)
    _, _, ws2 = acp.forward(a["q"], a["k"], a["v"], torch.from_numpy(lf_ref).to(dev), EPS)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lf.cpu().numpy(), lf_ref)
    plan_g = {n: t.cpu().numpy() for n, t in _plan(ws, B, H, L, d, torch.bfloat16).items()}
    plan_s = {n: t.cpu().numpy() for n, t in _plan(ws2, B, H, L, d, torch.bfloat16).items()}
    flag = np.where(spans >= 105, acp.FLAG_INEXACT_CUMSUM, 0)
    np.testing.assert_array_equal(plan_g["flags"], flag)
    np.testing.assert_array_equal(plan_s["flags"], flag)
    exact = spans < 105
    assert exact.any() and (spans[exact] > 53).any() and (~exact).any()
    np.testing.assert_array_equal(plan_g["c"][exact], c_ref[exact])
    np.testing.assert_array_equal(plan_s["c"][exact], c_ref[exact])
    for n in ("row_start", "col_end", "kept"):
        np.testing.assert_array_equal(plan_g[n][exact], plan_s[n][exact])
