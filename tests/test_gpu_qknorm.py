"""Stage 1 with the logit bound from QK-norm scales (App. E): the boundary must
be bit-identical to the oracle's plan with U = gamma_q gamma_k sqrt(d), the
attention on top of it must match the oracle, and no pass over Q and K runs."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads
from tests._helpers import EPS, ensure_built, f64, head_inputs, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _u(x, h, d):
    return orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), d)


def test_boundary_qknorm_bit_exact():
    w = workloads.custom("qk", 2, 6, 2048, 64, "bf16", 31, mu=(0.5, 1.5, 3.0, 5.0, 8.0, 20.0),
                         qk_norm=True)
    print(f"case: boundary_qknorm {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    g = to_gpu({n: x[n] for n in ("log_f", "gamma_q", "gamma_k")})
    got = acp.boundary_qknorm(g["log_f"], g["gamma_q"], g["gamma_k"], w.d, w.eps)
    torch.cuda.synchronize()
    got = {n: t.cpu().numpy() for n, t in got.items()}
    c_ref = orc.cumsum_log_gates(x["log_f"].numpy())
    np.testing.assert_array_equal(got["c"], c_ref)
    pruned = 0
    for b in range(w.B):
        for h in range(w.H):
            U = _u(x, h, w.d)
            delta = orc.threshold(U, w.L, w.eps)
            assert got["bound_u"][b, h] == U and got["delta"][b, h] == delta, (b, h)
            rs, ce = orc.boundary_from_block_keep(orc.block_keep_topright(c_ref[b, h], delta))
            np.testing.assert_array_equal(got["row_start"][b, h], rs, err_msg=f"{b},{h}")
            np.testing.assert_array_equal(got["col_end"][b, h], ce, err_msg=f"{b},{h}")
            assert got["kept"][b, h] == orc.kept_tiles(rs) and got["flags"][b, h] == 0
            pruned += orc.causal_tiles(w.M) - orc.kept_tiles(rs)
    assert pruned > 0


@pytest.mark.parametrize("d", [64, 128])
def test_forward_backward_qknorm_matches_oracle(d):
    w = workloads.custom("qk", 1, 3, 320, d, "bf16", 32, mu=(1.0, 3.0, 8.0), qk_norm=True)
    print(f"case: fwd/bwd qknorm {w.describe()}", flush=True)
    x = workloads.generate(w)
    g = to_gpu(x)
    acp.acp_timing_enable(True)
    acp.acp_timing_reset()
    o, lse, ws = acp.forward_qknorm(g["q"], g["k"], g["v"], g["log_f"], g["gamma_q"],
                                    g["gamma_k"], EPS)
    dq, dk, dv, dlf = acp.backward(g["q"], g["k"], g["v"], o, g["do"], ws)
    torch.cuda.synchronize()
    kt = acp.acp_timing_read()
    acp.acp_timing_enable(False)
    assert kt["rownorm"][0] == 0 and kt["plan"][0] == 1 and kt["fwd"][0] == 1
    got = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv, "dlog_f": dlf}
    for h in range(w.H):
        q, k, v, do, lf = head_inputs(x, 0, h)
        ref = orc.run_head(q, k, v, lf, EPS, do=do, U=_u(x, h, w.d))
        errs = {n: float(np.max(np.abs(f64(got[n][0, h]) - ref[n]))) for n in got}
        # bf16 outputs carry a relative rounding of 2^-9: where O or a gradient
        # exceeds 1 in size (dQ of QK-normed rows at d = 128) its bound is relative
        # to it, as in the attention tests; LSE and dlog f keep the absolute bound
        bound = {n: 2e-2 * (max(1.0, float(np.max(np.abs(ref[n])))) if n in ("o", "dq", "dk", "dv")
                            else 1.0) for n in got}
        print(f"  head {h}: kept {ref['kept']} of {orc.causal_tiles(w.M)}, errors {errs}, "
              f"bounds {bound}", flush=True)
        assert all(errs[n] <= bound[n] for n in got), (h, errs, bound)


def test_qknorm_bad_scale_is_flagged():
    w = workloads.custom("qk", 1, 2, 256, 64, "bf16", 33, qk_norm=True)
    x = workloads.generate(w, with_grad=False)
    g = to_gpu({n: x[n] for n in ("log_f", "gamma_q", "gamma_k")})
    g["gamma_q"][1] = -1.0
    g["gamma_k"][0] = float("nan")
    got = acp.boundary_qknorm(g["log_f"], g["gamma_q"], g["gamma_k"], w.d, w.eps)
    torch.cuda.synchronize()
    flags = got["flags"].cpu().numpy()
    assert np.all(flags & 8)
