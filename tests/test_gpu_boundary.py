"""Stage 1 on the GPU against the oracle: c, U, delta, row_start, col_end and the
kept-block count must be bit-identical, for every head of every workload."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads
from tests._helpers import EPS, ensure_built, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _gpu_plan(x, eps):
    g = to_gpu({n: x[n] for n in ("q", "k", "log_f")})
    out = acp.boundary(g["q"], g["k"], g["log_f"], eps)
    torch.cuda.synchronize()
    return {n: t.cpu().numpy() for n, t in out.items()}


def _check_plan(x, got, eps, brute_heads=()):
    B, H, L, d = x["q"].shape
    lf = x["log_f"].numpy()
    c_ref = orc.cumsum_log_gates(lf)
    np.testing.assert_array_equal(got["c"], c_ref)
    for b in range(B):
        for h in range(H):
            q = x["q"][b, h].float().numpy()
            k = x["k"][b, h].float().numpy()
            rq, rk = orc.row_norm_sq_max(q), orc.row_norm_sq_max(k)
            U = orc.logit_bound(rq, rk, d)
            delta = orc.threshold(U, L, eps)
            assert got["bound_u"][b, h] == U, (b, h)
            assert got["delta"][b, h] == delta, (b, h)
            method = "bruteforce" if (b, h) in brute_heads else "topright"
            kb = (orc.block_keep_bruteforce if method == "bruteforce" else
                  orc.block_keep_topright)(c_ref[b, h], delta)
            rs, ce = orc.boundary_from_block_keep(kb)
            np.testing.assert_array_equal(got["row_start"][b, h], rs, err_msg=f"{b},{h}")
            np.testing.assert_array_equal(got["col_end"][b, h], ce, err_msg=f"{b},{h}")
            assert got["kept"][b, h] == orc.kept_tiles(rs)
            assert got["flags"][b, h] == 0


@pytest.mark.parametrize("name", ["tiny", "125m", "360m", "760m", "adv"])
def test_boundary_bit_exact(name):
    w = workloads.WORKLOADS[name]
    print(f"case: boundary {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, w.eps)
    brute = {(0, 0), (0, 1)} if w.L <= 4096 else set()
    _check_plan(x, got, w.eps, brute_heads=brute)
    if name == "adv":
        # the sweep spans nothing-pruned to nearly-all-pruned heads
        frac = 1.0 - got["kept"] / orc.causal_tiles(w.M)
        assert frac.min() == 0.0 and frac.max() > 0.9


@pytest.mark.parametrize("L,sigma", [(4160, 0.5), (32768, 0.5), (4160, 6.0), (32768, 6.0)])
def test_boundary_lengths_off_the_vector_path(L, sigma):
    # L = 4160: runs of 5 gates per thread (scalar path); L = 32768: runs longer
    # than the registers hold (re-read from memory); both bit-exact.  A logit
    # spread of 6 takes every head to spans of 73-90 bits (the double-double round).
    if sigma > 1.0:
        w = workloads.custom("lenw", 1, 3, L, 64, "bf16", 13, mu=(0.5, 10.0, 20.0), gate_sigma=sigma)
    else:
        w = workloads.custom("len", 1, 3, L, 64, "bf16", 12, mu=(0.5, 3.0, 9.0))
    print(f"case: boundary {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, w.eps)
    _check_plan(x, got, w.eps)


def test_boundary_many_heads_exercise_sqrt_and_division():
    # 4096 heads of one block each, Q/K rows scaled per head over six decades:
    # U and delta must match the host's IEEE float64 arithmetic bit for bit.
    g = torch.Generator().manual_seed(11)
    B, H, L, d = 2, 2048, 64, 64
    sq = torch.exp(torch.randn(B, H, 1, 1, generator=g, dtype=torch.float64) * 3).float()
    sk = torch.exp(torch.randn(B, H, 1, 1, generator=g, dtype=torch.float64) * 3).float()
    x = {"q": (torch.randn(B, H, L, d, generator=g) * sq).bfloat16(),
         "k": (torch.randn(B, H, L, d, generator=g) * sk).bfloat16(),
         "log_f": workloads.log_sigmoid_f32_t(torch.randn(B, H, L, generator=g) + 1.0)}
    got = _gpu_plan(x, EPS)
    _check_plan(x, got, EPS)


def test_boundary_eps_zero_and_extremes():
    w = workloads.custom("ext", 1, 3, 1024, 64, "bf16", 5, mu=(0.0, 2.0, 4.0))
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, 0.0)
    assert np.all(got["row_start"] == 0)
    assert np.all(got["delta"] == -np.inf)
    _check_plan(x, got, 0.0)
    x["log_f"] = torch.full_like(x["log_f"], -1e4)
    got = _gpu_plan(x, EPS)
    assert np.all(got["row_start"] == np.arange(16))
    _check_plan(x, got, EPS)
    x["log_f"] = torch.zeros_like(x["log_f"])
    got = _gpu_plan(x, EPS)
    assert np.all(got["row_start"] == 0)


def test_boundary_flags_bad_gates():
    w = workloads.custom("flags", 1, 4, 256, 64, "f32", 6, mu=(2.0,))
    x = workloads.generate(w, with_grad=False)
    lf = x["log_f"].clone()
    lf[0, 1, 17] = 0.25           # f > 1
    lf[0, 2, 100] = float("nan")
    lf[0, 3, 0] = -1e-30          # tiny gate next to ordinary ones: a span beyond 105 bits
    x["log_f"] = lf
    got = _gpu_plan(x, EPS)
    assert got["flags"][0, 0] == 0
    assert got["flags"][0, 1] & acp.FLAG_POSITIVE_GATE
    assert got["flags"][0, 2] & acp.FLAG_NONFINITE_GATE
    assert got["flags"][0, 3] & acp.FLAG_INEXACT_CUMSUM
    # span check agrees with the oracle's own bound
    assert orc.cumsum_span_bits(lf[0, 3].numpy()) >= 105
    assert orc.cumsum_span_bits(lf[0, 0].numpy()) < 105


SPANS = (52, 53, 54, 104, 105, 106)


def test_inexact_cumsum_flag_at_105_bits_and_c_overflow():
    """Flag bit 2 against the oracle's rule on hand-built gates whose partial sums
    span 52, 53, 54, 104, 105 and 106 bits (63 gates of -6 and one full-significand
    gate of ulp 2^(E - span)); c bit-identical to the rounded exact sum wherever
    the flag is clear, also past the 53 bits a float64 sum holds.  A head whose
    cumulative sum leaves the float32 range (finite gates of -3e38) carries flag
    bit 1."""
    H = len(SPANS) + 2
    w = workloads.custom("span", 1, H, 64, 64, "f32", 8, mu=(2.0,))
    x = workloads.generate(w, with_grad=False)
    lf = torch.full((1, H, 64), -6.0, dtype=torch.float32)
    for h, span in enumerate(SPANS):
        lf[0, h, -1] = -(1.0 + 2.0 ** -23) * 2.0 ** (9 + 23 - span)
        assert orc.cumsum_span_bits(lf[0, h].numpy()) == span
    lf[0, H - 2, :2] = -3.0e38
    x["log_f"] = lf
    print("case: span flags " + "/".join(map(str, SPANS)) + ", c overflow", flush=True)
    got = _gpu_plan(x, EPS)
    for h, span in enumerate(SPANS):
        want = acp.FLAG_INEXACT_CUMSUM if orc.cumsum_inexact_flag(lf[0, h].numpy()) else 0
        assert want == (acp.FLAG_INEXACT_CUMSUM if span >= 105 else 0)
        assert got["flags"][0, h] == want, (h, got["flags"][0, h])
        if not want:
            np.testing.assert_array_equal(got["c"][0, h], orc.cumsum_log_gates(lf[0, h].numpy()))
            np.testing.assert_array_equal(got["c"][0, h], orc.cumsum_exact_fraction(lf[0, h].numpy()))
    assert got["flags"][0, H - 2] & acp.FLAG_NONFINITE_GATE
    assert not np.all(np.isfinite(orc.cumsum_log_gates(lf[0, H - 2].numpy())))
    assert got["flags"][0, H - 1] == 0


def test_boundary_is_deterministic():
    w = workloads.WORKLOADS["125m"]
    x = workloads.generate(w, with_grad=False)
    a = _gpu_plan(x, w.eps)
    b = _gpu_plan(x, w.eps)
    for n in a:
        np.testing.assert_array_equal(a[n], b[n])


def test_wide_gate_spreads_stay_exact():
    """Gates with a wide spread (logits N(mu, 3): log f from about -15 to -1e-17 in
    one head) give cumulative sums spanning more than the 53 bits of a float64 on
    many heads, and less than 105 on all.  No flag may be raised, and c, U, delta
    and the boundary must be bit-exact on every head: c is the float32 rounding of
    the exact prefix sum."""
    w = workloads.custom("wide", 2, 8, 4096, 64, "bf16", 91,
                         mu=(-2.0, 0.0, 3.0, 6.0, 10.0, 15.0, 20.0, 28.0), gate_sigma=3.0)
    print(f"case: boundary {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, w.eps)
    lf = x["log_f"].numpy()
    c_ref = orc.cumsum_log_gates(lf)
    wide = narrow = 0
    for b in range(w.B):
        for h in range(w.H):
            q = x["q"][b, h].float().numpy()
            k = x["k"][b, h].float().numpy()
            U = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), w.d)
            delta = orc.threshold(U, w.L, w.eps)
            assert got["bound_u"][b, h] == U and got["delta"][b, h] == delta, (b, h)
            span = orc.cumsum_span_bits(lf[b, h])
            fl = int(got["flags"][b, h])
            assert span < 105 and fl == 0, (b, h, span, fl)
            if span > 53:
                wide += 1
            else:
                narrow += 1
            np.testing.assert_array_equal(got["c"][b, h], c_ref[b, h])
            rs, ce = orc.boundary_from_block_keep(orc.block_keep_topright(c_ref[b, h], delta))
            np.testing.assert_array_equal(got["row_start"][b, h], rs)
            np.testing.assert_array_equal(got["col_end"][b, h], ce)
            assert got["kept"][b, h] == orc.kept_tiles(rs)
    print(f"  {wide} heads spanning more than 53 bits, {narrow} within 53", flush=True)
    assert wide > 0 and narrow > 0


def test_gate_spreads_near_105_bits():
    """Logits N(mu, 8) spread the gates of a head over 2^60 and more, so that the
    spans of the cumulative sums straddle 105 bits (84 to 108 here).  Flag bit 2
    must be set exactly from 105 bits on; below, c and the boundary are bit-exact
    (the float32 rounding of the exact sum); flagged heads keep c within one
    float32 ulp of it, and U and delta stay exact everywhere."""
    w = workloads.custom("wider", 2, 8, 4096, 64, "bf16", 93,
                         mu=(0.0, 5.0, 10.0, 15.0, 20.0, 25.0, 30.0, 35.0), gate_sigma=8.0)
    print(f"case: boundary {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, w.eps)
    lf = x["log_f"].numpy()
    c_ref = orc.cumsum_log_gates(lf)
    flagged = exact = 0
    for b in range(w.B):
        for h in range(w.H):
            q = x["q"][b, h].float().numpy()
            k = x["k"][b, h].float().numpy()
            U = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), w.d)
            delta = orc.threshold(U, w.L, w.eps)
            assert got["bound_u"][b, h] == U and got["delta"][b, h] == delta, (b, h)
            span = orc.cumsum_span_bits(lf[b, h])
            fl = int(got["flags"][b, h])
            assert fl == (acp.FLAG_INEXACT_CUMSUM if span >= 105 else 0), (b, h, span, fl)
            if fl:
                flagged += 1
                ulp = np.spacing(np.abs(c_ref[b, h]).astype(np.float32))
                assert np.all(np.abs(got["c"][b, h] - c_ref[b, h]) <= ulp), (b, h)
                continue
            exact += 1
            np.testing.assert_array_equal(got["c"][b, h], c_ref[b, h])
            rs, ce = orc.boundary_from_block_keep(orc.block_keep_topright(c_ref[b, h], delta))
            np.testing.assert_array_equal(got["row_start"][b, h], rs)
            np.testing.assert_array_equal(got["col_end"][b, h], ce)
    print(f"  {flagged} heads flagged, {exact} exact", flush=True)
    assert flagged > 0 and exact > 0


def test_wide_spreads_at_the_760m_shape():
    """The 760M-shaped layer (B = 2, H = 24, L = 16384, the longest held-in-register
    runs) with logit spreads of 8: every head goes through the double-double round;
    flag bit 2 exactly from 105 bits on, c and the boundary bit-exact below."""
    w = workloads.custom("wide760", 2, 24, 16384, 64, "bf16", 95,
                         mu=tuple(float(m) for m in np.linspace(0.0, 36.0, 24)), gate_sigma=8.0)
    print(f"case: boundary {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    got = _gpu_plan(x, w.eps)
    lf = x["log_f"].numpy()
    c_ref = orc.cumsum_log_gates(lf)
    spans = np.array([[orc.cumsum_span_bits(lf[b, h]) for h in range(w.H)] for b in range(w.B)])
    assert spans.min() > 53
    np.testing.assert_array_equal(got["flags"], np.where(spans >= 105, acp.FLAG_INEXACT_CUMSUM, 0))
    for b in range(w.B):
        for h in range(w.H):
            if spans[b, h] >= 105:
                continue
            np.testing.assert_array_equal(got["c"][b, h], c_ref[b, h])
            q = x["q"][b, h].float().numpy()
            k = x["k"][b, h].float().numpy()
            U = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), w.d)
            delta = orc.threshold(U, w.L, w.eps)
            rs, ce = orc.boundary_from_block_keep(orc.block_keep_topright(c_ref[b, h], delta))
            np.testing.assert_array_equal(got["row_start"][b, h], rs)
            np.testing.assert_array_equal(got["col_end"][b, h], ce)
