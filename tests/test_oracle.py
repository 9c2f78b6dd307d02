"""Pins for the CPU oracle: closed forms, textbook special cases, the paper's
error bound, independent derivations (exact rationals, autograd, finite
differences) and brute force.  None of these re-types the oracle's own formula.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import workloads

EPS = math.exp(-10.0)


def _rng(seed):
    return np.random.default_rng(seed)


def _gates(rng, L, mu, sigma=0.5):
    a = mu + sigma * rng.standard_normal(L)
    return workloads.log_sigmoid_f32(a)


# --------------------------------------------------------------------------
# c (Sec. 2): exact rational prefix sums and a dyadic closed form
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mu", [0.0, 1.0, 3.0, 6.0, 12.0, 20.0])
def test_cumsum_equals_exact_rational(mu):
    lf = _gates(_rng(1), 512, mu)
    assert orc.cumsum_span_bits(lf) <= 53
    np.testing.assert_array_equal(orc.cumsum_log_gates(lf), orc.cumsum_exact_fraction(lf))


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_cumsum_of_wide_rows_is_the_rounded_exact_sum(seed):
    # strong gates mixed with nearly saturated ones (log f down to about -1e-18):
    # the partial sums span far more than 53 bits, so float64 running sums round,
    # yet c is the float32 rounding of the exact sum, whatever the order
    rng = _rng(seed)
    a = np.concatenate([3.0 * rng.standard_normal(1500), 40.0 + rng.standard_normal(1500)])
    rng.shuffle(a)
    lf = workloads.log_sigmoid_f32(a)
    assert orc.cumsum_span_bits(lf) > 80
    c = orc.cumsum_log_gates(lf)
    np.testing.assert_array_equal(c, orc.cumsum_exact_fraction(lf))
    np.testing.assert_array_equal(orc.cumsum_log_gates(lf[::-1].copy())[-1], c[-1])


def test_cumsum_dyadic_constant_gate_closed_form():
    lam = 2.0 ** -3
    L = 4096
    c = orc.cumsum_log_gates(np.full(L, -lam, dtype=np.float32))
    np.testing.assert_array_equal(c, (-lam * (np.arange(L) + 1)).astype(np.float32))


def test_cumsum_span_of_paper_like_gates_is_far_below_53_bits():
    # 32k positions, every gate class of the workloads: partial sums stay exact.
    for mu in (0.0, 1.0, 3.0, 6.0, 10.0, 12.0, 20.0):
        assert orc.cumsum_span_bits(_gates(_rng(2), 32768, mu)) <= 45


def _span_gates(span):
    """63 gates of -6 (|sum| in [256, 512), so E = 9) and, last, one gate with a
    full 24-bit significand, -(1 + 2^-23) 2^a, whose ulp 2^(a - 23) is the
    smallest: the span is E - (a - 23) by construction."""
    a = 9 + 23 - span
    lf = np.full(64, -6.0, dtype=np.float32)
    lf[-1] = np.float32(-(1.0 + 2.0 ** -23) * 2.0 ** a)
    assert float(lf[-1]) == -(1.0 + 2.0 ** -23) * 2.0 ** a   # representable
    return lf


def _float64_prefix_sums_exact(lf) -> bool:
    """Every float64 running partial sum equals the exact rational one."""
    acc, exact = 0.0, Fraction(0)
    for v in np.asarray(lf, dtype=np.float32).astype(np.float64):
        acc += float(v)
        exact += Fraction(float(v))
        if Fraction(acc) != exact:
            return False
    return True


@pytest.mark.parametrize("span", [52, 53, 54, 104, 105, 106])
def test_cumsum_span_bits_hand_built(span):
    # the count itself (an off-by-one in E or in the ulp exponent fails here)
    lf = _span_gates(span)
    assert orc.cumsum_span_bits(lf) == span
    # what the count promises: up to 53 bits every float64 partial sum is exact;
    # at 54 the last one (bits 2^8 .. 2^-45) is not
    assert _float64_prefix_sums_exact(lf) == (span <= 53)
    # c is the rounded exact sum at any span
    np.testing.assert_array_equal(orc.cumsum_log_gates(lf), orc.cumsum_exact_fraction(lf))
    # flag bit 2 is raised from 105 bits on (the device's double-double sums)
    assert orc.cumsum_inexact_flag(lf) == (span >= 105)


def test_cumsum_span_bits_power_of_two_total_and_subnormal():
    # |sum| = 256 exactly: 2^8 <= 256 < 2^9, so E = 9; ulp of -4 is 2^-21
    assert orc.cumsum_span_bits(np.full(64, -4.0, dtype=np.float32)) == 9 + 21
    # a subnormal gate takes the smallest normal's ulp exponent, -149
    lf = np.array([-1.0, -2.0 ** -140], dtype=np.float32)
    assert orc.cumsum_span_bits(lf) == 1 + 149   # 1 <= |sum| < 2: E = 1
    assert orc.cumsum_span_bits(np.zeros(8, dtype=np.float32)) == 0


def test_fraction_rounding_is_single_rounding():
    # 1 + 2^-24 + 2^-60 must round up to 1 + 2^-23 (a float64 detour would round
    # 1 + 2^-24 + 2^-60 to 1 + 2^-24 and then tie to even, giving 1).
    from oracle.acp_oracle import _fraction_to_f32
    x = Fraction(1) + Fraction(1, 2 ** 24) + Fraction(1, 2 ** 60)
    assert _fraction_to_f32(x) == np.float32(1 + 2.0 ** -23)
    assert _fraction_to_f32(Fraction(1) + Fraction(1, 2 ** 24)) == np.float32(1.0)
    assert _fraction_to_f32(-Fraction(3, 2 ** 150)) == np.float32(-3 * 2.0 ** -150)


# --------------------------------------------------------------------------
# rho, U, delta (Sec. 3): closed forms
# --------------------------------------------------------------------------

def test_norm_and_bound_closed_form_axis_rows():
    L, d, r = 256, 64, 4.0
    q = np.zeros((L, d)); q[:, 0] = r
    k = np.zeros((L, d)); k[:, 5] = -r
    assert orc.row_norm_sq_max(q) == r * r
    U = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), d)
    assert U == r * r / 8.0  # sqrt(64) = 8


def test_norm_picks_the_largest_row():
    rng = _rng(3)
    x = np.sign(rng.standard_normal((128, 16)))  # every row has squared norm 16
    x[77] *= 3.0                                  # one row with squared norm 144
    assert orc.row_norm_sq_max(x) == 144.0


def test_bound_dominates_every_logit_and_is_attained():
    rng = _rng(4)
    L, d = 200, 32
    q = rng.standard_normal((L, d)); k = rng.standard_normal((L, d)) * 3
    U = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), d)
    assert np.max(np.abs(q @ k.T)) / math.sqrt(d) <= U
    # parallel extremal rows attain the bound
    iq = np.argmax(np.sum(q * q, 1)); ik = np.argmax(np.sum(k * k, 1))
    k2 = k.copy(); k2[ik] = q[iq] * np.linalg.norm(k[ik]) / np.linalg.norm(q[iq])
    U2 = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k2), d)
    assert abs(q[iq] @ k2[ik] / math.sqrt(d) - U2) <= 1e-12 * U2


def _rms_rows(x):
    return x / np.sqrt(np.mean(x * x, axis=1, keepdims=True))


def test_qknorm_bound_attained_by_constant_rows():
    # RMSNorm of a constant row is all ones; with every weight at gamma the rows are
    # gamma_q 1 and gamma_k 1, whose logit gamma_q gamma_k d / sqrt(d) is the bound.
    d, gq, gk = 64, 1.375, 0.8125            # dyadic: every step below is exact
    q = _rms_rows(np.full((3, d), -2.5)) * gq
    k = _rms_rows(np.full((5, d), 7.0)) * gk
    U = orc.logit_bound_qknorm(gq, gk, d)
    assert U == gq * gk * 8.0
    assert np.max(np.abs(q @ k.T)) / math.sqrt(d) == U


def test_qknorm_bound_dominates_normalised_scaled_rows():
    rng = _rng(11)
    L, d = 300, 64
    wq = rng.uniform(-1.7, 1.7, d); wk = rng.uniform(0.2, 0.9, d)
    q = _rms_rows(rng.standard_normal((L, d)) * rng.uniform(0.1, 9.0, (L, 1))) * wq
    k = _rms_rows(rng.standard_normal((L, d))) * wk
    U = orc.logit_bound_qknorm(np.max(np.abs(wq)), np.max(np.abs(wk)), d)
    assert np.max(np.abs(q @ k.T)) / math.sqrt(d) <= U
    # it is never tighter than the bound from the actual row norms
    U_rows = orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), d)
    assert U_rows <= U


def test_plan_with_given_bound_prunes_a_subset():
    # a larger (still valid) U lowers delta, so the pruned blocks shrink
    w = workloads.custom("qk", 1, 2, 512, 64, "f32", 21, mu=(1.0, 2.0), qk_norm=True)
    x = workloads.generate(w, with_grad=False)
    for h in range(2):
        q = workloads.to_f64(x["q"][0, h]); k = workloads.to_f64(x["k"][0, h])
        lf = x["log_f"][0, h].numpy()
        U = orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), 64)
        pn = orc.plan_head(q, k, lf, EPS)
        pq = orc.plan_head(q, k, lf, EPS, U=U)
        assert pq["U"] == U and pn["U"] <= U
        assert pq["delta"] == orc.threshold(U, 512, EPS)
        assert np.all(pq["row_start"] <= pn["row_start"])
        kb = orc.block_keep_bruteforce(pq["c"], pq["delta"])
        np.testing.assert_array_equal(pq["row_start"], orc.boundary_from_block_keep(kb)[0])


def test_threshold_hand_value():
    # U = 2, L = 512, eps = e^-10: delta = -(4 + 9 ln 2 + 10)
    delta = orc.threshold(2.0, 512, EPS)
    assert abs(delta - (-(14.0 + 9.0 * math.log(2.0)))) <= 4 * np.spacing(abs(delta))
    assert orc.threshold(2.0, 512, 0.0) == -math.inf


# --------------------------------------------------------------------------
# Boundary (Sec. 3, block rule and Algorithm 1)
# --------------------------------------------------------------------------

def _closed_form_row_start(M, lam, delta):
    # constant gate -lam: top-right entry of block (m, n<m) is -lam (64 (m-n) - 63)
    W = -delta / lam
    return np.maximum(0, np.arange(M) - math.floor((W + 63.0) / 64.0)).astype(np.int32)


@pytest.mark.parametrize("lam,r", [(2.0 ** -3, 4.0), (2.0 ** -5, 3.0), (0.75, 1.0)])
def test_boundary_constant_gate_closed_form(lam, r):
    L, d = 2048, 64
    M = L // 64
    q = np.zeros((L, d)); q[:, 0] = r
    k = np.zeros((L, d)); k[:, 1] = r
    lf = np.full(L, -lam, dtype=np.float32)
    for method in ("bruteforce", "topright", "alg1"):
        plan = orc.plan_head(q, k, lf, EPS, method=method)
        W = -plan["delta"] / lam
        assert abs((W + 63) / 64 - round((W + 63) / 64)) > 1e-6  # not on a knife edge
        np.testing.assert_array_equal(plan["row_start"], _closed_form_row_start(M, lam, plan["delta"]))


def test_boundary_tie_is_kept():
    lam = 2.0 ** -3
    L = 1024
    c = orc.cumsum_log_gates(np.full(L, -lam, dtype=np.float32))
    for k_ in (1, 2, 3):
        delta = -lam * (64 * k_ - 63)       # block (m, m-k) top-right entry exactly delta
        for kb in (orc.block_keep_bruteforce(c, delta), orc.block_keep_topright(c, delta)):
            rs, _ = orc.boundary_from_block_keep(kb)
            np.testing.assert_array_equal(rs, np.maximum(0, np.arange(L // 64) - k_))
        np.testing.assert_array_equal(orc.boundary_alg1(c, delta), np.maximum(0, np.arange(L // 64) - k_))
        # an ulp lower bound flips the block (m, m-k) to pruned -> back to m-k+1
        d2 = np.nextafter(delta, 0.0)
        np.testing.assert_array_equal(orc.boundary_alg1(c, d2), np.maximum(0, np.arange(L // 64) - k_ + 1))


def test_boundary_extremes():
    L, d = 1024, 16
    rng = _rng(5)
    q = rng.standard_normal((L, d)); k = rng.standard_normal((L, d))
    M = L // 64
    p0 = orc.plan_head(q, k, np.zeros(L, np.float32), EPS)
    np.testing.assert_array_equal(p0["row_start"], np.zeros(M))
    assert p0["kept"] == orc.causal_tiles(M)
    p1 = orc.plan_head(q, k, np.full(L, -1e4, np.float32), EPS)
    np.testing.assert_array_equal(p1["row_start"], np.arange(M))
    np.testing.assert_array_equal(p1["col_end"], np.arange(M))
    assert p1["kept"] == M
    pz = orc.plan_head(q, k, np.full(L, -1e4, np.float32), 0.0)   # eps = 0: nothing pruned
    np.testing.assert_array_equal(pz["row_start"], np.zeros(M))


@pytest.mark.parametrize("seed", range(6))
def test_boundary_three_ways_agree_and_staircase(seed):
    rng = _rng(100 + seed)
    L = int(rng.choice([512, 1024, 1536]))
    d = int(rng.choice([16, 64]))
    mu = float(rng.choice([-1.0, 0.0, 1.0, 2.0, 3.0, 5.0]))
    q = rng.standard_normal((L, d)) * rng.choice([0.3, 1.0, 2.0])
    k = rng.standard_normal((L, d))
    lf = _gates(rng, L, mu, sigma=float(rng.choice([0.5, 2.0])))
    pb = orc.plan_head(q, k, lf, EPS, method="bruteforce")
    pt = orc.plan_head(q, k, lf, EPS, method="topright")
    pa = orc.plan_head(q, k, lf, EPS, method="alg1")
    for p in (pt, pa):
        np.testing.assert_array_equal(pb["row_start"], p["row_start"])
        np.testing.assert_array_equal(pb["col_end"], p["col_end"])
    rs = pb["row_start"]; M = L // 64
    assert np.all(np.diff(rs) >= 0) and np.all(rs <= np.arange(M)) and np.all(rs >= 0)
    np.testing.assert_array_equal(pb["col_end"], orc.col_end_from_row_start(rs))


def test_tiny_workload_prunes_local_head_only():
    w = workloads.WORKLOADS["tiny"]
    x = workloads.generate(w, with_grad=False)
    kept = []
    for h in range(w.H):
        q = workloads.to_f64(x["q"][0, h]); k = workloads.to_f64(x["k"][0, h])
        lf = x["log_f"][0, h].numpy()
        kept.append(orc.plan_head(q, k, lf, EPS)["kept"])
    assert kept[1] == orc.causal_tiles(w.M)          # mu = 8: nothing pruned
    assert kept[0] < orc.causal_tiles(w.M)           # mu = 2: some blocks pruned


# --------------------------------------------------------------------------
# Forward (eq. 1-3): textbook special cases, closed forms, App. A bound
# --------------------------------------------------------------------------

def test_forward_no_forgetting_is_causal_sdpa():
    rng = _rng(6)
    L, d = 256, 32
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    o, _ = orc.forward(q, k, v, np.zeros(L), orc.causal_mask(L))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None], is_causal=True)[0]
    np.testing.assert_allclose(o, ref.numpy(), rtol=0, atol=1e-12)


def test_forward_zero_queries_constant_gate_closed_form():
    # q = 0: weights are the gate decay alone, w_ij ~ exp(-lam (i - j)).
    L, d, lam = 192, 8, 0.3
    rng = _rng(7)
    v = rng.standard_normal((L, d))
    c = -lam * (np.arange(L) + 1.0)
    o, lse = orc.forward(np.zeros((L, d)), rng.standard_normal((L, d)), v, c, orc.causal_mask(L))
    i = np.arange(L)
    np.testing.assert_allclose(lse, np.log((1 - np.exp(-lam * (i + 1))) / (1 - math.exp(-lam))),
                               rtol=0, atol=1e-12)
    for ii in (0, 1, 50, L - 1):
        w = np.exp(-lam * (ii - np.arange(ii + 1)))
        np.testing.assert_allclose(o[ii], (w[:, None] * v[:ii + 1]).sum(0) / w.sum(), atol=1e-12)


def test_forward_strong_forgetting_returns_values():
    rng = _rng(8)
    L, d = 256, 16
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    out = orc.run_head(q, k, v, np.full(L, -1e4, np.float32), EPS)
    np.testing.assert_allclose(out["o"], v, atol=1e-12)


@pytest.mark.parametrize("mu", [-1.0, 0.5, 2.0])
def test_pruned_mass_bound_and_output_change(mu):
    rng = _rng(9)
    L, d = 1024, 64
    q = rng.standard_normal((L, d)); k = rng.standard_normal((L, d)); v = rng.standard_normal((L, d))
    lf = _gates(rng, L, mu)
    out = orc.run_head(q, k, v, lf, EPS, method="bruteforce")
    assert out["kept"] < orc.causal_tiles(L // 64)              # pruning is active
    mass_blk = orc.pruned_mass(q, k, out["c"], out["mask"])
    mass_ent = orc.pruned_mass(q, k, out["c"], orc.entry_mask(out["c"], out["delta"]))
    assert np.all(mass_blk <= mass_ent + 1e-300)
    assert np.all(mass_ent < EPS)                             # App. A
    o_full, _ = orc.forward(q, k, v, out["c"], orc.causal_mask(L))
    bound = 2 * mass_blk * np.max(np.abs(v))
    assert np.all(np.max(np.abs(out["o"] - o_full), axis=1) <= bound + 1e-12)


def test_pruned_mass_bound_is_nearly_tight():
    # Last row: s_LL = -U, s_Lj = +U and D_Lj just below delta for every j < L-1.
    # Its entry-level pruned mass is (L-1)/L * eps (up to the gap below delta);
    # a threshold built with U instead of 2U would prune e^U times more.
    L, d, a = 256, 16, 2.0
    U = a * a / 4.0
    q = np.zeros((L, d)); q[:, 0] = a
    k = np.zeros((L, d)); k[:, 0] = a; k[L - 1, 0] = -a
    delta = orc.threshold(orc.logit_bound(orc.row_norm_sq_max(q), orc.row_norm_sq_max(k), d), L, EPS)
    lf = np.zeros(L, np.float32); lf[L - 1] = np.float32(delta - 1e-3)
    c = orc.cumsum_log_gates(lf)
    mass = orc.pruned_mass(q, k, c, orc.entry_mask(c, delta))[L - 1]
    assert mass < EPS
    assert mass > 0.95 * (L - 1) / L * EPS
    delta_1u = -(U + orc.log_len_over_eps(L, EPS))
    assert math.exp(U + U + delta_1u) * (L - 1) > EPS  # the weaker threshold breaks the bound


# --------------------------------------------------------------------------
# Backward: autograd, finite differences, identities
# --------------------------------------------------------------------------

def _torch_loss(q, k, v, log_f, mask, do):
    d = q.shape[1]
    c = torch.cumsum(log_f, 0)
    x = q @ k.T / math.sqrt(d) + (c[:, None] - c[None, :])
    x = x.masked_fill(~mask, float("-inf"))
    o = torch.softmax(x, dim=1) @ v
    return (o * do).sum()


def _case(seed, L=192, d=16, mu=-0.5):
    rng = _rng(seed)
    q = rng.standard_normal((L, d)); k = rng.standard_normal((L, d)); v = rng.standard_normal((L, d))
    do = rng.standard_normal((L, d))
    lf = _gates(rng, L, mu, sigma=1.0).astype(np.float64)
    plan = orc.plan_head(q, k, lf.astype(np.float32), EPS)
    mask = orc.block_mask(plan["row_start"], L)
    return q, k, v, do, lf, mask, plan


@pytest.mark.parametrize("seed", [0, 1])
def test_backward_matches_autograd(seed):
    q, k, v, do, lf, mask, plan = _case(20 + seed)
    assert plan["kept"] < orc.causal_tiles(q.shape[0] // 64)
    c = np.cumsum(lf)
    g = orc.backward(q, k, v, c, mask, do)
    t = [torch.tensor(a, requires_grad=True) for a in (q, k, v, lf)]
    _torch_loss(*t, torch.from_numpy(mask), torch.from_numpy(do)).backward()
    for name, tt in zip(("dq", "dk", "dv", "dlog_f"), t):
        np.testing.assert_allclose(g[name], tt.grad.numpy(), rtol=0, atol=1e-11)


def test_backward_finite_differences():
    q, k, v, do, lf, mask, _ = _case(30, L=128, d=8, mu=-1.0)
    rng = _rng(31)

    def loss(q_, k_, v_, lf_):
        o, _ = orc.forward(q_, k_, v_, np.cumsum(lf_), mask)
        return float(np.sum(o * do))

    g = orc.backward(q, k, v, np.cumsum(lf), mask, do)
    h = 1e-6
    args = [q, k, v, lf]
    for idx, name in enumerate(("dq", "dk", "dv", "dlog_f")):
        for _ in range(3):
            r = rng.standard_normal(args[idx].shape)
            plus = list(args); minus = list(args)
            plus[idx] = args[idx] + h * r; minus[idx] = args[idx] - h * r
            fd = (loss(*plus) - loss(*minus)) / (2 * h)
            an = float(np.sum(g[name] * r))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_backward_identities():
    q, k, v, do, lf, mask, _ = _case(40, L=256, d=16, mu=0.0)
    c = np.cumsum(lf)
    g = orc.backward(q, k, v, c, mask, do)
    ds = g["ds"]
    np.testing.assert_allclose(ds.sum(axis=1), 0.0, atol=1e-12)          # rowsum(dS) = 0
    L = q.shape[0]
    rect = np.array([ds[l:, :l].sum() for l in range(L)])                 # sum_{i>=l, j<l} dS_ij
    np.testing.assert_allclose(g["dlog_f"], rect, atol=1e-11)
    assert abs(g["dlog_f"][0]) <= 1e-11                                   # log f_1 never enters D


def test_backward_no_forgetting_is_sdpa_autograd():
    rng = _rng(50)
    L, d = 128, 16
    q, k, v, do = (rng.standard_normal((L, d)) for _ in range(4))
    g = orc.backward(q, k, v, np.zeros(L), orc.causal_mask(L), do)
    t = [torch.tensor(a, requires_grad=True) for a in (q, k, v)]
    o = torch.nn.functional.scaled_dot_product_attention(t[0][None], t[1][None], t[2][None], is_causal=True)[0]
    (o * torch.from_numpy(do)).sum().backward()
    for name, tt in zip(("dq", "dk", "dv"), t):
        np.testing.assert_allclose(g[name], tt.grad.numpy(), rtol=0, atol=1e-11)


# --------------------------------------------------------------------------
# Decoding with an online boundary pointer (App. F)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mu", [1.0, 3.0])
def test_decode_pointer_is_first_block_with_a_kept_entry_and_monotone(mu):
    rng = _rng(int(10 * mu))
    L = 700
    lf = workloads.log_sigmoid_f32(rng.normal(mu, 0.5, L))
    c = orc.cumsum_log_gates(lf)
    delta = -12.0
    prev = 0
    for t in range(L):
        row = orc.entry_keep(c, delta)[t]                 # eq. 3, one row
        kept_blocks = [n for n in range(t // 64 + 1) if np.any(row[n * 64:(n + 1) * 64])]
        n = orc.decode_pointer(c, t, delta)
        assert n == kept_blocks[0], t
        assert n >= prev                                 # never moves back
        prev = n
    assert prev > 0


def test_decode_row_without_pruning_is_the_causal_row():
    rng = _rng(17)
    L, d = 150, 32
    q, k, v = rng.standard_normal((3, L, d))
    lf = workloads.log_sigmoid_f32(rng.normal(2.0, 0.5, L))
    c = orc.cumsum_log_gates(lf)
    o_full, lse_full = orc.forward(q, k, v, c, orc.causal_mask(L))
    for t in (0, 63, 64, 149):
        o, lse, n = orc.decode_row(q[t], k, v, c, t, -math.inf)
        assert n == 0
        np.testing.assert_allclose(o, o_full[t], rtol=0, atol=1e-12)
        assert abs(lse - lse_full[t]) <= 1e-12


def test_decode_prunes_at_least_the_prefill_blocks_and_stays_within_eps():
    rng = _rng(23)
    L, d = 512, 64
    q, k, v = rng.standard_normal((3, L, d))
    lf = workloads.log_sigmoid_f32(rng.normal(1.0, 0.5, L))
    p = orc.plan_head(q, k, lf, EPS)
    c, delta = p["c"], p["delta"]
    c64 = c.astype(np.float64)
    full = np.where(orc.causal_mask(L), q @ k.T / math.sqrt(d) + c64[:, None] - c64[None, :], -np.inf)
    a = np.exp(full - np.max(full, axis=1, keepdims=True))
    a /= np.sum(a, axis=1, keepdims=True)
    for t in range(0, L, 37):
        n = orc.decode_pointer(c, t, delta)
        assert n >= p["row_start"][t // 64]              # one row prunes at least its block's keys
        assert np.sum(a[t, :64 * n]) < EPS                # App. A bound, L = context length
        o, _, _ = orc.decode_row(q[t], k, v, c, t, delta)
        assert np.max(np.abs(o - a[t] @ v)) <= 2 * EPS * np.max(np.abs(v))


def test_decode_ring_row_matches_brute_force_key_sets():
    """Ring cache of C positions: the attended keys are the entries j in
    [t - C + 1, t] whose block holds some entry kept by eq. 3 (or is t's own
    block), found here entry by entry; `lost` is whether such a block also has
    keys before t - C + 1."""
    rng = _rng(29)
    L, d = 400, 16
    q, k, v = rng.standard_normal((3, L, d))
    lf = workloads.log_sigmoid_f32(rng.normal(0.5, 0.5, L))
    c = orc.cumsum_log_gates(lf)
    c64 = c.astype(np.float64)
    delta = -20.0
    keep = orc.entry_keep(c, delta)
    for C in (64, 128, 192):
        prev = 0
        for t in range(0, L, 7):
            blocks = {n for n in range(t // 64 + 1)
                      if n == t // 64 or np.any(keep[t, n * 64:(n + 1) * 64])}
            held = [j for j in range(max(0, t - C + 1), t + 1) if j // 64 in blocks]
            lost_ref = any(j // 64 in blocks for j in range(0, max(0, t - C + 1)))
            x = q[t] @ k[held].T / math.sqrt(d) + c64[t] - c64[held]
            p = np.exp(x - np.max(x))
            o_ref = (p / p.sum()) @ v[held]
            o, lse, ptr, lost = orc.decode_ring_row(q[t], k, v, c, t, delta, C)
            assert lost == lost_ref, (C, t)
            np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
            assert abs(lse - (np.max(x) + math.log(p.sum()))) <= 1e-12
            assert ptr >= prev and ptr * 64 <= held[0] < (ptr + 1) * 64 + (0 if not lost else 64)
            prev = ptr
        assert prev > 0


def test_decode_ring_row_without_pruning_is_sliding_window_attention():
    """eps = 0 (delta = -inf): the ring reduces to attention over the last C
    positions, checked against torch's attention with an additive mask."""
    rng = _rng(31)
    L, d, C = 300, 32, 128
    q, k, v = rng.standard_normal((3, L, d))
    lf = workloads.log_sigmoid_f32(rng.normal(2.0, 0.5, L))
    c = orc.cumsum_log_gates(lf).astype(np.float64)
    for t in (0, 127, 128, 200, 299):
        j = np.arange(L)
        bias = np.where((j <= t) & (j >= t - C + 1), c[t] - c, -np.inf)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[t][None, None]), torch.from_numpy(k[None]), torch.from_numpy(v[None]),
            attn_mask=torch.from_numpy(bias[None, None]))[0, 0].numpy()
        o, _, ptr, lost = orc.decode_ring_row(q[t], k, v, c.astype(np.float32), t, -math.inf, C)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
        assert lost == (t >= C)
        assert ptr == max(0, t - C + 1) // 64


def test_decode_ring_row_with_room_is_decode_row():
    rng = _rng(37)
    L, d = 260, 16
    q, k, v = rng.standard_normal((3, L, d))
    lf = workloads.log_sigmoid_f32(rng.normal(1.0, 0.5, L))
    c = orc.cumsum_log_gates(lf)
    for t in (5, 100, 259):
        a = orc.decode_row(q[t], k, v, c, t, -15.0)
        b = orc.decode_ring_row(q[t], k, v, c, t, -15.0, 320)
        np.testing.assert_array_equal(a[0], b[0])
        assert a[1] == b[1] and a[2] == b[2] and b[3] is False



def test_qk_projection_matches_the_sum_written_out():
    """Q[b, h, l, e] = sum_k X[b L + l, k] W[k, h d + e] (Sec. 2), by explicit loops."""
    rng = _rng(41)
    B, L, Dm, H, d = 2, 3, 5, 2, 4
    x = rng.standard_normal((B * L, Dm))
    w = rng.standard_normal((Dm, H * d))
    q = orc.qk_projection(x, w, B, H, d)
    assert q.shape == (B, H, L, d)
    for b in range(B):
        for h in range(H):
            for l in range(L):
                for e in range(d):
                    ref = sum(x[b * L + l, k] * w[k, h * d + e] for k in range(Dm))
                    assert abs(q[b, h, l, e] - ref) <= 1e-12


def test_qk_projection_by_a_permutation_moves_columns():
    """W a permutation matrix: the projection only rearranges X's columns, exactly."""
    rng = _rng(43)
    B, L, H, d = 2, 4, 3, 4
    Dm = H * d
    x = rng.standard_normal((B * L, Dm))
    perm = rng.permutation(Dm)
    w = np.zeros((Dm, Dm))
    w[perm, np.arange(Dm)] = 1.0                  # column c of X W is column perm[c] of X
    q = orc.qk_projection(x, w, B, H, d)
    for b in range(B):
        for h in range(H):
            np.testing.assert_array_equal(q[b, h], x[b * L:(b + 1) * L][:, perm[h * d:(h + 1) * d]])


# --------------------------------------------------------------------------
# Gate projection (Sec. 2, f = sigmoid(w_f^T x + b_f)): float32 dot products in
# ascending feature order, log sigmoid in float64
# --------------------------------------------------------------------------

def test_gate_logits_dyadic_closed_form():
    # dyadic x and w whose partial sums all stay exact in float32: the logit is
    # the exact dot product plus the bias
    rng = _rng(11)
    T, Dm, H = 5, 64, 3
    x = rng.integers(-8, 9, size=(T, Dm)) / 8.0
    w = rng.integers(-8, 9, size=(Dm, H)) / 16.0
    b = np.array([1.5, -2.25, 0.0], dtype=np.float32)
    a = orc.gate_logits(x, w, b)
    for t in range(T):
        for h in range(H):
            exact = sum(Fraction(float(x[t, k])) * Fraction(float(w[k, h])) for k in range(Dm))
            assert Fraction(float(a[t, h])) == exact + Fraction(float(b[h]))


def test_gate_logits_sum_in_ascending_feature_order():
    # 1 followed by 2^-25 terms: each float32 step rounds 1 + 2^-25 back to 1, so
    # the ascending sum is exactly 1; a float64 or reversed sum would not be
    Dm = 64
    x = np.full((1, Dm), 2.0 ** -25, dtype=np.float32)
    x[0, 0] = 1.0
    w = np.ones((Dm, 1), dtype=np.float32)
    a = orc.gate_logits(x, w, np.zeros(1, dtype=np.float32))
    assert a[0, 0] == np.float32(1.0)
    assert float(np.sum(x.astype(np.float64))) != 1.0


def test_log_sigmoid_special_values():
    lf = orc.log_sigmoid(np.array([0.0, 3.0, 30.0, -30.0, -200.0], dtype=np.float32))
    assert lf[0] == np.float32(math.log(0.5))
    assert lf[1] == np.float32(math.log(1.0 / (1.0 + math.exp(-3.0))))
    # large a: log sigmoid(a) = -e^-a (1 - e^-a / 2 + ...); float32 keeps it nonzero
    assert lf[2] == np.float32(-math.exp(-30.0) * (1.0 - math.exp(-30.0) / 2.0))
    assert lf[2] < 0.0
    assert lf[3] == np.float32(-30.0 - math.log1p(math.exp(-30.0)))
    assert lf[4] == np.float32(-200.0)
    assert np.all(lf <= 0.0)


def test_gate_log_forget_layout_and_head_permutation():
    p = workloads.gate_inputs(2, 128, 64, 3, seed=12)
    x, w, b = (p[n].float().numpy() for n in ("x", "w_f", "b_f"))
    lf = orc.gate_log_forget(x, w, b, 2)
    assert lf.shape == (2, 3, 128) and lf.dtype == np.float32
    a = orc.gate_logits(x, w, b)
    np.testing.assert_array_equal(lf[1, 2, 5], orc.log_sigmoid(a[128 + 5, 2]))
    perm = [2, 0, 1]
    lf2 = orc.gate_log_forget(x, w[:, perm], b[perm], 2)
    np.testing.assert_array_equal(lf2, lf[:, perm])


def test_exact_roundings_agree_with_ieee_casts():
    """The oracle's two exact roundings to float32 (from a rational, from an
    integer times a power of two) against numpy's IEEE float64 -> float32 cast
    (round to nearest, ties to even) on values a float64 holds exactly: normal,
    subnormal, near the overflow threshold, and float32 midpoints."""
    from oracle.acp_oracle import _fraction_to_f32, _int_to_f32
    rng = np.random.default_rng(17)
    vals = list(rng.standard_normal(2000) * np.exp2(rng.integers(-160, 128, 2000).astype(np.float64)))
    for e in (-149, -140, -126, -1, 0, 60, 127):
        for m in range(1 << 23, (1 << 23) + 40):
            vals.append(math.ldexp(m + 0.5, e - 23))     # a float32 midpoint (float64 holds it)
    vals += [3.4028235677973366e38, -3.4028235677973366e38, 3.40282356779733e38, 2.0 ** -150, 2.0 ** -151]
    with np.errstate(over="ignore"):
        for v in vals:
            want = np.float32(v)
            assert _fraction_to_f32(Fraction(v)) == want, v
            m, e = math.frexp(v)
            n, lsb = int(m * 2 ** 53), e - 53                 # v = n * 2^lsb exactly
            got = _int_to_f32(n, lsb)
            assert got == want or (np.isinf(got) and np.isinf(want) and np.sign(got) == np.sign(want)), v
