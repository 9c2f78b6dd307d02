"""Forward and backward on the GPU against the oracle.

Tolerances: float32 path max |err| <= 1e-4; bfloat16 inputs with float32
accumulation max |err| <= 2e-2 on O, LSE and every gradient (relative to the
largest reference value where rows are scaled up beyond norm sqrt(d)).  Dense
comparison of every entry where the oracle finishes in seconds (tiny, small
ragged cases, strong gates, all 96 heads of the 125M-shaped layer); whole heads
by row groups for the 8k/16k-token layers; whole key blocks and sampled rows at
L = 131072."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads
from tests._helpers import EPS, ensure_built, f64, oracle_head, to_gpu

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _run_gpu(x, eps, grads=True):
    g = to_gpu(x)
    o, lse, ws = acp.forward(g["q"], g["k"], g["v"], g["log_f"], eps)
    out = {"o": o, "lse": lse, "ws": ws}
    if grads:
        dq, dk, dv, dlf = acp.backward(g["q"], g["k"], g["v"], o, g["do"], ws)
        out.update({"dq": dq, "dk": dk, "dv": dv, "dlog_f": dlf})
    torch.cuda.synchronize()
    return out


def _bound(tol, name, want):
    """The bound on one output, relative to the largest reference value where that
    exceeds 1 (see _scaled_tol): on the bfloat16 path for O, dQ, dK and dV (LSE and
    dlog f are float32 outputs and keep the absolute bound); on the float32 path
    for every output, whose float32 sums over up to L terms carry a relative error
    of order sqrt(L) 2^-24 (dlog f reaches about 60 with rows of norm 16)."""
    if tol < 1e-2 or name in ("o", "dq", "dk", "dv"):
        return _scaled_tol(tol, want)
    return tol


def _compare_head(got, ref, b, h, tol, names=("o", "lse", "dq", "dk", "dv", "dlog_f")):
    errs = {}
    for n in names:
        a = f64(got[n][b, h])
        e = float(np.max(np.abs(a - ref[n])))
        errs[n] = e
        assert np.all(np.isfinite(a)), (n, b, h)
    bad = {n: e for n, e in errs.items() if e > _bound(tol, n, ref[n])}
    assert not bad, f"head ({b},{h}) errors over the bound: {errs}"
    return errs


def _full_parity(w, heads=None, eps=None, x=None):
    eps = w.eps if eps is None else eps
    x = workloads.generate(w) if x is None else x
    got = _run_gpu(x, eps)
    B, H = w.B, w.H
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else heads
    tol = TOL[w.dtype]
    worst = {}
    for b, h in heads:
        ref = oracle_head(x, b, h, eps)
        errs = _compare_head(got, ref, b, h, tol)
        for n, e in errs.items():
            worst[n] = max(worst.get(n, 0.0), e)
        pv = acp.plan_views(got["ws"], w.B, w.H, w.L, w.d, x["q"].dtype)
        np.testing.assert_array_equal(pv["row_start"][b, h].cpu().numpy(), ref["row_start"])
    print(f"{w.describe()} eps={eps:g}: worst abs errors {worst}", flush=True)
    return got, x


def test_tiny_f32_full():
    w = workloads.WORKLOADS["tiny"]
    print(f"case: fwd/bwd {w.describe()}", flush=True)
    _full_parity(w)


def test_tiny_f32_pruning_changes_output_by_at_most_2eps():
    w = workloads.WORKLOADS["tiny"]
    x = workloads.generate(w)
    a = _run_gpu(x, EPS, grads=False)
    z = _run_gpu(x, 0.0, grads=False)
    kept = acp.plan_views(a["ws"], w.B, w.H, w.L, w.d, torch.float32)["kept"].cpu().numpy()
    assert kept[0, 0] < orc.causal_tiles(w.M)          # head 0 prunes
    vmax = float(x["v"].abs().max())
    diff = (a["o"] - z["o"]).abs().max().item()
    assert diff <= 2 * EPS * vmax + 1e-5


@pytest.mark.parametrize("B,H,L,d,mu,seed", [
    (2, 3, 320, 64, (0.5, 2.0, 8.0), 21),     # ragged: L % 128 == 64
    (1, 2, 384, 128, (1.0, 6.0), 22),
    (2, 2, 320, 128, (0.5, 3.0), 27),         # d = 128 ragged: the last workgroup's second
                                              # block of keys is past L (its waves idle)
    (1, 2, 64, 64, (1.0, 3.0), 23),           # a single block
    (1, 3, 64, 128, (0.0, 1.0, 6.0), 28),     # a single block at d = 128
    (1, 1, 1024, 64, (0.0,), 24),             # mu = 0: strongly local
])
def test_small_bf16_full(B, H, L, d, mu, seed):
    w = workloads.custom(f"small{seed}", B, H, L, d, "bf16", seed, mu=mu)
    print(f"case: fwd/bwd {w.describe()}", flush=True)
    _full_parity(w)


def _random_cases(n=8, seed=2025):
    """Seeded random shapes: ragged lengths (any multiple of 64 up to 768), odd head
    counts, both head dims, per-head gate means from strong to no forgetting, and
    pruning from light to heavy (eps up to 0.5)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        B = int(rng.integers(1, 3))
        H = int(rng.integers(1, 6 if B == 1 else 4))
        L = 64 * int(rng.integers(1, 13))
        d = int(rng.choice([64, 128]))
        mu = tuple(float(m) for m in rng.uniform(-1.0, 12.0, size=H))
        eps = float(rng.choice([math.exp(-10), math.exp(-3), 0.5]))
        out.append((B, H, L, d, mu, eps, 100 + i))
    return out


_RANDOM = _random_cases()


@pytest.mark.parametrize("B,H,L,d,mu,eps,seed", _RANDOM,
                         ids=[f"B{c[0]}H{c[1]}L{c[2]}d{c[3]}eps{c[5]:.3g}" for c in _RANDOM])
def test_random_shapes_full(B, H, L, d, mu, eps, seed):
    w = workloads.custom(f"rand{seed}", B, H, L, d, "bf16", seed, mu=mu)
    print(f"case: fwd/bwd {w.describe()} eps={eps:g}", flush=True)
    _full_parity(w, eps=eps)


def _random_long_cases(n=6, seed=2026):
    """Longer seeded shapes (1024 to 2560 positions, ragged multiples of 64), so
    that every key block's loop over query tiles runs long and the d = 128 dK/dV
    pass adds its wave pairs' partial sums after many tiles, compared in full."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        H = int(rng.integers(1, 4))
        L = 64 * int(rng.integers(16, 41))
        d = 128 if i % 2 == 0 else 64
        mu = tuple(float(m) for m in rng.uniform(-1.0, 12.0, size=H))
        eps = float(rng.choice([math.exp(-10), math.exp(-3)]))
        out.append((1, H, L, d, mu, eps, 200 + i))
    return out


_RANDOM_LONG = _random_long_cases()


@pytest.mark.parametrize("B,H,L,d,mu,eps,seed", _RANDOM_LONG,
                         ids=[f"B{c[0]}H{c[1]}L{c[2]}d{c[3]}eps{c[5]:.3g}" for c in _RANDOM_LONG])
def test_random_long_shapes_full(B, H, L, d, mu, eps, seed):
    w = workloads.custom(f"rlong{seed}", B, H, L, d, "bf16", seed, mu=mu)
    print(f"case: fwd/bwd {w.describe()} eps={eps:g}", flush=True)
    _full_parity(w, eps=eps)


def _random_mixed_cases(n=12, seed=2029):
    """Seeded shapes that also vary what the other families hold fixed: per-head
    row norms from 0.5 to 16 (logit bounds up to 2048), gate spreads from 0.1 to 2,
    eps up to 0.9, and the float32 path."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        B = int(rng.integers(1, 3))
        H = int(rng.integers(1, 5))
        L = 64 * int(rng.integers(1, 33))
        d = int(rng.choice([64, 128]))
        mu = tuple(float(m) for m in rng.uniform(-2.0, 25.0, size=H))
        eps = float(rng.choice([0.0, math.exp(-20), math.exp(-10), math.exp(-3), 0.3, 0.9]))
        dtype = "f32" if i % 4 == 3 else "bf16"
        rn = tuple(float(r) for r in rng.choice([0.5, 1.0, 4.0, 8.0, 16.0], size=H))
        sig = float(rng.choice([0.1, 0.5, 2.0]))
        out.append((B, H, L, d, dtype, mu, rn, sig, eps, 400 + i))
    return out


_RANDOM_MIXED = _random_mixed_cases()


@pytest.mark.parametrize("B,H,L,d,dtype,mu,rn,sig,eps,seed", _RANDOM_MIXED,
                         ids=[f"B{c[0]}H{c[1]}L{c[2]}d{c[3]}{c[4]}eps{c[8]:.3g}" for c in _RANDOM_MIXED])
def test_random_mixed_shapes_full(B, H, L, d, dtype, mu, rn, sig, eps, seed):
    w = workloads.custom(f"rmix{seed}", B, H, L, d, dtype, seed, mu=mu, row_norms=rn,
                         gate_sigma=sig)
    print(f"case: fwd/bwd {w.describe()} eps={eps:g}", flush=True)
    _full_parity(w, eps=eps)


def test_small_f32_d128_full():
    w = workloads.custom("f32d128", 1, 2, 192, 128, "f32", 25, mu=(0.5, 4.0))
    print(f"case: fwd/bwd {w.describe()}", flush=True)
    _full_parity(w)


def test_eps_zero_is_unpruned_attention():
    w = workloads.custom("eps0", 1, 2, 512, 64, "bf16", 26, mu=(0.5, 1.5))
    print(f"case: fwd/bwd eps=0 {w.describe()}", flush=True)
    got, _ = _full_parity(w, eps=0.0)
    kept = acp.plan_views(got["ws"], 1, 2, 512, 64, torch.bfloat16)["kept"].cpu().numpy()
    assert np.all(kept == orc.causal_tiles(8))


def test_no_forgetting_and_full_forgetting():
    w = workloads.custom("gates", 1, 2, 256, 64, "bf16", 27, mu=(2.0, 2.0))
    x = workloads.generate(w)
    x["log_f"] = torch.zeros_like(x["log_f"])
    _full_parity(w, x=x)
    # f = e^-200: every key but the query itself is damped by e^-200 per step,
    # so O = V row by row
    x = workloads.generate(w)
    x["log_f"] = torch.full_like(x["log_f"], -200.0)
    got, _ = _full_parity(w, x=x)
    np.testing.assert_allclose(f64(got["o"][0]), f64(x["v"][0]), atol=2e-2)


@pytest.mark.parametrize("dtype,lf,norm", [
    ("bf16", -80.0, None),       # N(0,1) rows: only the diagonal blocks are kept
    ("bf16", -1000.0, None),
    ("bf16", -80.0, 15.97),      # U = 31.9, fixed stabiliser: block (m, m-1) kept too
    ("bf16", -200.0, 40.0),      # U = 200, online maximum: block (m, m-1) kept too
    ("bf16", -30.0, 24.0),       # U = 72, online maximum: block (m, m-1) kept too
    ("f32", -200.0, None),
    ("f32", -80.0, 16.2),        # U = 32.8: block (m, m-1) kept too
])
def test_strong_forgetting(dtype, lf, norm):
    """Gates far below the generator's range (f = e^-30 .. e^-1000, constant), the
    ABI's domain being any finite log f <= 0: every entry of every kept block must
    meet the tolerance, including the blocks next to the diagonal that a large
    logit bound keeps.  Gradients scale with the row norm, so with scaled rows the
    bound is relative to the largest reference value."""
    L = 1024 if dtype == "bf16" else 256
    w = workloads.custom(f"strong{int(-lf)}", 1, 2, L, 64, dtype, 31,
                         row_norms=None if norm is None else (norm,))
    print(f"case: fwd/bwd log f = {lf} row norm {norm} {w.describe()}", flush=True)
    x = workloads.generate(w)
    x["log_f"] = torch.full_like(x["log_f"], lf)
    got = _run_gpu(x, w.eps)
    pv = acp.plan_views(got["ws"], 1, 2, L, 64, x["q"].dtype)
    kept = pv["kept"].cpu().numpy()
    M = L // 64
    # scaled rows keep the block before the diagonal one as well
    assert np.all(kept == (M if norm is None else 2 * M - 1)), kept
    tol = TOL[dtype]
    for h in range(2):
        ref = oracle_head(x, 0, h, w.eps)
        np.testing.assert_array_equal(pv["row_start"][0, h].cpu().numpy(), ref["row_start"])
        for n in ("o", "lse", "dq", "dk", "dv", "dlog_f"):
            a = f64(got[n][0, h])
            assert np.all(np.isfinite(a)), (h, n)
            err = float(np.max(np.abs(a - ref[n])))
            scale = 1.0 if norm is None else max(1.0, float(np.max(np.abs(ref[n]))))
            assert err <= tol * scale, (h, n, err, scale)


def test_125m_every_head_dense():
    """The 125M-shaped layer at full size, in the benchmark's launch
    configuration: all 96 heads against the dense oracle, entry by entry."""
    w = workloads.WORKLOADS["125m"]
    print(f"case: fwd/bwd all heads {w.describe()}", flush=True)
    x = workloads.generate(w)
    got = _run_gpu(x, w.eps)
    tol = TOL[w.dtype]
    pv = acp.plan_views(got["ws"], w.B, w.H, w.L, w.d, x["q"].dtype)
    worst = {}
    for b in range(w.B):
        for h in range(w.H):
            ref = oracle_head(x, b, h, w.eps)
            np.testing.assert_array_equal(pv["row_start"][b, h].cpu().numpy(), ref["row_start"])
            for n, e in _compare_head(got, ref, b, h, tol).items():
                worst[n] = max(worst.get(n, 0.0), e)
        print(f"  batch {b}: 12 heads ok, worst so far {worst}", flush=True)


def test_forward_is_deterministic():
    w = workloads.custom("det", 2, 2, 1024, 64, "bf16", 28)
    x = workloads.generate(w)
    a = _run_gpu(x, w.eps)
    b = _run_gpu(x, w.eps)
    for n in ("o", "lse", "dq", "dk", "dv", "dlog_f"):
        assert torch.equal(a[n], b[n]), n


def test_side_stream_matches_default_stream():
    """Every launch goes to the caller's stream: on a side stream whose inputs are
    produced on that stream just before the call, fwd + bwd give the same bits as
    on the default stream, at d = 64 and d = 128."""
    for d, seed in ((64, 41), (128, 42)):
        w = workloads.custom("strm", 2, 3, 1088, d, "bf16", seed, mu=(0.5, 2.0, 8.0))
        print(f"case: side stream {w.describe()}", flush=True)
        x = workloads.generate(w)
        ref = _run_gpu(x, w.eps)
        g = to_gpu(x)
        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            # copies queued on the side stream: a launch on any other stream could
            # read them before they land
            h = {n: g[n].clone() for n in ("q", "k", "v", "log_f", "do")}
            o, lse, ws = acp.forward(h["q"], h["k"], h["v"], h["log_f"], w.eps)
            dq, dk, dv, dlf = acp.backward(h["q"], h["k"], h["v"], o, h["do"], ws)
        side.synchronize()
        got = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv, "dlog_f": dlf}
        for n, t in got.items():
            assert torch.equal(t, ref[n]), (d, n)


def _check_sampled(w, x, got, heads, method="bruteforce"):
    """Sampled rows (O, lse, dQ) and the last key block (dK, dV, dlog f) of some
    heads against the oracle's row and column functions."""
    tol = TOL[w.dtype]
    L = w.L
    for n in ("o", "lse", "dq", "dk", "dv", "dlog_f"):
        assert torch.isfinite(got[n].float()).all(), n
    rng = np.random.default_rng(w.seed)
    rows = sorted({0, 63, 64, L // 2, L - 65, L - 64, L - 1, *rng.integers(0, L, 5).tolist()})
    tail = list(range(L - 64, L))
    for b, h in heads:
        q = x["q"][b, h].float().numpy().astype(np.float64)
        k = x["k"][b, h].float().numpy().astype(np.float64)
        v = x["v"][b, h].float().numpy().astype(np.float64)
        do = x["do"][b, h].float().numpy().astype(np.float64)
        plan = orc.plan_head(q, k, x["log_f"][b, h].numpy(), w.eps, method=method)
        rs, c = plan["row_start"], plan["c"]
        pv = acp.plan_views(got["ws"], w.B, w.H, w.L, w.d, x["q"].dtype)
        np.testing.assert_array_equal(pv["row_start"][b, h].cpu().numpy(), rs)
        o, lse = orc.forward_rows(q, k, v, c, rs, rows)
        dq, rsum = orc.backward_rows(q, k, v, c, rs, do, rows)
        assert np.max(np.abs(f64(got["o"][b, h])[rows] - o)) <= tol
        assert np.max(np.abs(f64(got["lse"][b, h])[rows] - lse)) <= tol
        assert np.max(np.abs(f64(got["dq"][b, h])[rows] - dq)) <= tol
        dk, dv, csum = orc.backward_cols(q, k, v, c, rs, do, tail)
        assert np.max(np.abs(f64(got["dk"][b, h])[tail] - dk)) <= tol
        assert np.max(np.abs(f64(got["dv"][b, h])[tail] - dv)) <= tol
        _, rs_tail = orc.backward_rows(q, k, v, c, rs, do, tail)
        dlf_tail = np.cumsum((rs_tail - csum)[::-1])[::-1]
        assert np.max(np.abs(f64(got["dlog_f"][b, h])[tail] - dlf_tail)) <= tol
    # every row of P sums to one, so sum_j dV_j = sum_i dO_i for every head
    sdv = got["dv"].double().sum(dim=2).cpu()
    sdo = x["do"].double().sum(dim=2)
    assert torch.max(torch.abs(sdv - sdo)).item() <= 0.02 * math.sqrt(L)


def _head_f64(x, b, h):
    return tuple(workloads.to_f64(x[n][b, h]) for n in ("q", "k", "v", "do"))


def _scaled_tol(tol, ref):
    """bf16 outputs carry a relative rounding of 2^-9 (half an ulp: 2^-6 = 0.016
    for values in [4, 8)), so where an output exceeds 1 in size (rows scaled
    beyond norm sqrt(d), or attention concentrated on a few keys by strong
    forgetting, which makes dV approach dO) the bound is taken relative to the
    largest reference value."""
    return tol * max(1.0, float(np.max(np.abs(ref))))


def _check_whole_heads(w, x, got, heads):
    """Every query row and every key column of the given heads against the dense
    oracle evaluated a group of rows at a time (backward_row_range over all rows:
    O, LSE, dQ per row; dK, dV and the column sums per key; dlog f from the row
    and column sums)."""
    tol = TOL[w.dtype]
    pv = acp.plan_views(got["ws"], w.B, w.H, w.L, w.d, x["q"].dtype)
    for b, h in heads:
        q, k, v, do = _head_f64(x, b, h)
        plan = orc.plan_head(q, k, x["log_f"][b, h].numpy(), w.eps, method="topright")
        np.testing.assert_array_equal(pv["row_start"][b, h].cpu().numpy(), plan["row_start"])
        r = orc.backward_row_range(q, k, v, plan["c"], plan["row_start"], do, 0, w.L)
        ref = {"o": r["o"], "lse": r["lse"], "dq": r["dq"], "dk": r["dk"], "dv": r["dv"],
               "dlog_f": np.cumsum((r["rowsum"] - r["colsum"])[::-1])[::-1]}
        errs = {}
        for n, want in ref.items():
            a = f64(got[n][b, h])
            errs[n] = float(np.max(np.abs(a - want)))
            assert errs[n] <= _bound(tol, n, want), (b, h, n, errs[n])
        print(f"  head ({b},{h}) kept {plan['kept']}: {errs}", flush=True)


def _check_key_blocks(w, x, got, b, h, blocks):
    """dK, dV and dlog f of whole 64-key blocks against the oracle, from every
    query row that keeps them (rows 64 n .. 64 col_end[n] + 63): the columns'
    sums over all their kept query blocks, and dlog f at the block's first key by
    the rectangle identity (the same rows hold every kept key before it)."""
    tol = TOL[w.dtype]
    q, k, v, do = _head_f64(x, b, h)
    plan = orc.plan_head(q, k, x["log_f"][b, h].numpy(), w.eps, method="topright")
    ce = plan["col_end"]
    for n in blocks:
        l = 64 * n
        r = orc.backward_row_range(q, k, v, plan["c"], plan["row_start"], do, l,
                                   64 * int(ce[n]) + 64, ls=(l,))
        cols = slice(l, l + 64)
        for name, want, gotv in (("dk", r["dk"][cols], got["dk"][b, h, cols]),
                                 ("dv", r["dv"][cols], got["dv"][b, h, cols])):
            err = float(np.max(np.abs(f64(gotv) - want)))
            assert err <= _scaled_tol(tol, want), (b, h, n, name, err)
        err = abs(float(got["dlog_f"][b, h, l]) - r["rect"][l])
        assert err <= tol, (b, h, n, "dlog_f", err)
        print(f"  head ({b},{h}) key block {n} (kept by {int(ce[n]) - n + 1} query blocks) ok",
              flush=True)


@pytest.mark.parametrize("name", ["360m", "760m", "adv"])
def test_long_layers_whole_heads(name):
    """The 8k- and 16k-token layers at full size in the benchmark's launch
    configuration: a fast- and a slow-decay head compared in full (every row,
    every key column), a third head on sampled rows and its last key block, and
    sum_j dV_j = sum_i dO_i on every head."""
    w = workloads.WORKLOADS[name]
    print(f"case: fwd/bwd whole heads {w.describe()}", flush=True)
    x = workloads.generate(w)
    got = _run_gpu(x, w.eps)
    mu = np.asarray(x["mu"])
    if name == "adv":
        # (mu 0, rows of norm 16): fast decay, largest bound; (mu 20, norm 16): slow
        heads = [(0, 5), (1, 14)]
    else:
        heads = [(0, int(np.argmin(mu))), (w.B - 1, int(np.argmax(mu)))]
    _check_whole_heads(w, x, got, heads)
    rng = np.random.default_rng(w.seed)
    _check_sampled(w, x, got, [(0, int(rng.integers(w.H)))])


@pytest.mark.parametrize("d", [64, 128])
def test_max_length_sampled(d):
    """L = 131072, the longest sequence the ABI takes (2048 pruning blocks per
    head; stage 1 off its register path, 1024 row-norm chunks), at both head
    sizes: a fast- and a slow-decay head, sampled against the oracle (its
    boundary decided on the blocks' top-right entries, since the entry-by-entry
    form needs L x L)."""
    w = workloads.custom(f"maxlen{d}", 1, 2, 64 * 2048, d, "bf16", 71, mu=(1.0, 6.0))
    print(f"case: fwd/bwd sampled {w.describe()}", flush=True)
    x = workloads.generate(w)
    got = _run_gpu(x, w.eps)
    _check_sampled(w, x, got, [(0, 0), (0, 1)], method="topright")
    # whole key blocks: first, middle and last - 8 of the fast head (each kept by
    # a few query blocks), last - 8 of the slow one (kept by the 8 after it)
    _check_key_blocks(w, x, got, 0, 0, [0, 1024, 2039])
    _check_key_blocks(w, x, got, 0, 1, [2039])


def test_max_head_count_sampled():
    """B * H = 65535, the most heads the ABI takes (grid sizes, per-head tables
    and the head-order schedule at their limit), L = 128: heads with strong
    forgetting (block (1, 0) pruned), moderate and weak, sampled against the
    oracle head by head; every head must keep sum_j dV_j = sum_i dO_i."""
    w = workloads.custom("maxheads", 3, 21845, 128, 64, "bf16", 73, mu=(-80.0, 0.0, 6.0))
    print(f"case: fwd/bwd sampled {w.describe()}", flush=True)
    x = workloads.generate(w)
    got = _run_gpu(x, w.eps)
    kept = acp.plan_views(got["ws"], w.B, w.H, w.L, w.d, x["q"].dtype)["kept"].cpu().numpy()
    want = np.where(np.arange(w.H) % 3 == 0, 2, 3)   # log f near -80 prunes block (1, 0)
    np.testing.assert_array_equal(kept.reshape(w.B, w.H), np.broadcast_to(want, (w.B, w.H)))
    tol = TOL[w.dtype]
    rng = np.random.default_rng(w.seed)
    heads = [(0, 0), (0, 1), (0, 2), (w.B - 1, w.H - 1)] + \
        [(int(rng.integers(w.B)), int(rng.integers(w.H))) for _ in range(4)]
    for b, h in heads:
        _compare_head(got, oracle_head(x, b, h, w.eps), b, h, tol)
    sdv = got["dv"].double().sum(dim=2).cpu()
    sdo = x["do"].double().sum(dim=2)
    assert torch.max(torch.abs(sdv - sdo)).item() <= 0.02 * math.sqrt(w.L)


@pytest.mark.parametrize("d", [64, 128])
def test_online_max_variant_for_large_logit_bound(d):
    # rho_q ~ 40 makes U ~ 50 > 32 on head 0, so its forward takes the
    # online-maximum variant; head 1 keeps the fixed stabiliser.  Gradients
    # scale with |q|, so the bound is 2e-2 relative to the largest reference value.
    w = workloads.custom("bigU", 1, 2, 384, d, "bf16", 29, mu=(1.0, 4.0))
    print(f"case: online maximum {w.describe()}", flush=True)
    x = workloads.generate(w)
    q = x["q"].float()
    q[0, 0] = q[0, 0] / q[0, 0].norm(dim=-1, keepdim=True) * 40.0
    x["q"] = q.bfloat16()
    got = _run_gpu(x, w.eps)
    u = acp.plan_views(got["ws"], 1, 2, 384, d, torch.bfloat16)["bound_u"].cpu().numpy()
    assert u[0, 0] > 32.0 and u[0, 1] < 32.0
    for h in range(2):
        ref = oracle_head(x, 0, h, w.eps)
        for n in ("o", "lse", "dq", "dk", "dv", "dlog_f"):
            err = float(np.max(np.abs(f64(got[n][0, h]) - ref[n])))
            scale = max(1.0, float(np.max(np.abs(ref[n]))))
            assert err <= 2e-2 * scale, (h, n, err, scale)
