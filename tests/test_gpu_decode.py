"""Decoding with ACP on the GPU (App. F, inference-time ACP) against the oracle: after a
prompt, each step's output, log-sum-exp and boundary pointer must match the
oracle's single-row decoding, with the threshold sized for L_max and the bound
from QK-norm scales; a ring cache too small for the kept window must report it
and attend to what it still holds."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2504_06949_amd import acp, workloads
from tests._helpers import EPS, ensure_built, head_inputs, to_gpu

pytestmark = pytest.mark.gpu

TOL = {"bf16": (2e-2, 1e-3), "f32": (1e-4, 1e-4)}   # (O, lse) max abs error


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def _token(g, name, t):
    # a fresh allocation: a slice that is already contiguous (B = H = 1) would
    # keep the offset of position t and miss the ABI's 16-byte alignment
    return g[name][:, :, t].clone(memory_format=torch.contiguous_format)


def _run(w, L0, C, eps, L_max, poke=None):
    """Prompt of L0 tokens, then one step per remaining position of the workload.
    Returns the inputs, the per-step GPU results and the decoder's final views."""
    x = workloads.generate(w, with_grad=False)
    g = to_gpu(x)
    dec = acp.Decoder(w.B, w.H, C, w.d, dtype=g["k"].dtype)
    dec.init(g["k"][:, :, :L0].contiguous(), g["v"][:, :, :L0].contiguous(),
             g["log_f"][:, :, :L0].contiguous(), g["gamma_q"], g["gamma_k"], eps, L_max)
    vw = dec.views()
    init = {n: vw[n].clone() for n in ("flags", "delta")}
    init["pointer"] = dec.current_pointer().clone()
    steps = []
    for t in range(L0, w.L):
        lf = _token(g, "log_f", t)
        if poke is not None:
            poke(t, lf)
        o, lse = dec.step(_token(g, "q", t), _token(g, "k", t), _token(g, "v", t), lf)
        steps.append((t, o, lse, dec.current_pointer().clone(), vw["flags"].clone()))
    torch.cuda.synchronize()
    steps = [(t, o.double().cpu().numpy(), lse.double().cpu().numpy(), p.cpu(), f.cpu())
             for t, o, lse, p, f in steps]
    init = {n: v.cpu() for n, v in init.items()}
    fin = {n: v.cpu() for n, v in vw.items()}
    fin["cum_now"] = dec.current_cum().cpu()
    return x, init, steps, fin


def _check(w, L0, C, eps, L_max, expect_lost=None):
    print(f"case: decode {w.describe()} L0={L0} C={C} eps={eps:.3g} L_max={L_max}", flush=True)
    x, init, steps, fin = _run(w, L0, C, eps, L_max)
    tol_o, tol_l = TOL[w.dtype]
    c_ref = orc.cumsum_log_gates(x["log_f"].numpy())
    lost_any = False
    worst = (0.0, 0.0)
    for b in range(w.B):
        for h in range(w.H):
            q, k, v, _, _ = head_inputs(x, b, h)
            U = orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), w.d)
            delta = orc.threshold(U, L_max, eps)
            assert float(init["delta"][b, h]) == delta
            _, _, p0, lost = orc.decode_ring_row(q[L0 - 1], k, v, c_ref[b, h], L0 - 1, delta, C)
            assert int(init["pointer"][b, h]) == p0, (b, h)
            sticky = lost
            assert int(init["flags"][b, h]) == (16 if sticky else 0), (b, h)
            for t, o, lse, ptr, fl in steps:
                o_ref, lse_ref, p_ref, lost = orc.decode_ring_row(q[t], k, v, c_ref[b, h], t,
                                                                  delta, C)
                sticky = sticky or lost
                assert int(ptr[b, h]) == p_ref, (b, h, t)
                assert int(fl[b, h]) == (16 if sticky else 0), (b, h, t)
                eo = float(np.max(np.abs(o[b, h] - o_ref)))
                el = abs(float(lse[b, h]) - lse_ref)
                assert eo <= tol_o and el <= tol_l, (b, h, t, eo, el)
                worst = (max(worst[0], eo), max(worst[1], el))
            lost_any = lost_any or sticky
            # the ring's c and the float32 rounding of the running sum
            T = w.L
            for pos in range(max(0, T - C), T):
                assert float(fin["c"][b, h, pos % C]) == float(c_ref[b, h, pos])
            # the pair is the exact sum, its leading part that sum's float64 rounding
            hi, lo = (float(v) for v in fin["cum_now"][b, h])
            exact = sum(Fraction(float(v)) for v in x["log_f"][b, h, :T].numpy())
            assert Fraction(hi) + Fraction(lo) == exact and hi == float(exact), (b, h)
            kc = fin["k_cache"][b, h]
            pos = T - 1
            assert torch.equal(kc[pos % C], x["k"][b, h, pos])
    print(f"  max errors: O {worst[0]:.3g}, lse {worst[1]:.3g}; a kept key lost: {lost_any}",
          flush=True)
    if expect_lost is not None:
        assert lost_any == expect_lost
    return steps


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("f32", 64), ("bf16", 128), ("f32", 128)])
def test_decode_matches_oracle(dtype, d):
    w = workloads.custom("dec", 2, 4, 448, d, dtype, 41, mu=(0.0, 1.0, 3.0, 20.0), qk_norm=True)
    steps = _check(w, 333, 512, EPS, 4096, expect_lost=False)
    # strongly decaying heads move their pointer while the step runs
    assert int(steps[-1][3][0, 0]) > int(steps[0][3][0, 0]) > 0


def _random_decode_cases(n=6, seed=2027):
    """Seeded random decoding set-ups: head counts, head dims, dtypes, prompt
    lengths from 1 token up (not multiples of 64), rings from smaller than the
    kept window to larger than the context, eps from none to heavy pruning, and
    L_max from the final length up to four times it."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        B = int(rng.integers(1, 3))
        H = int(rng.integers(1, 6))
        d = int(rng.choice([64, 128]))
        dtype = "f32" if i == n - 1 else "bf16"
        L0 = int(rng.integers(1, 600))
        L = L0 + int(rng.integers(20, 90))
        C = int(rng.choice([64, 192, 512, 1024]))
        eps = float(rng.choice([0.0, math.exp(-10), math.exp(-3)]))
        L_max = L * int(rng.integers(1, 5))
        mu = tuple(float(m) for m in rng.uniform(-1.0, 20.0, size=H))
        out.append((B, H, d, dtype, L0, L, C, eps, L_max, mu, 300 + i))
    return out


_RANDOM_DEC = _random_decode_cases()


@pytest.mark.parametrize("B,H,d,dtype,L0,L,C,eps,L_max,mu,seed", _RANDOM_DEC,
                         ids=[f"B{c[0]}H{c[1]}d{c[2]}{c[3]}L0_{c[4]}C{c[6]}" for c in _RANDOM_DEC])
def test_decode_random_setups(B, H, d, dtype, L0, L, C, eps, L_max, mu, seed):
    w = workloads.custom("decr", B, H, L, d, dtype, seed, mu=mu, qk_norm=True)
    _check(w, L0, C, eps, L_max)


def test_decode_wide_gate_spans_stay_exact():
    """Logits N(mu, 8): the prompt's cumulative sums span 69-94 bits and the
    running sum reaches 99 bits during the steps, past the 53 bits a float64 holds.
    The set-up's double-double scan and each step's pair addition keep c and the
    running sum exact (no flag), and the outputs follow the oracle."""
    w = workloads.custom("decw", 1, 4, 448, 64, "bf16", 45, mu=(5.0, 15.0, 25.0, 35.0),
                         gate_sigma=8.0, qk_norm=True)
    lf = workloads.generate(w, with_grad=False)["log_f"].numpy()
    assert min(orc.cumsum_span_bits(lf[0, h, :333]) for h in range(w.H)) > 53
    _check(w, 333, 512, EPS, 4096, expect_lost=False)


def test_decode_ring_smaller_than_window():
    """C = 128: heads with a long kept window lose keys (flag bit 4) and attend to
    the kept keys the ring still holds; the fast-decaying head fits."""
    w = workloads.custom("dec", 1, 4, 448, 64, "bf16", 42, mu=(0.0, 1.0, 3.0, 20.0), qk_norm=True)
    _check(w, 200, 128, EPS, 4096, expect_lost=True)


def test_decode_without_pruning_and_short_prompt():
    """eps = 0: nothing is pruned, the pointer stays 0 and every step is the full
    causal row; a prompt shorter than one block."""
    w = workloads.custom("dec", 1, 2, 192, 64, "bf16", 43, mu=(0.0, 3.0), qk_norm=True)
    steps = _check(w, 10, 256, 0.0, 1 << 20, expect_lost=False)
    assert all(int(p.max()) == 0 for _, _, _, p, _ in steps)


def test_decode_flags_a_positive_gate():
    w = workloads.custom("dec", 1, 2, 128, 64, "bf16", 44, mu=(1.0, 3.0), qk_norm=True)

    def poke(t, lf):
        if t == 100:
            lf[0, 1] = 0.25

    _, init, steps, fin = _run(w, 64, 128, EPS, 4096, poke=poke)
    assert int(init["flags"].max()) == 0
    assert int(fin["flags"][0, 1]) & 1 and int(fin["flags"][0, 0]) == 0
    assert all(int(fl[0, 1]) & 1 == (1 if t >= 100 else 0) for t, _, _, _, fl in steps)


def test_decode_flags_a_rounding_step():
    """Flag bit 2 in the steps: a gate of -1e-30 fits into the running pair's low
    part exactly (no flag); a later gate of -3e-20 would need 59 bits there, so that
    addition rounds and the flag is set from that step on.  The other head stays
    clean."""
    w = workloads.custom("dec", 1, 2, 128, 64, "bf16", 46, mu=(1.0, 3.0), qk_norm=True)

    def poke(t, lf):
        if t == 80:
            lf[0, 1] = -1e-30
        if t == 90:
            lf[0, 1] = -3e-20

    print("case: decode flag bit 2 at a rounding step", flush=True)
    _, init, steps, fin = _run(w, 64, 128, EPS, 4096, poke=poke)
    assert int(init["flags"].max()) == 0
    for t, _, _, _, fl in steps:
        assert int(fl[0, 0]) == 0, t
        assert int(fl[0, 1]) == (acp.FLAG_INEXACT_CUMSUM if t >= 90 else 0), (t, int(fl[0, 1]))


def test_decode_steps_captured_in_a_graph_match_eager():
    """Eight steps captured in a HIP graph: each replay (after an eager re-init of
    the state in between) must give exactly the eager outputs and state."""
    w = workloads.custom("dec", 2, 3, 320, 64, "bf16", 45, mu=(0.0, 1.0, 6.0), qk_norm=True)
    x = workloads.generate(w, with_grad=False)
    g = to_gpu(x)
    L0, n = 290, 8
    prompt = [g[n_][:, :, :L0].contiguous() for n_ in ("k", "v", "log_f")]
    toks = [[_token(g, n_, t) for n_ in ("q", "k", "v", "log_f")] for t in range(L0, L0 + n)]
    eager = acp.Decoder(w.B, w.H, 256, w.d).init(*prompt, g["gamma_q"], g["gamma_k"], EPS, 4096)
    ref = [tuple(r.clone() for r in eager.step(*tk)) for tk in toks]
    ref_ptr = eager.current_pointer().clone()

    dec = acp.Decoder(w.B, w.H, 256, w.d).init(*prompt, g["gamma_q"], g["gamma_k"], EPS, 4096)
    outs = [(torch.empty_like(o), torch.empty_like(l)) for o, l in ref]
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for tk, buf in zip(toks, outs):
            dec.step(*tk, out=buf)
    for rep in range(3):
        print(f"case: decode graph replay {rep}", flush=True)
        dec.init(*prompt, g["gamma_q"], g["gamma_k"], EPS, 4096)   # eager work in between
        torch.cuda.synchronize()
        for buf in outs:
            buf[0].fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        dec.t = L0 + n
        for (o, l), (ro, rl) in zip(outs, ref):
            assert torch.equal(o, ro) and torch.equal(l, rl), rep
        assert torch.equal(dec.current_pointer(), ref_ptr)


def test_decode_at_the_bench_shape_sampled():
    """The bench's decoding configuration (B=8, H=12, d=64, prompt 4096, ring and
    L_max 8192): four steps, every head's pointer and three heads' outputs against
    the oracle."""
    w = workloads.custom("dec", 8, 12, 4160, 64, "bf16", 1, qk_norm=True)
    print(f"case: decode at the bench shape {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    g = to_gpu(x)
    L0, C, L_max = 4096, 8192, 8192
    dec = acp.Decoder(w.B, w.H, C, w.d).init(g["k"][:, :, :L0].contiguous(),
                                              g["v"][:, :, :L0].contiguous(),
                                              g["log_f"][:, :, :L0].contiguous(),
                                              g["gamma_q"], g["gamma_k"], EPS, L_max)
    steps = []
    for t in range(L0, L0 + 4):
        o, lse = dec.step(_token(g, "q", t), _token(g, "k", t), _token(g, "v", t),
                          _token(g, "log_f", t))
        steps.append((t, o.double().cpu().numpy(), lse.double().cpu().numpy(),
                      dec.current_pointer().cpu().numpy()))
    flags = dec.views()["flags"].cpu().numpy()
    assert flags.max() == 0
    c_ref = orc.cumsum_log_gates(x["log_f"].numpy())
    for b in range(w.B):
        for h in range(w.H):
            U = orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), w.d)
            delta = orc.threshold(U, L_max, EPS)
            for t, o, lse, ptr in steps:
                assert int(ptr[b, h]) == orc.decode_pointer(c_ref[b, h], t, delta), (b, h, t)
    for b, h in ((0, 0), (3, 5), (7, 11)):
        q, k, v, _, _ = head_inputs(x, b, h)
        U = orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), w.d)
        delta = orc.threshold(U, L_max, EPS)
        for t, o, lse, _ in steps:
            o_ref, lse_ref, _ = orc.decode_row(q[t], k, v, c_ref[b, h], t, delta)
            assert float(np.max(np.abs(o[b, h] - o_ref))) <= 2e-2 and abs(lse[b, h] - lse_ref) <= 1e-3


def test_decode_long_ring_sampled():
    """A ring of 66048 positions after a 66000-token prompt: each step launches
    258 key chunks per head, more than 256, so their partial sums go through the
    1024-thread variant of the merge kernel.  Three steps, every head's pointer
    and output against the oracle."""
    w = workloads.custom("declong", 1, 4, 66003, 64, "bf16", 5, qk_norm=True, mu=(1.0, 3.0, 6.0, 9.0))
    print(f"case: decode long ring {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    g = to_gpu(x)
    L0, C, L_max = 66000, 66048, 131072
    dec = acp.Decoder(w.B, w.H, C, w.d).init(g["k"][:, :, :L0].contiguous(),
                                              g["v"][:, :, :L0].contiguous(),
                                              g["log_f"][:, :, :L0].contiguous(),
                                              g["gamma_q"], g["gamma_k"], EPS, L_max)
    steps = []
    for t in range(L0, L0 + 3):
        o, lse = dec.step(_token(g, "q", t), _token(g, "k", t), _token(g, "v", t),
                          _token(g, "log_f", t))
        steps.append((t, o.double().cpu().numpy(), lse.double().cpu().numpy(),
                      dec.current_pointer().cpu().numpy()))
    assert dec.views()["flags"].cpu().numpy().max() == 0
    c_ref = orc.cumsum_log_gates(x["log_f"].numpy())
    for h in range(w.H):
        q, k, v, _, _ = head_inputs(x, 0, h)
        U = orc.logit_bound_qknorm(float(x["gamma_q"][h]), float(x["gamma_k"][h]), w.d)
        delta = orc.threshold(U, L_max, EPS)
        for t, o, lse, ptr in steps:
            assert int(ptr[0, h]) == orc.decode_pointer(c_ref[0, h], t, delta), (h, t)
            o_ref, lse_ref, _ = orc.decode_row(q[t], k, v, c_ref[0, h], t, delta)
            assert float(np.max(np.abs(o[0, h] - o_ref))) <= 2e-2, (h, t)
            assert abs(lse[0, h] - lse_ref) <= 1e-3, (h, t)
