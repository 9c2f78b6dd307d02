"""Seeded synthetic inputs for FoX attention with adaptive computation pruning.

This module draws the inputs only: Q, K, V, the per-head log forget gates and
the upstream gradient dO.  It holds none of the method's arithmetic (no cumsum,
no bound, no threshold, no attention), so that the oracle and the HIP path can
both be fed from it without sharing any of the computation they are compared on.

Shapes follow the paper's model table (App. B, Table 2: d_head = 64; 12/16/24
heads for the 125M/360M/760M models) and its training batches (App. B: each
gradient-accumulation step holds 32k tokens, so B*L = 32768 per GPU).  The
trained LongCrawl64 activations the paper measures on are not available; random
N(0,1) queries/keys/values with gate logits a ~ N(mu_h, 0.5) stand in for them.
The forget gate is f = sigmoid(a) (Sec. 2, eq. 1); log f = -softplus(-a) is
evaluated in float64 and rounded once to float32, so that strongly remembering
gates (mu = 20) do not round to log f = 0.

Draw order (torch.Generator on the CPU): per-head mu, Q, K, V, gate noise, dO,
then (QK-norm workloads only) the per-head norm weights.  Floating draws are
float32 N(0,1) (rounded to nearest-even bfloat16 for the bf16 workloads).

QK-norm workloads stand in for a model with normalised queries and keys (the
setting of the paper's App. E): every q and k row is RMS-normalised and scaled
elementwise by a per-head weight vector drawn from U[0.5, 1.5]^d; gamma_q[h] and
gamma_k[h] are the largest weight magnitudes.  The normalised row is shrunk by
1 - 2^-7 first, so that rounding to bfloat16 (at most 2^-9 per element) keeps
|q| <= gamma_q sqrt(d).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    L: int
    d: int
    dtype: str  # "f32" or "bf16"
    seed: int
    mu: Optional[Sequence[float]] = None  # per-head gate mean; None: U[1,10] per head
    gate_sigma: float = 0.5
    row_norms: Optional[Sequence[float]] = None  # per-head q/k row L2 norm (cycled)
    eps: float = math.exp(-10.0)
    qk_norm: bool = False  # RMS-normalised, weight-scaled q/k rows (see the module note)

    @property
    def M(self) -> int:
        return self.L // 64

    def describe(self) -> str:
        return (f"{self.name}: B={self.B} H={self.H} L={self.L} d={self.d} {self.dtype}, "
                f"seed={self.seed}")


# The five workloads: a tiny fp32 case, three single layers shaped like the
# paper's 125M / 360M / 760M models at L = 4k / 8k / 16k, and a d=128 sweep
# whose heads span nearly-all-pruned to nothing-pruned.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 2, 512, 64, "f32", 0, mu=(2.0, 8.0)),
    "125m": Workload("125m", 8, 12, 4096, 64, "bf16", 1),
    "360m": Workload("360m", 4, 16, 8192, 64, "bf16", 2),
    "760m": Workload("760m", 2, 24, 16384, 64, "bf16", 3),
    "adv": Workload("adv", 2, 16, 16384, 128, "bf16", 4,
                    mu=tuple((0.0, 3.0, 6.0, 12.0, 20.0)[h % 5] for h in range(16)),
                    row_norms=tuple((1.0, 4.0, 16.0)[h % 3] for h in range(16))),
}


def custom(name: str, B: int, H: int, L: int, d: int, dtype: str, seed: int,
           mu=None, row_norms=None, gate_sigma: float = 0.5, qk_norm: bool = False) -> Workload:
    return Workload(name, B, H, L, d, dtype, seed, mu=None if mu is None else tuple(mu),
                    gate_sigma=gate_sigma,
                    row_norms=None if row_norms is None else tuple(row_norms), qk_norm=qk_norm)


def _torch_dtype(dt: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dt]


def log_sigmoid_f32(a: np.ndarray) -> np.ndarray:
    """log(sigmoid(a)) = -softplus(-a), evaluated in float64, rounded to float32."""
    a = np.asarray(a, dtype=np.float64)
    return (-np.logaddexp(0.0, -a)).astype(np.float32)


def log_sigmoid_f32_t(a: torch.Tensor) -> torch.Tensor:
    """Tensor form of log_sigmoid_f32."""
    return torch.from_numpy(log_sigmoid_f32(a.numpy()))


def generate(w: Workload, with_grad: bool = True) -> dict:
    """Draw one seeded input set for workload `w` (CPU tensors).

    Returns a dict with q, k, v (and do) as [B,H,L,d] tensors of the workload
    dtype, log_f as a [B,H,L] float32 tensor, and mu as the per-head gate means.
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(w.seed)
    B, H, L, d = w.B, w.H, w.L, w.d
    if w.mu is None:
        mu = torch.rand(H, generator=g, dtype=torch.float64) * 9.0 + 1.0
        mu = mu.tolist()
    else:
        mu = [float(w.mu[h % len(w.mu)]) for h in range(H)]
    shape = (B, H, L, d)
    q = torch.randn(shape, generator=g, dtype=torch.float32)
    k = torch.randn(shape, generator=g, dtype=torch.float32)
    v = torch.randn(shape, generator=g, dtype=torch.float32)
    if w.row_norms is not None:
        r = torch.tensor([float(w.row_norms[h % len(w.row_norms)]) for h in range(H)],
                         dtype=torch.float32).view(1, H, 1, 1)
        q = q / q.norm(dim=-1, keepdim=True) * r
        k = k / k.norm(dim=-1, keepdim=True) * r
    z = torch.randn((B, H, L), generator=g, dtype=torch.float32)
    a = np.asarray(mu, dtype=np.float64).reshape(1, H, 1) + w.gate_sigma * z.numpy().astype(np.float64)
    log_f = torch.from_numpy(log_sigmoid_f32(a))
    out = {"q": q, "k": k, "v": v, "log_f": log_f, "mu": mu}
    if with_grad:
        out["do"] = torch.randn(shape, generator=g, dtype=torch.float32)
    if w.qk_norm:
        for name in ("q", "k"):
            wt = torch.rand((H, d), generator=g, dtype=torch.float32) + 0.5
            x = out[name].double()
            xn = x / torch.sqrt((x * x).mean(dim=-1, keepdim=True)) * (1.0 - 2.0 ** -7)
            out[name] = (xn * wt.double().view(1, H, 1, d)).float()
            out["gamma_" + name] = wt.abs().amax(dim=-1).contiguous()
    td = _torch_dtype(w.dtype)
    for name in ("q", "k", "v", "do"):
        if name in out:
            out[name] = out[name].to(td).contiguous()
    return out


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of a float32/bfloat16 CPU tensor to a float64 numpy array."""
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def projection_inputs(B: int, L: int, d_model: int, H: int, d: int, seed: int) -> dict:
    """Seeded inputs of the Q/K projection: layer inputs X [B*L, d_model] ~ N(0, 1)
    and weights Wq, Wk [d_model, H*d] ~ N(0, 0.02^2) (the initialisation the
    paper's models use, App. B), all rounded to bfloat16 (CPU tensors)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    x = torch.randn((B * L, d_model), generator=g, dtype=torch.float32)
    wq = torch.randn((d_model, H * d), generator=g, dtype=torch.float32) * 0.02
    wk = torch.randn((d_model, H * d), generator=g, dtype=torch.float32) * 0.02
    return {"x": x.bfloat16().contiguous(), "wq": wq.bfloat16().contiguous(),
            "wk": wk.bfloat16().contiguous()}


def gate_inputs(B: int, L: int, d_model: int, H: int, seed: int, mu=None) -> dict:
    """Seeded inputs of the forget-gate projection (Sec. 2, f = sigmoid(w_f^T x + b_f)
    per head): layer inputs X [B*L, d_model] ~ N(0, 1) and weights w_f [d_model, H]
    ~ N(0, 0.02^2), both rounded to bfloat16, and float32 biases b_f [H] ~ U[1, 10]
    (or the given per-head values), so that the gate logits spread like the
    workloads' a ~ N(mu_h, 0.5).  CPU tensors."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    x = torch.randn((B * L, d_model), generator=g, dtype=torch.float32)
    w = torch.randn((d_model, H), generator=g, dtype=torch.float32) * 0.02
    b = torch.rand(H, generator=g, dtype=torch.float32) * 9.0 + 1.0
    if mu is not None:
        b = torch.tensor([float(mu[h % len(mu)]) for h in range(H)], dtype=torch.float32)
    return {"x": x.bfloat16().contiguous(), "w_f": w.bfloat16().contiguous(), "b_f": b}


def long_decode_inputs(B: int, H: int, L: int, d: int, seed: int, device) -> dict:
    """Seeded inputs for timing decoding after a long prompt (16k-64k tokens),
    drawn on `device` so that tens of millions of rows need no host round trip:
    q, k, v [B, H, L, d] bf16 with q and k RMS-normalised and scaled by per-head
    weights from U[0.5, 1.5]^d (the QK-norm setting of App. E, shrunk by 1 - 2^-7
    as in generate()), gates a ~ N(mu_h, 0.5) with mu_h ~ U[1, 10] (drawn on the
    CPU, log f = -softplus(-a) in float64 rounded to float32), and the scale
    bounds gamma_q, gamma_k [H]."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    mu = torch.rand(H, generator=g, dtype=torch.float64) * 9.0 + 1.0
    z = torch.randn((B, H, L), generator=g, dtype=torch.float32)
    a = mu.numpy().reshape(1, H, 1) + 0.5 * z.numpy().astype(np.float64)
    out = {"log_f": torch.from_numpy(log_sigmoid_f32(a)).to(device)}
    gd = torch.Generator(device=device)
    gd.manual_seed(seed)
    for name in ("q", "k", "v"):
        x = torch.randn((B, H, L, d), generator=gd, dtype=torch.float32, device=device)
        if name != "v":
            wt = torch.rand((H, d), generator=g, dtype=torch.float32) + 0.5
            x = x / torch.sqrt((x * x).mean(dim=-1, keepdim=True)) * (1.0 - 2.0 ** -7)
            x = x * wt.to(device).view(1, H, 1, d)
            out["gamma_" + name] = wt.abs().amax(dim=-1).contiguous().to(device)
        out[name] = x.to(torch.bfloat16).contiguous()
    return out
