"""Savings of ACP against its error tolerance eps, and the per-head spread of the
pruned fraction, on the seeded synthetic workloads.

The paper reports FLOP savings against eps (Sec. 4, Fig. 7) and the spread of
per-head savings, which is bimodal for trained models (local and global heads;
Sec. 4, Figs. 4-5).  Neither the trained weights nor the validation loss are
available here, so only the shape of those analyses is reproduced: for each eps
the pruned fraction of 64x64 blocks (the paper's proxy for FLOP and memory
savings), its per-head values binned into a 20-bin histogram, and optionally the
measured fwd+bwd time and speedup over eps = 0.

    python -m paper_2504_06949_amd.sweep [--workload 125m] [--time]

prints one JSON line.  Every number comes from the HIP library (stage 1 and, with
--time, the attention passes); nothing here computes any part of the method.
"""
from __future__ import annotations

import argparse
import json
import math

import numpy as np
import torch

from . import acp, workloads

DEFAULT_EPS = tuple(math.exp(-k) for k in (1, 2, 5, 10, 15, 20, 30)) + (0.0,)


def pruned_fraction_by_head(plan: dict, M: int) -> np.ndarray:
    """[B, H] pruned fraction of the causal 64x64 blocks, from stage 1's kept counts."""
    kept = plan["kept"].cpu().numpy().astype(np.float64)
    return 1.0 - kept / (M * (M + 1) / 2)


def head_histogram(fracs: np.ndarray, bins: int = 20) -> list:
    """Counts of heads per pruned-fraction bin [i/bins, (i+1)/bins) (last bin closed)."""
    counts, _ = np.histogram(np.asarray(fracs).ravel(), bins=bins, range=(0.0, 1.0))
    return counts.tolist()


def _time_step(g, eps, ws, out_f, out_b, steps, warmup) -> float:
    def step():
        acp.forward(g["q"], g["k"], g["v"], g["log_f"], eps, ws=ws, out=out_f)
        acp.backward(g["q"], g["k"], g["v"], out_f[0], g["do"], ws, out=out_b)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def eps_sweep(w: workloads.Workload, eps_list=DEFAULT_EPS, time_it: bool = False,
              steps: int = 20, warmup: int = 5) -> dict:
    x = workloads.generate(w, with_grad=time_it)
    dev = torch.device("cuda:0")
    g = {k: (v.to(dev) if torch.is_tensor(v) else v) for k, v in x.items()}
    ws = acp.workspace(g["q"])
    if time_it:
        out_f = (torch.empty_like(g["q"]),
                 torch.empty(g["log_f"].shape, dtype=torch.float32, device=dev))
        out_b = (torch.empty_like(g["q"]), torch.empty_like(g["k"]), torch.empty_like(g["v"]),
                 torch.empty(g["log_f"].shape, dtype=torch.float32, device=dev))
        _time_step(g, 0.0, ws, out_f, out_b, steps, 3 * warmup)   # clocks and caches settle
    rows = []
    for eps in eps_list:
        plan = acp.boundary(g["q"], g["k"], g["log_f"], eps, ws=ws)
        fr = pruned_fraction_by_head(plan, w.M)
        row = {"eps": eps, "log_eps": (math.log(eps) if eps > 0 else None),
               "pruned_fraction": round(float(fr.mean()), 4),
               "heads_fully_kept": int(np.sum(fr == 0.0)),
               "head_histogram": head_histogram(fr)}
        if time_it:
            row["ms"] = round(_time_step(g, eps, ws, out_f, out_b, steps, warmup), 4)
        rows.append(row)
    if time_it:
        ms0 = _time_step(g, 0.0, ws, out_f, out_b, steps, warmup)
        for row in rows:
            row["speedup_vs_eps0"] = round(ms0 / row["ms"], 3)
    return {"workload": w.describe(), "heads": w.B * w.H, "rows": rows}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="125m", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--time", action="store_true", help="also time fwd+bwd at each eps")
    args = ap.parse_args()
    res = eps_sweep(workloads.WORKLOADS[args.workload], time_it=args.time)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
