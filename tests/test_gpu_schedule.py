"""The workgroup schedule of the bf16 attention kernels (a property of this
implementation, not of the paper): the tables that the forward writes into the
plan, checked against a host model of the rules stated in include/acp.h and
acp_plan.hip.  Each table must be a permutation of the (head, 128-row block)
items; logical workgroup ids are split into 8 contiguous ranges, one per XCD;
with B*H a multiple of 8 and at most 64 the heads are placed on the XCDs by
kept-block count (largest first, each on the least loaded XCD with room, lowest
index on ties); inside each range the items run in non-increasing order of
their kept tiles."""
import numpy as np
import pytest
import torch

from paper_2504_06949_amd import acp, workloads

pytestmark = pytest.mark.gpu


def xcd_ranges(nblocks):
    q, r = divmod(nblocks, 8)
    out = []
    for x in range(8):
        lo = x * q + min(x, r)
        out.append((lo, lo + q + (1 if x < r else 0)))
    return out


def placement(kept):
    """Greedy placement of heads on 8 XCDs with BH / 8 heads each; returns the
    head of each slot (XCD j owns slots j * per .. j * per + per - 1)."""
    BH = len(kept)
    per = BH // 8
    order = sorted(range(BH), key=lambda h: (-int(kept[h]), h))
    load, count = [0] * 8, [0] * 8
    slots = [None] * BH
    for h in order:
        best = min((j for j in range(8) if count[j] < per), key=lambda j: (load[j], j))
        slots[best * per + count[best]] = h
        count[best] += 1
        load[best] += int(kept[h])
    return slots


def item_work(table, bh, blk, M, row_start, col_end):
    w = 0
    for m in (2 * blk, 2 * blk + 1):
        if m < M:
            w += (m - int(row_start[bh, m]) + 1) if table == "q" else (int(col_end[bh, m]) - m + 1)
    return w


@pytest.mark.parametrize("B,H,L,mu,seed", [
    (2, 16, 2048, (0.0, 3.0, 6.0, 12.0), 61),       # 32 heads: placed, 4 per XCD
    (4, 16, 1024, (0.5, 2.0, 5.0, 9.0, 20.0), 62),  # 64 heads: placed, 8 per XCD
    (1, 8, 1024, (1.0, 4.0), 63),                   # 8 heads: one per XCD
    (3, 4, 1344, (0.5, 3.0, 8.0), 64),              # 12 heads: head order; ragged last block
])
def test_schedule_tables(B, H, L, mu, seed):
    w = workloads.custom(f"sched{seed}", B, H, L, 64, "bf16", seed, mu=mu)
    print(f"case: schedule {w.describe()}", flush=True)
    x = workloads.generate(w, with_grad=False)
    g = {k: (v.cuda() if torch.is_tensor(v) else v) for k, v in x.items()}
    ws = acp.workspace(g["q"])
    o = torch.empty_like(g["q"])
    lse = torch.empty(g["log_f"].shape, dtype=torch.float32, device="cuda")
    acp.forward(g["q"], g["k"], g["v"], g["log_f"], w.eps, ws=ws, out=(o, lse))
    torch.cuda.synchronize()
    pv = {k: v.cpu().numpy() for k, v in acp.plan_views(ws, B, H, L, 64, torch.bfloat16).items()}
    BH, M, nb = B * H, L // 64, (L + 127) // 128
    rs = pv["row_start"].reshape(BH, M)
    ce = pv["col_end"].reshape(BH, M)
    kept = pv["kept"].reshape(BH)
    place = BH % 8 == 0 and 8 <= BH <= 64
    slots = placement(kept) if place else list(range(BH))
    for table in ("q", "k"):
        sched = pv["sched_" + table].astype(np.int64)
        assert sorted(sched.tolist()) == list(range(BH * nb)), "not a permutation"
        for lo, hi in xcd_ranges(BH * nb):
            # the items the range must hold: logical id -> (slot head, block)
            want = set()
            for lid in range(lo, hi):
                bh = slots[lid // nb]
                idx = lid % nb
                blk = nb - 1 - idx if table == "q" else idx
                want.add(bh * nb + blk)
            got = sched[lo:hi].tolist()
            assert set(got) == want
            works = [item_work(table, e // nb, e % nb, M, rs, ce) for e in got]
            assert all(a >= b for a, b in zip(works, works[1:])), "not largest first"
