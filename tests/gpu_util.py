"""Helpers shared by the GPU tests: run the HIP path through the C ABI on
seeded inputs and compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from oracle import sampled


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def new_buffers(w, device="cuda", sentinel=float("nan")):
    import torch
    send = torch.full((w.B, w.sum_dim), sentinel, dtype=torch.float32, device=device)
    recv = torch.full((w.B, w.sum_dim), sentinel, dtype=torch.float32, device=device)
    flags = torch.zeros(w.n_chunks, dtype=torch.int32, device=device)
    return send, recv, flags


def make_plan(w, **opts):
    import paper_2305_06942_amd as ebag
    return ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, **opts)


def run(plan, w, dev, send, flags, fused=True, stream=None):
    f = plan.forward if fused else plan.unfused_forward
    f(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags, stream=stream)


def flags_np(flags):
    return flags.cpu().numpy().view(np.uint32)


def check_full(inp, send_np, s64=None, a64=None, exact=False):
    """Element-by-element comparison with the C oracle (small workloads)."""
    if s64 is None:
        s64, a64, _ = oracle.pool_inputs(inp)
    if exact:
        want = s64.astype(np.float32)
        bad = np.argwhere(send_np.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, f"{len(bad)} elements differ bitwise, first at {bad[0].tolist()}"
        return
    ok, err, bound = oracle.within_tolerance(send_np, s64, a64)
    if not ok:
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"outside tolerance at {i}: gpu={send_np[i]} oracle={s64[i]} bound={bound[i]}")


def check_sampled(inp, send, n_bags=300, seed=0):
    """Sampled bags at full size: each bag's fp64 value recomputed from the
    generator's rows, compared element by element with the GPU row."""
    import torch
    w = inp.w
    bags = sampled.sample_bags(w, n_bags, seed=seed)
    exp = sampled.pool_bags(inp, bags)
    rows = torch.tensor(sorted({e[2] for e in exp}), dtype=torch.int64, device=send.device)
    got_rows = send.index_select(0, rows).cpu().numpy()
    where = {int(r): i for i, r in enumerate(rows.cpu().tolist())}
    for t, b, row, col, s, a in exp:
        g = got_rows[where[row], col:col + w.dims[t]]
        ok, err, bound = oracle.within_tolerance(g, s, a)
        assert ok, f"bag (t={t}, b={b}) outside tolerance: max excess {(err - bound).max()}"
    return len(exp)
