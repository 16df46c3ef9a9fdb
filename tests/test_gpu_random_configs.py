"""Seeded random configurations through the C ABI against the oracle.

Each case draws a storage type, per-table widths (16-byte multiples, some not
a power of two in 16-byte vectors), table sizes, batch split (B, R, C), bag
length law (with empty and long bags), weights or mean pooling, slice
granule, slice and run order and launch options, then checks the fused and unfused
results element by element, the flags, and the consumer's copy."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, run, say

pytestmark = pytest.mark.gpu

N_CASES = 96
_QUEUE = []


def _queue_stream():
    import paper_2305_06942_amd as ebag
    if not _QUEUE:
        _QUEUE.append(ebag.queue_stream())
    return _QUEUE[0]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _case(seed):
    rng = np.random.default_rng([2305, 6942, 77, seed])
    dtype = int(rng.integers(0, 3))
    elt = 4 if dtype == synth.F32 else 2
    T = int(rng.integers(1, 10))
    vec_choices = [1, 2, 3, 4, 5, 8, 16, 32, 64, 96]
    dims = [int(rng.choice(vec_choices)) * 16 // elt for _ in range(T)]
    rows = [int(rng.integers(1, 3000)) for _ in range(T)]
    R = int(rng.choice([1, 2, 3, 4, 8]))
    C = int(rng.choice([1, 2, 5, 8, 16, 32]))
    B = R * C * int(rng.integers(1, 5))
    law = int(rng.integers(0, 4))
    if law == 0:
        L = rng.integers(0, 4, size=T * B)
    elif law == 1:
        L = rng.integers(1, 80, size=T * B)
    elif law == 2:
        L = np.minimum(rng.poisson(30, size=T * B), 600)
    else:
        L = rng.integers(0, 2, size=T * B) * rng.integers(100, 700, size=T * B)
    off = np.zeros(T * B + 1, dtype=np.int64)
    off[1:] = np.cumsum(L)
    idx = np.concatenate([rng.integers(0, rows[t], size=int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)]).astype(np.int32) if off[-1] else np.zeros(0, np.int32)
    tabs = []
    for t in range(T):
        v = rng.standard_normal((rows[t], dims[t])).astype(np.float32)
        if dtype == synth.F16:
            v = v.astype(np.float16)
        elif dtype == synth.BF16:
            v = synth.gen.f32_to_bf16_bits(v)
        tabs.append(v)
    mode = int(rng.integers(0, 3))  # 0 sum, 1 weighted sum, 2 mean
    wts = rng.random(int(off[-1]), dtype=np.float32) if mode == 1 else None
    w = synth.Workload(f"random{seed}", 9, T, tuple(rows), tuple(dims), dtype, B, R, C, "fixed:1", "uniform",
                       mode == 1, "normal")
    inp = synth.Inputs(w, L.astype(np.int64), off, idx, wts, tabs)
    opts = dict(pooling_mode=1 if mode == 2 else 0, slice_granule=int(rng.integers(0, 2)),
                chunk_order=int(rng.integers(0, 2)), self_rank=int(rng.integers(0, R)),
                waves_per_wg=int(rng.choice([1, 2, 4, 8])), bags_per_run=int(rng.choice([1, 3, 16, 40])),
                rows_in_flight=int(rng.choice([4, 8])), persistent_wgs_per_cu=int(rng.choice([0, 0, 1, 3])),
                check_indices=int(rng.integers(0, 2)), stream_rows=int(rng.integers(0, 2)))
    opts["table_major"] = int(rng.integers(0, 3))
    opts["consume_nontemporal"] = int(rng.integers(0, 2))
    opts["release_mode"] = int(rng.random() < 0.25)
    return inp, opts


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_config(seed):
    import torch
    inp, opts = _case(seed)
    w = inp.w
    say("random", seed, dict(dtype=w.dtype, T=w.T, dims=w.dims, B=w.B, R=w.R, C=w.C, nnz=inp.nnz), opts)
    dev = sdev.to_device(inp)
    mean = opts["pooling_mode"] == 1
    s64, a64, _ = oracle.pool_inputs(inp, mean=mean)
    plan = make_plan(w, **opts)
    per_slice = w.T if opts["slice_granule"] else 1
    n_flags = w.n_chunks * per_slice
    cons = _queue_stream()
    main = torch.cuda.current_stream()
    outs = []
    for fused in (True, False):
        send = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
        recv = torch.full_like(send, float("nan"))
        flags = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
        ready = main.record_event()  # buffers initialised; the forward follows on main
        run(plan, w, dev, send, flags, fused=fused)
        cons.wait_event(ready)
        with torch.cuda.stream(cons):
            plan.consume(send, flags, recv, w.B, w.R, 1)
        torch.cuda.synchronize()
        assert plan.status_ex() == (0, -1, 0, -1)
        got = send.cpu().numpy()
        check_full(inp, got, s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1, per_slice=per_slice))
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32))
        outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
