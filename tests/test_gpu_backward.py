"""Embedding backward (per-lookup gradient rows) through the C ABI against the
oracle, bulk-synchronous and fused with the gradient's arrival.  Every value
is one fp32 multiply or divide of a received gradient value, so GPU and
oracle agree bit for bit."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import make_plan, say
from tests.test_gpu_parity import EDGE, SMALL, _custom_inputs

pytestmark = pytest.mark.gpu

_QUEUES = []


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _queues():
    import paper_2305_06942_amd as ebag
    if not _QUEUES:
        _QUEUES.extend([ebag.queue_stream(), ebag.queue_stream()])
    return _QUEUES


def _grad(w, seed):
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randn((w.B, w.sum_dim), generator=g, device="cuda")


def _n_values(inp):
    w = inp.w
    return int(sum((inp.offsets[(t + 1) * w.B] - inp.offsets[t * w.B]) * w.dims[t] for t in range(w.T)))


def _expected(inp, grad, mean):
    return oracle.backward(inp.w.dims, inp.offsets, inp.weights, grad.cpu().numpy(), inp.w.B, inp.w.R, mean=mean)


def _check(inp, grad, values, mean):
    want = _expected(inp, grad, mean)
    got = values.cpu().numpy()
    bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
    assert bad.size == 0, f"{bad.size} values differ, first at {bad[0]}: gpu {got[bad[0]]} oracle {want[bad[0]]}"


def _unweighted(inp):
    return dataclasses.replace(inp, w=inp.w.with_(weighted=False), weights=None)


@pytest.mark.parametrize("granule", [0, 1])
@pytest.mark.parametrize("mean", [False, True])
@pytest.mark.parametrize("name", sorted(SMALL))
def test_backward_bulk_synchronous(name, mean, granule):
    import torch
    inp = synth.make_inputs(SMALL[name])
    if mean:
        inp = _unweighted(inp)
    w = inp.w
    dev = sdev.to_device(inp)
    grad = _grad(w, 5)
    plan = make_plan(w, pooling_mode=int(mean), slice_granule=granule)
    values = torch.full((_n_values(inp),), float("nan"), device="cuda")
    plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values)
    torch.cuda.synchronize()
    _check(inp, grad, values, mean)


@pytest.mark.parametrize("name", sorted(EDGE))
def test_backward_edge_cases(name):
    import torch
    inp = _custom_inputs(*EDGE[name], seed=len(name))
    w = inp.w
    dev = sdev.to_device(inp)
    grad = _grad(w, 9)
    plan = make_plan(w)
    values = torch.full((max(_n_values(inp), 1),), float("nan"), device="cuda")
    plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values)
    torch.cuda.synchronize()
    _check(inp, grad, values[:_n_values(inp)], False)


_SHAPE_CASES = {
    "tables_300": (synth.F32, [4, 8, 12] * 100, [5] * 300, 4, 2, 1, lambda r, n: r.integers(0, 4, n), True),
    "chunk_128_wide": (synth.F32, [256, 1024], [50, 50], 256, 2, 128, lambda r, n: r.integers(0, 7, n), True),
}


@pytest.mark.parametrize("case", ["fp16_wide_ragged", "wide_rows_512", "many_tables", "tables_300", "chunk_128_wide"])
@pytest.mark.parametrize("bags,waves", [(1, 1), (3, 2), (7, 16), (64, 4), (1000, 1)])
def test_backward_launch_shapes(case, bags, waves):
    """Bags per workgroup and workgroup sizes that put the per-thread walk over
    the run's rows in every relation to the row width (step below, equal to,
    above a row; several rows per step), bag counts past the LDS and thread
    caps, and more tables than one pass of the table-size scan."""
    import torch
    spec = EDGE[case] if case in EDGE else _SHAPE_CASES[case]
    inp = _custom_inputs(*spec, seed=len(case) + bags)
    w = inp.w
    dev = sdev.to_device(inp)
    grad = _grad(w, bags * 17 + waves)
    plan = make_plan(w, backward_bags_per_run=bags, backward_waves_per_wg=waves)
    n = _n_values(inp)
    values = torch.full((n + 64,), float("nan"), device="cuda")
    plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values)
    torch.cuda.synchronize()
    _check(inp, grad, values[:n], False)
    assert torch.isnan(values[n:]).all(), "stores past the last lookup row"


def _fused(plan, w, dev, grad_dp, grad_recv, flags, values, epoch):
    import torch
    main = torch.cuda.current_stream()
    send_q, bwd_q = _queues()
    send_q.wait_stream(main)
    bwd_q.wait_stream(main)
    with torch.cuda.stream(send_q):  # the gradient arriving, slice by slice
        plan.deliver(grad_dp, grad_recv, flags, w.B, w.R)
    with torch.cuda.stream(bwd_q):   # expanded as it arrives
        plan.backward(grad_recv, dev.offsets, dev.weights, w.B, w.R, values, grad_flags=flags, expected_epoch=epoch)
    torch.cuda.synchronize()


@pytest.mark.parametrize("opts", [dict(), dict(slice_granule=1), dict(chunk_order=1, self_rank=1),
                                  dict(pooling_mode=1)], ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()) or "default")
def test_backward_fused_with_delivery(opts):
    import torch
    inp = synth.make_inputs(SMALL["mixed_small"])
    if opts.get("pooling_mode"):
        inp = _unweighted(inp)
    w = inp.w
    dev = sdev.to_device(inp)
    plan = make_plan(w, **opts)
    per_slice = w.T if opts.get("slice_granule") else 1
    flags = torch.zeros(w.n_chunks * per_slice, dtype=torch.int32, device="cuda")
    grad_recv = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
    for epoch in (1, 2, 3):
        grad_dp = _grad(w, 100 + epoch)
        values = torch.full((_n_values(inp),), float("nan"), device="cuda")
        _fused(plan, w, dev, grad_dp, grad_recv, flags, values, epoch)
        assert plan.status_ex() == (0, -1, 0, -1)
        assert np.all(flags.cpu().numpy() == epoch)
        assert torch.equal(grad_dp, grad_recv)
        _check(inp, grad_dp, values, bool(opts.get("pooling_mode")))


@pytest.mark.parametrize("granule", [0, 1])
@pytest.mark.parametrize("wgs,waves", [(1, 1), (1, 16), (3, 4), (32, 8), (16, 16), (2048, 1)])
def test_delivery_shapes(wgs, waves, granule):
    """The gradient's arrival stand-in over its launch shapes: one wavefront
    doing every item, a few wide workgroups, more wavefronts than items.  Whole
    slices here are 22.5 pieces of 32 KiB (a ragged last piece), so the
    per-slice piece counter is exercised; per-table slices take one item per
    (slice, table).  Two epochs, fused with the backward: the delivered
    gradient equals its source bit for bit, every flag holds the epoch, the
    piece counters re-arm, and the backward matches the oracle."""
    import torch
    inp = synth.make_inputs(SMALL["mixed_small"])
    w = inp.w
    assert (w.C * w.sum_dim) % 8192 != 0  # the last piece of a slice is ragged
    dev = sdev.to_device(inp)
    plan = make_plan(w, slice_granule=granule, table_major=granule, deliver_wgs=wgs, deliver_waves_per_wg=waves)
    say("delivery shape", wgs, waves, granule)
    flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
    for epoch in (1, 2):
        grad_dp = _grad(w, 300 + epoch)
        grad_recv = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
        values = torch.full((_n_values(inp),), float("nan"), device="cuda")
        _fused(plan, w, dev, grad_dp, grad_recv, flags, values, epoch)
        assert plan.status_ex() == (0, -1, 0, -1)
        assert np.all(flags.cpu().numpy() == epoch), f"epoch {epoch}: flags"
        assert torch.equal(grad_dp.view(torch.int32), grad_recv.view(torch.int32)), f"epoch {epoch}: delivered gradient"
        _check(inp, grad_dp, values, False)
    plan.close()


def test_backward_times_out_without_delivery():
    import torch
    w = SMALL["dlrm_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, consume_timeout_us=20000)
    flags = torch.zeros(w.n_chunks, dtype=torch.int32, device="cuda")
    values = torch.full((_n_values(inp),), float("nan"), device="cuda")
    plan.backward(_grad(w, 1), dev.offsets, dev.weights, w.B, w.R, values, grad_flags=flags, expected_epoch=1)
    timed_out, missing = plan.status()
    assert timed_out == 1 and missing == 0
    plan.reset()
    assert torch.isnan(values).all()


def test_backward_full_size_dlrm_fused():
    """dlrm size: every value of the fused delivery + backward, bit for bit."""
    import torch
    w = synth.FULL["dlrm"]
    say("backward full dlrm")
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    flags = torch.zeros(w.n_chunks, dtype=torch.int32, device="cuda")
    grad_recv = torch.empty((w.B, w.sum_dim), device="cuda")
    grad_dp = _grad(w, 7)
    values = torch.full((_n_values(inp),), float("nan"), device="cuda")
    _fused(plan, w, dev, grad_dp, grad_recv, flags, values, 1)
    assert plan.status_ex() == (0, -1, 0, -1)
    _check(inp, grad_dp, values, False)
    del values
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["skewed", "large", "mixed"])
def test_backward_full_size_sampled(name):
    """Full workload sizes in the launch configuration the backward benchmark
    times (the workload's plan options without the row-cache and grid ones),
    fused with the delivery: sampled bags bit for bit against the per-bag
    oracle, every value bit for bit against the C oracle, every flag, and no
    value left unwritten."""
    import torch
    import bench
    from oracle import sampled
    w = synth.FULL[name]
    say("backward full", name)
    inp = synth.make_inputs(w)
    opts = {k: v for k, v in bench.PLAN_OPTS.get(name, {}).items()
            if k not in ("stream_rows", "persistent_wgs_per_cu")}
    plan = make_plan(w, **opts)
    offsets = torch.from_numpy(inp.offsets).cuda()
    weights = None if inp.weights is None else torch.from_numpy(inp.weights).cuda()
    dev = sdev.DeviceInputs(None, None, offsets, weights)
    flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
    grad_recv = torch.empty((w.B, w.sum_dim), device="cuda")
    grad_dp = _grad(w, 9)
    n = _n_values(inp)
    say("backward full", name, "values", n)
    values = torch.full((n,), float("nan"), device="cuda")
    _fused(plan, w, dev, grad_dp, grad_recv, flags, values, 1)
    assert plan.status_ex() == (0, -1, 0, -1)
    assert np.all(flags.cpu().numpy() == 1)
    assert not torch.isnan(values).any().item(), "some value was never written"
    g = grad_dp.cpu().numpy()
    for t, b in sampled.sample_bags(w, 300, seed=5):
        want = sampled.backward_bag(inp, g, t, b)
        o = sampled.backward_value_offset(inp, t, b)
        got = values[o:o + want.size].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.reshape(-1).view(np.uint32)), f"bag (t={t}, b={b})"
    # Every value, bit for bit, against the C oracle, a group of tables at a
    # time (its gradient columns and its block of values).
    B, base = w.B, 0
    for t0 in range(0, w.T, 16):
        t1 = min(t0 + 16, w.T)
        lo, hi = int(inp.offsets[t0 * B]), int(inp.offsets[t1 * B])
        c0, c1 = w.col_off[t0], w.col_off[t1 - 1] + w.dims[t1 - 1]
        want = oracle.backward(w.dims[t0:t1], inp.offsets[t0 * B:t1 * B + 1] - lo,
                               None if inp.weights is None else inp.weights[lo:hi],
                               np.ascontiguousarray(g[:, c0:c1]), B, w.R)
        got = values[base:base + want.size].cpu().numpy()
        bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, f"tables {t0}..{t1 - 1}: {bad.size} values differ, first at {base + bad[0]}"
        base += want.size
    assert base == n
    say("backward full", name, "every value checked")
    del values, grad_recv
    torch.cuda.empty_cache()
