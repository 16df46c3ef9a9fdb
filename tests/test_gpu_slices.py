"""Per-table slices (slice_granule = 1): the paper's slice is a group of
pooled vectors of one table (Sec. III-A), so each (slice, table) pair gets
its own ready flag at index g * T + t.  The pooled data is the same as with
whole slices; the flags, the counters behind them and the consumer's work
items change."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, run, say
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _buffers(w):
    import torch
    send = torch.full((w.B, w.sum_dim), float("nan"), dtype=torch.float32, device="cuda")
    recv = torch.full_like(send, float("nan"))
    flags = torch.zeros(w.n_chunks * w.T, dtype=torch.int32, device="cuda")
    return send, recv, flags


_STREAMS = []


def _streams():
    import torch
    import paper_2305_06942_amd as ebag
    if not _STREAMS:
        _STREAMS.extend([torch.cuda.Stream(), ebag.queue_stream()])
    return _STREAMS


def _concurrent(plan, w, dev, send, recv, flags, epoch, fused=True):
    import torch
    main = torch.cuda.current_stream()
    prod, cons = _streams()
    prod.wait_stream(main)
    cons.wait_stream(main)
    with torch.cuda.stream(prod):
        run(plan, w, dev, send, flags, fused=fused)
    with torch.cuda.stream(cons):
        plan.consume(send, flags, recv, w.B, w.R, epoch)
    main.wait_stream(prod)
    main.wait_stream(cons)
    torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["tiny", "dlrm_small", "mixed_small"])
@pytest.mark.parametrize("chunk_order", [0, 1])
def test_per_table_flags_and_data(name, chunk_order):
    """Same pooled bits as whole slices, every per-table flag equal to the
    epoch, fused and unfused."""
    import torch
    w = SMALL[name]
    say("per-table", name, chunk_order)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    ref_plan = make_plan(w)
    ref, _, ref_flags = _buffers(w)
    run(ref_plan, w, dev, ref, ref_flags[:w.n_chunks])
    plan = make_plan(w, slice_granule=1, chunk_order=chunk_order, self_rank=w.R - 1)
    assert plan.n_flags(w.B) == w.n_chunks * w.T
    for fused in (True, False):
        send, _, flags = _buffers(w)
        for epoch in (1, 2):
            run(plan, w, dev, send, flags, fused=fused)
            torch.cuda.synchronize()
            assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, epoch, per_slice=w.T))
        got = send.cpu().numpy()
        check_full(inp, got, s64, a64)
        assert np.array_equal(got.view(np.uint32), ref.cpu().numpy().view(np.uint32))
    assert plan.status_ex() == (0, -1, 0, -1)


@pytest.mark.parametrize("fused", [True, False])
def test_per_table_consumer_drains_every_slice(fused):
    import torch
    w = SMALL["mixed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, slice_granule=1, trace=1)
    send, recv, flags = _buffers(w)
    n = plan.n_flags(w.B)
    for epoch in (1, 2, 3):
        recv.fill_(float("nan"))
        _concurrent(plan, w, dev, send, recv, flags, epoch, fused)
        assert plan.status_ex() == (0, -1, 0, -1)
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32))
        assert np.all(flags_np(flags) == epoch)
        rel, drn, _ = plan.trace(n)
        assert np.all(rel > 0) and np.all(drn >= rel)


def test_per_table_overlap_full_size():
    """At the dlrm size the per-table slices are drained while pooling runs."""
    import torch
    w = synth.FULL["dlrm"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, slice_granule=1, trace=1)
    send, recv, flags = _buffers(w)
    _concurrent(plan, w, dev, send, recv, flags, 1)
    assert plan.status_ex() == (0, -1, 0, -1)
    assert torch.equal(send.view(torch.int32), recv.view(torch.int32))
    rel, drn, tpu = plan.trace(plan.n_flags(w.B))
    assert np.all(drn >= rel)
    assert (drn < rel.max()).sum() >= plan.n_flags(w.B) // 4


def test_per_table_suppressed_flag_is_named():
    import torch
    w = synth.TINY
    k = 2 * w.T + 3  # slice 2, table 3
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, slice_granule=1, debug_suppress_flag=k, consume_timeout_us=20000)
    send, recv, flags = _buffers(w)
    _concurrent(plan, w, dev, send, recv, flags, 1)
    f = flags_np(flags)
    assert f[k] == 0 and np.all(np.delete(f, k) == 1)
    timed_out, missing = plan.status()
    assert timed_out == 1 and missing == k
    plan.reset()
    check_full(inp, send.cpu().numpy())
    torch.cuda.synchronize()
