"""Consumer kernel, overlap, and failure paths (timeouts, suppressed flags,
bad indices) -- every kernel exits normally; failures are forced from the host."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, new_buffers, run, say
from tests.test_gpu_parity import SMALL

SMALL_MIXED = SMALL["mixed_small"]

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


_STREAMS = []


def _streams():
    """Producer on an ordinary stream, consumer on a stream with a hardware
    queue of its own; the producer is enqueued first."""
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


@pytest.mark.parametrize("fused", [True, False])
def test_consumer_drains_every_slice(fused):
    import torch
    w = synth.TINY
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, trace=1)
    send, recv, flags = new_buffers(w)
    s64, a64, _ = oracle.pool_inputs(inp)
    for epoch in (1, 2, 3):
        recv.fill_(float("nan"))
        _concurrent(plan, w, dev, send, recv, flags, epoch, fused)
        assert plan.status_ex() == (0, -1, 0, -1)
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32))
        check_full(inp, recv.cpu().numpy(), s64, a64)
        assert np.all(flags_np(flags) == epoch)
        rel, drn, _ = plan.trace(w.n_chunks)
        assert np.all(rel > 0) and np.all(drn >= rel)


@pytest.mark.parametrize("name", ["dlrm", "mixed"])
def test_overlap_full_size(name):
    """The consumer drains slices while pooling is still running: the first
    drain happens before the last slice is released."""
    import torch
    w = synth.FULL[name]
    say("overlap", name)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, trace=1)
    send, recv, flags = new_buffers(w)
    for epoch in (1, 2):
        _concurrent(plan, w, dev, send, recv, flags, epoch)
    assert plan.status_ex() == (0, -1, 0, -1)
    assert torch.equal(send.view(torch.int32), recv.view(torch.int32))
    assert np.all(flags_np(flags) == 2)
    rel, drn, tpu = plan.trace(w.n_chunks)
    assert np.all(drn >= rel)
    say("overlap", name, "first drain before last release by", (rel.max() - drn.min()) / tpu, "us")
    assert drn.min() < rel.max()
    assert (drn < rel.max()).sum() >= w.n_chunks // 4


def test_queue_stream_runs_concurrently():
    """A consumer enqueued *before* its producer on the dedicated-queue stream
    still sees every slice: the two kernels run at the same time."""
    import torch
    w = synth.FULL["dlrm"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, consume_timeout_us=2_000_000, trace=1)
    send, recv, flags = new_buffers(w)
    main = torch.cuda.current_stream()
    prod, cons = _streams()
    prod.wait_stream(main)
    cons.wait_stream(main)
    for epoch in (1, 2, 3):
        with torch.cuda.stream(cons):
            plan.consume(send, flags, recv, w.B, w.R, epoch)
        with torch.cuda.stream(prod):
            run(plan, w, dev, send, flags)
        torch.cuda.synchronize()
        assert plan.status_ex() == (0, -1, 0, -1), f"epoch {epoch}"
        rel, drn, tpu = plan.trace(w.n_chunks)
        assert drn.min() < rel.max(), "no slice was drained while pooling was still running"
    assert torch.equal(send.view(torch.int32), recv.view(torch.int32))


def test_consumer_times_out_without_producer():
    w = synth.TINY
    plan = make_plan(w, consume_timeout_us=2000)
    send, recv, flags = new_buffers(w)
    plan.consume(send, flags, recv, w.B, w.R, 1)
    timed_out, missing = plan.status()
    assert timed_out == 1 and missing == 0
    plan.reset()
    assert plan.status_ex() == (0, -1, 0, -1)


@pytest.mark.parametrize("fused", [True, False])
def test_suppressed_flag_is_named(fused):
    import torch
    w = synth.TINY
    k = 5
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, debug_suppress_flag=k, consume_timeout_us=20000)
    send, recv, flags = new_buffers(w)
    _concurrent(plan, w, dev, send, recv, flags, 1, fused)
    f = flags_np(flags)
    assert f[k] == 0 and np.all(np.delete(f, k) == 1)
    timed_out, missing = plan.status()
    assert timed_out == 1 and missing == k
    plan.reset()
    # the data itself is complete even though the flag was withheld
    check_full(inp, send.cpu().numpy())
    torch.cuda.synchronize()


def test_double_publication_is_reported():
    """Flags already ahead of the expected epoch are reported, not hidden."""
    w = synth.TINY
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    send, recv, flags = new_buffers(w)
    run(plan, w, dev, send, flags)
    run(plan, w, dev, send, flags)
    plan.consume(send, flags, recv, w.B, w.R, 1)
    st = plan.status_ex()
    assert st[0] == 0 and st[2] == w.n_chunks


def test_bad_index_reported_and_skipped():
    """With check_indices the kernel bounds-checks every index and offset,
    skips bad rows and names the first bad bag."""
    import torch
    w = synth.TINY
    inp = synth.make_inputs(w)
    bad_bag = 3 * w.B + 17
    inp.indices[inp.offsets[bad_bag] + 1] = w.rows[0] + 5
    dev = sdev.to_device(inp)
    plan = make_plan(w, check_indices=1)
    send, _, flags = new_buffers(w)
    run(plan, w, dev, send, flags)
    torch.cuda.synchronize()
    st = plan.status_ex()
    assert st[3] == bad_bag
    assert np.all(flags_np(flags) == 1)


@pytest.mark.parametrize("opts", [dict(), dict(slice_granule=1, consume_nontemporal=1),
                                  dict(persistent_wgs_per_cu=-1, chunk_order=1, self_rank=3),
                                  dict(table_major=1, slice_granule=1, consume_nontemporal=1, release_mode=0)],
                         ids=["default", "per_table_nt", "persistent_comm_aware", "table_major_nt_release0"])
def test_stress_100_epochs_across_flag_wraparound(opts):
    """100 forwards, each drained concurrently by the consumer, with the epoch
    flags starting 50 below 2^32 so that they wrap to 0 midway: every epoch
    must be fully drained (recv == send bit for bit, sentinel-filled before),
    with every flag at the epoch and no timeout or double publication."""
    import torch
    w = SMALL_MIXED
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, **opts)
    send, recv, _ = new_buffers(w)
    base = (1 << 32) - 50
    flags = torch.full((plan.n_flags(w.B),), base - (1 << 32), dtype=torch.int32, device="cuda")
    say("stress", opts)
    for k in range(1, 101):
        epoch = (base + k) & 0xFFFFFFFF
        recv.fill_(float("nan"))
        _concurrent(plan, w, dev, send, recv, flags, epoch)
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32)), f"epoch {k}"
        assert np.all(flags_np(flags) == epoch), f"epoch {k}"
    assert plan.status_ex() == (0, -1, 0, -1)
    check_full(inp, send.cpu().numpy())


def test_stress_100_backward_epochs_across_flag_wraparound():
    """100 backwards, each fed by the delivery stand-in on its own queue and
    waiting per slice, flags wrapping through 2^32: every epoch equals the
    oracle's per-lookup gradient bit for bit."""
    import torch
    import paper_2305_06942_amd as ebag
    w = SMALL_MIXED
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    grad = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(3), device="cuda")
    want = torch.from_numpy(oracle.backward(w.dims, inp.offsets, inp.weights, grad.cpu().numpy(), w.B, w.R)).cuda()
    base = (1 << 32) - 50
    flags = torch.full((w.n_chunks,), base - (1 << 32), dtype=torch.int32, device="cuda")
    recv = torch.empty_like(grad)
    values = torch.empty_like(want)
    main = torch.cuda.current_stream()
    send_q, bwd_q = ebag.queue_stream(), ebag.queue_stream()
    for k in range(1, 101):
        epoch = (base + k) & 0xFFFFFFFF
        recv.fill_(float("nan"))
        values.fill_(float("nan"))
        send_q.wait_stream(main)
        bwd_q.wait_stream(main)
        with torch.cuda.stream(send_q):
            plan.deliver(grad, recv, flags, w.B, w.R)
        with torch.cuda.stream(bwd_q):
            plan.backward(recv, dev.offsets, dev.weights, w.B, w.R, values, grad_flags=flags, expected_epoch=epoch)
        torch.cuda.synchronize()
        assert torch.equal(values.view(torch.int32), want.view(torch.int32)), f"epoch {k}"
    assert plan.status_ex() == (0, -1, 0, -1)


def test_overlapping_forwards_on_two_streams_refused():
    """A forward enqueued on another stream while the plan's last forward has
    not completed returns EBAG_EBUSY and enqueues nothing; on the same stream,
    or once the last one completed, it runs.  The first forward is held back
    by a bounded spin kernel queued ahead of it."""
    import torch
    import paper_2305_06942_amd as ebag
    if not hasattr(torch.cuda, "_sleep"):
        pytest.skip("torch.cuda._sleep is not available")
    w = SMALL_MIXED
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    send, _, flags = new_buffers(w)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        torch.cuda._sleep(200_000_000)
        run(plan, w, dev, send, flags)
    for fused in (True, False):
        with pytest.raises(ebag.EbagError) as e:
            run(plan, w, dev, send, flags, fused=fused, stream=s2)
        assert e.value.code == ebag.abi.EBAG_EBUSY
    with torch.cuda.stream(s1):
        run(plan, w, dev, send, flags)  # same stream: ordered after the first
    torch.cuda.synchronize()
    run(plan, w, dev, send, flags, stream=s2)  # the others have completed
    torch.cuda.synchronize()
    assert np.all(flags_np(flags) == 3)
    s64, a64, _ = oracle.pool_inputs(inp)
    check_full(inp, send.cpu().numpy(), s64, a64)


def test_overlapping_backwards_and_deliveries_on_two_streams_refused():
    """Likewise for the backward (its table bases are shared) and the
    delivery (its piece counters are shared): a second one on another stream
    while the first is held back by a spin kernel returns EBAG_EBUSY and
    enqueues nothing; a backward and a delivery on two streams are
    independent and both run.  The results match the oracle bit for bit."""
    import torch
    import paper_2305_06942_amd as ebag
    if not hasattr(torch.cuda, "_sleep"):
        pytest.skip("torch.cuda._sleep is not available")
    w = SMALL_MIXED
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    g = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(41), device="cuda")
    want = oracle.backward(w.dims, inp.offsets, inp.weights, g.cpu().numpy(), w.B, w.R)
    values = torch.full((want.size,), float("nan"), device="cuda")
    recv = torch.full_like(g, float("nan"))
    flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        torch.cuda._sleep(200_000_000)
        plan.backward(g, dev.offsets, dev.weights, w.B, w.R, values)
        plan.deliver(g, recv, flags, w.B, w.R)
    with pytest.raises(ebag.EbagError) as e:
        plan.backward(g, dev.offsets, dev.weights, w.B, w.R, values, stream=s2)
    assert e.value.code == ebag.abi.EBAG_EBUSY
    with pytest.raises(ebag.EbagError) as e:
        plan.deliver(g, recv, flags, w.B, w.R, stream=s2)
    assert e.value.code == ebag.abi.EBAG_EBUSY
    torch.cuda.synchronize()
    assert np.all(flags.cpu().numpy() == 1), "one delivery ran, the refused one enqueued nothing"
    assert torch.equal(recv.view(torch.int32), g.view(torch.int32))
    assert np.array_equal(values.cpu().numpy().view(np.uint32), want.view(np.uint32))
    # a delivery on one stream and a backward waiting for it on another: both run
    values.fill_(float("nan"))
    with torch.cuda.stream(s1):
        plan.deliver(g, recv, flags, w.B, w.R)
    with torch.cuda.stream(s2):
        plan.backward(recv, dev.offsets, dev.weights, w.B, w.R, values, grad_flags=flags, expected_epoch=2)
    torch.cuda.synchronize()
    assert plan.status_ex() == (0, -1, 0, -1)
    assert np.array_equal(values.cpu().numpy().view(np.uint32), want.view(np.uint32))
