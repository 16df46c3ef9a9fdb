"""Table-major run order (option table_major): runs go table by table, and
with T a multiple of the XCD count each XCD works through its own tables.
Results must not depend on the order: every element against the oracle,
fused and unfused, whole and per-table slices, one-shot and persistent grids;
the consumer, the backward with its delivery and a full-size Zipf workload
under the same order."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, check_sampled, flags_np, make_plan, new_buffers, run, say
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu

WORKLOADS = {
    "mixed_small": SMALL["mixed_small"],                                   # T = 12: one table group
    "skewed_t16": synth.scaled(synth.SKEWED, rows=5000, B=8 * 64 * 2, T=16, name="skewed_t16"),  # 8 groups
    "large_t8": synth.scaled(synth.LARGE, rows=4000, B=64 * 32, T=8, name="large_t8"),
}


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("major", [1, 2], ids=["per_xcd", "device"])
@pytest.mark.parametrize("persistent", [0, -1], ids=["one_shot", "persistent"])
@pytest.mark.parametrize("granule", [0, 1])
@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_table_major_parity(name, granule, persistent, major):
    import torch
    w = WORKLOADS[name]
    say("table-major", name, granule, persistent, major)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    plan = make_plan(w, table_major=major, slice_granule=granule, persistent_wgs_per_cu=persistent)
    per_slice = w.T if granule else 1
    outs = []
    for fused in (True, False):
        send, _, _ = new_buffers(w)
        flags = torch.zeros(w.n_chunks * per_slice, dtype=torch.int32, device="cuda")
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        got = send.cpu().numpy()
        check_full(inp, got, s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1, per_slice=per_slice))
        outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    assert plan.status_ex() == (0, -1, 0, -1)


@pytest.mark.parametrize("major", [1, 2], ids=["per_xcd", "device"])
@pytest.mark.parametrize("name", ["skewed_t16", "mixed_small"])
def test_table_major_consumer_and_backward(name, major):
    """Consumer drains per-table slices in table-major order; the backward
    expands the gradient as the delivery (same order) lands; three epochs."""
    import torch
    import paper_2305_06942_amd as ebag
    w = WORKLOADS[name]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, table_major=major, slice_granule=1, chunk_order=1, self_rank=1)
    send, recv, _ = new_buffers(w)
    flags = torch.zeros(w.n_chunks * w.T, dtype=torch.int32, device="cuda")
    gflags = torch.zeros_like(flags)
    main = torch.cuda.current_stream()
    q1, q2 = ebag.queue_stream(), ebag.queue_stream()
    grad = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(4), device="cuda")
    want = oracle.backward(w.dims, inp.offsets, inp.weights, grad.cpu().numpy(), w.B, w.R)
    grad_recv = torch.empty_like(grad)
    values = torch.empty((want.size,), device="cuda")
    for epoch in (1, 2, 3):
        recv.fill_(float("nan"))
        values.fill_(float("nan"))
        q1.wait_stream(main)
        q2.wait_stream(main)
        with torch.cuda.stream(q1):
            run(plan, w, dev, send, flags)
        with torch.cuda.stream(q2):
            plan.consume(send, flags, recv, w.B, w.R, epoch)
        torch.cuda.synchronize()
        with torch.cuda.stream(q1):
            plan.deliver(grad, grad_recv, gflags, w.B, w.R)
        with torch.cuda.stream(q2):
            plan.backward(grad_recv, dev.offsets, dev.weights, w.B, w.R, values, grad_flags=gflags,
                          expected_epoch=epoch)
        torch.cuda.synchronize()
        assert plan.status_ex() == (0, -1, 0, -1), f"epoch {epoch}"
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32)), f"epoch {epoch}"
        assert np.all(flags_np(flags) == epoch) and np.all(flags_np(gflags) == epoch)
        assert np.array_equal(values.cpu().numpy().view(np.uint32), want.view(np.uint32)), f"epoch {epoch}"
    check_full(inp, send.cpu().numpy())


def test_table_major_full_size_skewed():
    """Full-size Zipf workload (64 tables: one table group per XCD), per-table
    slices, cached rows: sampled bags against the per-bag oracle, every flag."""
    import torch
    w = synth.FULL["skewed"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, table_major=1, slice_granule=1, stream_rows=0)
    send, _, _ = new_buffers(w)
    flags = torch.zeros(w.n_chunks * w.T, dtype=torch.int32, device="cuda")
    run(plan, w, dev, send, flags)
    torch.cuda.synchronize()
    assert not torch.isnan(send).any().item(), "some output element was never written"
    assert np.all(flags_np(flags) == 1)
    check_sampled(inp, send, n_bags=400)
    del dev, send
    torch.cuda.empty_cache()


@pytest.mark.parametrize("major", [0, 2], ids=["slice_major", "device"])
def test_consumer_drains_in_production_order(major):
    """The consumer takes (slice, table) items in the producer's run order.
    With one consumer workgroup and one flag never published, exactly the
    items before the missing one in that order are copied, and no other.
    (T = 5 is not a multiple of the XCD count, so table positions are the
    tables themselves.)"""
    import torch
    w = synth.scaled(synth.TINY, rows=1000, B=256, T=5, R=2, C=16, name="tiny_t5")  # 16 slices
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    T, n = w.T, w.n_chunks
    g_k, t_k = 5, 2
    k = g_k * T + t_k
    plan = make_plan(w, slice_granule=1, table_major=major, consumer_wgs=1, debug_suppress_flag=k,
                     consume_timeout_us=100_000)
    send, recv, _ = new_buffers(w)
    flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
    run(plan, w, dev, send, flags)
    torch.cuda.synchronize()
    plan.consume(send, flags, recv, w.B, w.R, 1)
    timed_out, missing = plan.status()
    assert (timed_out, missing) == (1, k)
    plan.reset()
    s, r = send.cpu().numpy(), recv.cpu().numpy()
    off = np.cumsum([0] + list(w.dims))
    for g in range(n):
        for t in range(T):
            before = (g, t) < (g_k, t_k) if major == 0 else (t, g) < (t_k, g_k)
            bs = s[g * w.C:(g + 1) * w.C, off[t]:off[t + 1]]
            br = r[g * w.C:(g + 1) * w.C, off[t]:off[t + 1]]
            if before:
                assert np.array_equal(br.view(np.uint32), bs.view(np.uint32)), f"item (slice {g}, table {t}) not drained"
            else:
                assert np.all(np.isnan(br)), f"item (slice {g}, table {t}) drained out of the producer's order"
