"""Cross-epoch staleness: many epochs in a row whose results differ from one
epoch to the next, so that a reader that saw a stale copy of the previous
epoch's data (a cache line, a reused slot) would be caught.

* forward + concurrent consumer: the index arrays (and weights) alternate
  between two draws of the same shape; every epoch's send and recv buffers are
  checked against that epoch's oracle, under both release protocols and both
  slice granules;
* backward fused with the gradient's arrival: the gradient alternates;
* GEMV + AllReduce: the vector x alternates, in both reduction modes (the
  reduction slots are reused every epoch).

Each case stops at its first mismatch and names the epoch."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import flags_np, make_plan, say

pytestmark = pytest.mark.gpu

EPOCHS = 24


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2305_06942_amd as ebag
    ebag.load()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


_Q = []


def _queues():
    """Producer and consumer each on a stream with a hardware queue of its own."""
    import paper_2305_06942_amd as ebag
    if not _Q:
        _Q.extend([ebag.queue_stream(), ebag.queue_stream()])
    return _Q


# Fixed bag lengths give both draws the same offsets, so only the rows (and
# weights) differ between epochs.
FWD = {
    "dlrm_like": synth.scaled(synth.DLRM, rows=4000, T=8, B=1024, name="stale_dlrm"),
    "mixed_like": synth.scaled(synth.MIXED.with_(lengths="fixed:20"), rows=3000, T=8, B=2048, name="stale_mixed"),
}


def _two_draws(w):
    """Two inputs with the same tables and offsets but different indices (and
    weights): the second draw comes from the workload's seed stream for
    another configuration id, keeping the first draw's tables."""
    import dataclasses
    a = synth.make_inputs(w)
    b = synth.make_inputs(w.with_(cfg_id=w.cfg_id + 100))
    assert np.array_equal(a.offsets, b.offsets)
    assert not np.array_equal(a.indices, b.indices)
    b = dataclasses.replace(b, w=w, host_tables=a.host_tables)
    return a, b


@pytest.mark.parametrize("release_mode", [0, 1])
@pytest.mark.parametrize("granule", [0, 1])
@pytest.mark.parametrize("name", sorted(FWD))
def test_forward_consumer_alternating_inputs(name, granule, release_mode):
    import torch
    w = FWD[name]
    opts = {"release_mode": release_mode, "slice_granule": granule}
    if granule == 1:
        opts["table_major"] = 1
    say("staleness forward", name, opts)
    draws = _two_draws(w)
    devs = [sdev.to_device(d) for d in draws]
    # one set of tables: the second draw reads the first draw's tables
    devs[1] = sdev.DeviceInputs(devs[0].tables, devs[1].indices, devs[1].offsets, devs[1].weights)
    want = []
    for d in draws:
        s64, a64, _ = oracle.pool_inputs(d)
        want.append((s64, a64))
    assert not np.array_equal(want[0][0], want[1][0])
    plan = make_plan(w, **opts)
    n_flags = w.n_chunks * (w.T if granule == 1 else 1)
    send = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
    recv = torch.full_like(send, float("nan"))
    flags = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    prod, cons = _queues()
    main = torch.cuda.current_stream()
    for epoch in range(1, EPOCHS + 1):
        dev = devs[epoch % 2]
        prod.wait_stream(main)
        cons.wait_stream(main)
        with torch.cuda.stream(prod):
            plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags)
        with torch.cuda.stream(cons):
            plan.consume(send, flags, recv, w.B, w.R, epoch)
        main.wait_stream(prod)
        main.wait_stream(cons)
        torch.cuda.synchronize()
        assert plan.status_ex() == (0, -1, 0, -1), f"epoch {epoch}: status {plan.status_ex()}"
        assert np.all(flags_np(flags) == epoch), f"epoch {epoch}: flags"
        s64, a64 = want[epoch % 2]
        for what, buf in (("send", send), ("recv", recv)):
            ok, err, bound = oracle.within_tolerance(buf.cpu().numpy(), s64, a64)
            assert ok, f"epoch {epoch}: {what} differs from this epoch's oracle (max excess {(err - bound).max()})"
        assert torch.equal(send.view(torch.int32), recv.view(torch.int32)), f"epoch {epoch}: recv != send"
    plan.close()


@pytest.mark.parametrize("granule", [0, 1])
def test_backward_delivery_alternating_gradients(granule):
    import torch
    w = FWD["mixed_like"]
    opts = {"slice_granule": granule, "table_major": 1 if granule else 0}
    say("staleness backward", opts)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    gen = torch.Generator(device="cuda").manual_seed(17)
    grads = [torch.randn((w.B, w.sum_dim), generator=gen, device="cuda") for _ in range(2)]
    want = [oracle.backward(w.dims, inp.offsets, inp.weights, g.cpu().numpy(), w.B, w.R) for g in grads]
    assert not np.array_equal(want[0], want[1])
    plan = make_plan(w, **opts)
    n_flags = w.n_chunks * (w.T if granule == 1 else 1)
    grad_recv = torch.full_like(grads[0], float("nan"))
    gflags = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    values = torch.full((want[0].size,), float("nan"), device="cuda")
    prod, cons = _queues()
    main = torch.cuda.current_stream()
    for epoch in range(1, EPOCHS + 1):
        prod.wait_stream(main)
        cons.wait_stream(main)
        with torch.cuda.stream(prod):
            plan.deliver(grads[epoch % 2], grad_recv, gflags, w.B, w.R)
        with torch.cuda.stream(cons):
            plan.backward(grad_recv, dev.offsets, dev.weights, w.B, w.R, values, grad_flags=gflags,
                          expected_epoch=epoch)
        main.wait_stream(prod)
        main.wait_stream(cons)
        torch.cuda.synchronize()
        assert plan.status_ex()[:2] == (0, -1), f"epoch {epoch}: status {plan.status_ex()}"
        got = values.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want[epoch % 2].view(np.uint32)), \
            f"epoch {epoch}: backward differs from this epoch's oracle"
    plan.close()


@pytest.mark.parametrize("mode", [0, 1])
def test_gemv_ar_alternating_vectors(mode):
    import torch
    import paper_2305_06942_amd as ebag
    R, M, Ks, dtype = 4, 4096 + 37, [1024, 512, 2048, 256], synth.F16
    say("staleness gemv", mode)
    rng = np.random.default_rng([2305, 6942, 977])
    A = [rng.standard_normal((M, K)).astype(np.float16) for K in Ks]
    xs = [[rng.standard_normal(K).astype(np.float16) for K in Ks] for _ in range(2)]
    want = [oracle.gemv_ar(A, x, dtype)[:2] for x in xs]
    assert not np.allclose(want[0][0], want[1][0])
    depth = 8 + max(-(-(K * 2 // 16) // 64) for K in Ks) + 6 + R
    rel = depth * 2.0 ** -24
    dA = [torch.from_numpy(a).cuda() for a in A]
    dxs = [[torch.from_numpy(v).cuda() for v in x] for x in xs]
    plan = ebag.GemvAR(R, M, Ks, dtype, reduce_mode=mode)
    P = plan.launch_info()[0]
    y = [torch.full((M,), float("nan"), device="cuda") for _ in range(R)]
    flags = torch.zeros(R * P, dtype=torch.int32, device="cuda")
    for epoch in range(1, EPOCHS + 1):
        plan.forward(dA, dxs[epoch % 2], y, flags)
        torch.cuda.synchronize()
        assert np.all(flags.cpu().numpy() == epoch), f"epoch {epoch}: flags"
        y64, abs64 = want[epoch % 2]
        for r in range(R):
            got = y[r].cpu().numpy().astype(np.float64)
            err = np.abs(got - y64)
            bound = rel * abs64 + 1e-30
            assert np.all(err <= bound), f"epoch {epoch}, rank {r}: differs from this epoch's oracle"
    assert plan.status() == (0, -1)
    plan.close()
