"""The entry points under HIP graph capture: a forward, a backward or a GEMV +
AllReduce captured once and replayed several times, with the program's own
eager work and synchronizations between the replays, gives the eager result
bit for bit on every replay, and the eager result itself matches the oracle.  Nothing they enqueue is a memset; slice and
arrival counters and the persistent grid's ticket re-arm themselves, so a
replay needs no host work, and epoch flags advance by one per replay.  Calls
that wait for a host-chosen epoch (the consumer, the backward with flags,
GEMV + AllReduce in reduce_mode 1) refuse to be captured."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, new_buffers, run, say
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _eager_noise():
    """Unrelated eager work between replays (allocation, kernels, a sync)."""
    import torch
    a = torch.randn(256, 256, device="cuda")
    (a @ a).sum().item()


def _capture(fn):
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "unfused"])
@pytest.mark.parametrize("name,opts", [("tiny", {}), ("mixed_small", {}),
                                       ("mixed_small", {"persistent_wgs_per_cu": -1}),
                                       ("dlrm_small", {"slice_granule": 1})],
                         ids=["tiny", "mixed_small", "mixed_small-persistent", "dlrm_small-per_table"])
def test_forward_graph_replays(name, opts, fused):
    import torch
    w = SMALL[name]
    say("graph forward", name, opts, fused)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, **opts)
    n_flags = plan.n_flags(w.B)
    send, _, _ = new_buffers(w)
    flags = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    run(plan, w, dev, send, flags, fused=fused)  # eager: also uploads the table pointers
    torch.cuda.synchronize()
    check_full(inp, send.cpu().numpy())
    want = send.cpu().numpy().view(np.uint32).copy()
    g = _capture(lambda: run(plan, w, dev, send, flags, fused=fused))
    assert np.all(flags_np(flags) == 1), "capture must not execute"
    for k in range(1, REPLAYS + 1):
        send.fill_(float("nan"))
        g.replay()
        _eager_noise()
        torch.cuda.synchronize()
        assert np.array_equal(send.cpu().numpy().view(np.uint32), want), f"replay {k}"
        assert np.all(flags_np(flags) == 1 + k), f"replay {k}"
    assert plan.status_ex() == (0, -1, 0, -1)


def test_backward_graph_replays():
    import torch
    w = SMALL["mixed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    n = int(sum((inp.offsets[(t + 1) * w.B] - inp.offsets[t * w.B]) * w.dims[t] for t in range(w.T)))
    grad = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(7), device="cuda")
    values = torch.empty((n,), device="cuda")
    plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values)
    torch.cuda.synchronize()
    want = values.cpu().numpy().view(np.uint32).copy()
    ref = oracle.backward(w.dims, inp.offsets, inp.weights, grad.cpu().numpy(), w.B, w.R)
    assert np.array_equal(want, ref.view(np.uint32)), "eager backward differs from the oracle"
    g = _capture(lambda: plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values))
    for k in range(1, REPLAYS + 1):
        values.fill_(float("nan"))
        g.replay()
        _eager_noise()
        torch.cuda.synchronize()
        assert np.array_equal(values.cpu().numpy().view(np.uint32), want), f"replay {k}"


def test_gemv_allreduce_graph_replays():
    import torch
    import paper_2305_06942_amd as ebag
    R, M, Ks = 4, 1000, [256, 512, 128, 384]
    g_ = torch.Generator(device="cuda").manual_seed(11)
    A = [torch.randn((M, K), generator=g_, device="cuda").half() for K in Ks]
    x = [torch.randn((K,), generator=g_, device="cuda").half() for K in Ks]
    y = [torch.empty((M,), device="cuda") for _ in range(R)]
    h = ebag.GemvAR(R, M, Ks, synth.F16, tile_rows=64)
    P = h.launch_info()[0]
    out_flags = torch.zeros(R * P, dtype=torch.int32, device="cuda")
    h.forward(A, x, y, out_flags)
    torch.cuda.synchronize()
    want = [t.cpu().numpy().view(np.uint32).copy() for t in y]
    y64, abs64, _ = oracle.gemv_ar([a.cpu().numpy() for a in A], [v.cpu().numpy() for v in x], synth.F16)
    depth = 8 + max(-(-(K * 2 // 16) // 64) for K in Ks) + 6 + R
    err = np.abs(want[0].view(np.float32).astype(np.float64) - y64)
    assert np.all(err <= depth * 2.0 ** -24 * abs64 + 1e-30), "eager GEMV + AllReduce differs from the oracle"
    g = _capture(lambda: h.forward(A, x, y, out_flags))
    for k in range(1, REPLAYS + 1):
        for t in y:
            t.fill_(float("nan"))
        g.replay()
        _eager_noise()
        torch.cuda.synchronize()
        for r in range(R):
            assert np.array_equal(y[r].cpu().numpy().view(np.uint32), want[r]), f"replay {k} rank {r}"
        assert np.all(flags_np(out_flags) == 1 + k), f"replay {k}"
    assert h.status() == (0, -1)
    h.close()


def test_epoch_waits_refuse_capture():
    """Each refusal is a host-side error before anything is enqueued; the
    capture then holds only the eager fill and ends normally."""
    import torch
    import paper_2305_06942_amd as ebag
    w = SMALL["tiny"]
    plan = make_plan(w)
    send, recv, flags = new_buffers(w)
    grad = torch.zeros((w.B, w.sum_dim), device="cuda")
    offsets = torch.zeros(w.T * w.B + 1, dtype=torch.int64, device="cuda")
    values = torch.empty(16, device="cuda")
    gm = ebag.GemvAR(2, 64, [64, 64], synth.F16, reduce_mode=1)
    A = [torch.zeros((64, 64), device="cuda").half() for _ in range(2)]
    x = [torch.zeros((64,), device="cuda").half() for _ in range(2)]
    y = [torch.zeros((64,), device="cuda") for _ in range(2)]
    torch.cuda.synchronize()
    errors = []
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for call in (lambda: plan.consume(send, flags, recv, w.B, w.R, 1),
                     lambda: plan.backward(grad, offsets, None, w.B, w.R, values, grad_flags=flags, expected_epoch=1),
                     lambda: gm.forward(A, x, y)):
            try:
                call()
            except ebag.EbagError as e:
                errors.append((e.code, str(e)))
        recv.fill_(0.0)
    torch.cuda.synchronize()
    assert [c for c, _ in errors] == [ebag.abi.EBAG_EUNSUPPORTED] * 3, errors
    assert all("graph" in m for _, m in errors), errors
    gm.close()
