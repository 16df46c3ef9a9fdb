"""Seeded random configurations of the embedding backward through the C ABI,
bit for bit against the oracle: the forward's random inputs (storage type,
widths, batch split, bag-length laws with empty and long bags, weights or
mean), random slice granule, slice and run order and backward launch shape,
both bulk-synchronous and fused with the delivery stand-in, with a NaN
guard past the last value."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import make_plan, say
from tests.test_gpu_random_configs import _case

pytestmark = pytest.mark.gpu

N_CASES = 64
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


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_backward(seed):
    import torch
    inp, fopts = _case(seed)
    w = inp.w
    rng = np.random.default_rng([2305, 6942, 99, seed])
    mean = fopts["pooling_mode"] == 1
    opts = dict(pooling_mode=fopts["pooling_mode"], slice_granule=fopts["slice_granule"],
                chunk_order=fopts["chunk_order"], self_rank=fopts["self_rank"], table_major=fopts["table_major"],
                backward_bags_per_run=int(rng.choice([1, 2, 3, 7, 64])),
                backward_waves_per_wg=int(rng.choice([1, 2, 8, 16])),
                deliver_wgs=int(rng.choice([1, 3, 32, 2048])),
                deliver_waves_per_wg=int(rng.choice([1, 4, 16])))
    say("random backward", seed, dict(T=w.T, dims=w.dims, B=w.B, R=w.R, C=w.C, nnz=inp.nnz), opts)
    plan = make_plan(w, **opts)
    offsets = torch.from_numpy(inp.offsets).cuda()
    weights = None if inp.weights is None else torch.from_numpy(inp.weights).cuda()
    g = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(seed), device="cuda")
    want = oracle.backward(w.dims, inp.offsets, inp.weights, g.cpu().numpy(), w.B, w.R, mean=mean)
    n = want.size
    q1, q2 = _queues()
    for fused in (False, True):
        values = torch.full((n + 64,), float("nan"), device="cuda")
        if fused:
            flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
            recv = torch.full_like(g, float("nan"))
            main = torch.cuda.current_stream()
            q1.wait_stream(main)
            q2.wait_stream(main)
            with torch.cuda.stream(q1):  # the gradient arrives, slice by slice
                plan.deliver(g, recv, flags, w.B, w.R)
            with torch.cuda.stream(q2):
                plan.backward(recv, offsets, weights, w.B, w.R, values, grad_flags=flags, expected_epoch=1)
        else:
            plan.backward(g, offsets, weights, w.B, w.R, values)
        torch.cuda.synchronize()
        assert plan.status_ex() == (0, -1, 0, -1)
        if fused:
            assert np.all(flags.cpu().numpy() == 1), "delivery flags"
            assert torch.equal(recv.view(torch.int32), g.view(torch.int32)), "delivered gradient"
        got = values.cpu().numpy()
        bad = np.flatnonzero(got[:n].view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, f"{'fused' if fused else 'bulk'}: {bad.size} values differ, first at {bad[0]}"
        assert np.isnan(got[n:]).all(), "stores past the last value"
    plan.close()
