"""Mean pooling (the sum / mean modes of the original pooling kernel,
Sec. III-A) through the C ABI against the oracle's mean mode."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, new_buffers, run, say
from tests.test_gpu_parity import EDGE, SMALL, _custom_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _unweighted(inp):
    return dataclasses.replace(inp, w=inp.w.with_(weighted=False), weights=None)


def test_mean_integer_tables_bit_exact():
    """Integer tables: the fp32 sum is exact, so the IEEE division gives the
    correctly rounded mean -- the oracle's fp64 mean rounded to fp32."""
    import torch
    w = synth.TINY_INT
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp, mean=True)
    for fused in (True, False):
        plan = make_plan(w, pooling_mode=1)
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        check_full(inp, send.cpu().numpy(), s64, a64, exact=True)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))


@pytest.mark.parametrize("name", sorted(SMALL))
def test_mean_parity_small_every_element(name):
    import torch
    inp = _unweighted(synth.make_inputs(SMALL[name]))
    w = inp.w
    say("mean parity", name, w.T, w.B)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp, mean=True)
    outs = []
    for fused in (True, False):
        plan = make_plan(w, pooling_mode=1)
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        got = send.cpu().numpy()
        check_full(inp, got, s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))
        outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


@pytest.mark.parametrize("name", ["empty_bags", "odd_vector_count", "long_bags_cross_stage"])
@pytest.mark.parametrize("check", [0, 1])
def test_mean_edge_cases(name, check):
    """Empty bags (zeros), row widths served by the general kernel, bags longer
    than one staging segment; with and without in-kernel index checks."""
    import torch
    inp = _unweighted(_custom_inputs(*EDGE[name], seed=len(name)))
    w = inp.w
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp, mean=True)
    plan = make_plan(w, pooling_mode=1, check_indices=check)
    send, _, flags = new_buffers(w)
    run(plan, w, dev, send, flags)
    torch.cuda.synchronize()
    check_full(inp, send.cpu().numpy(), s64, a64)
    assert plan.status_ex() == (0, -1, 0, -1)


def test_mean_rejects_weights():
    import torch
    import paper_2305_06942_amd as ebag
    w = SMALL["mixed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    plan = make_plan(w, pooling_mode=1)
    send, _, flags = new_buffers(w)
    for fused in (True, False):
        with pytest.raises(ebag.EbagError) as e:
            run(plan, w, dev, send, flags, fused=fused)
        assert e.value.code == -1 and "weights" in str(e.value)
    torch.cuda.synchronize()
    assert np.all(flags_np(flags) == 0)
