"""Every finite fp16 and bf16 bit pattern through the GPU gather: tables
whose rows hold all 65536 patterns (Inf/NaN patterns replaced by zero),
one-lookup bags, so each pooled value is 0 + (one widened table value) and
must equal it bit for bit: subnormals included (no flush to zero); a
negative zero pools to +0 (0 + -0 = +0 in IEEE arithmetic, as in the
oracle's sum).  Also with unit weights (fma(1, x, 0))."""
import numpy as np
import pytest

import synth
from synth import device as sdev
from synth.gen import Inputs
from tests.gpu_util import make_plan, new_buffers, run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _patterns(dtype):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    if dtype == synth.F16:
        special = (bits & 0x7C00) == 0x7C00
        bits[special] = 0
        wide = bits.view(np.float16).astype(np.float32)
    else:
        special = (bits & 0x7F80) == 0x7F80
        bits[special] = 0
        wide = (bits.astype(np.uint32) << 16).view(np.float32)
    return bits, wide


@pytest.mark.parametrize("weighted", [False, True], ids=["sum", "unit_weights"])
@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16], ids=["f16", "bf16"])
def test_every_bit_pattern_widens_exactly(dtype, weighted):
    import torch
    D, rows = 64, 1024
    B, R, C, T = rows, 2, 32, 2
    bits, wide = _patterns(dtype)
    tab = bits.reshape(rows, D)
    host = [tab.view(np.float16) if dtype == synth.F16 else tab, (tab[::-1].copy().view(np.float16)
                                                                   if dtype == synth.F16 else tab[::-1].copy())]
    w = synth.Workload("bits", 9, T, (rows, rows), (D, D), dtype, B, R, C, "fixed:1", "uniform", weighted, "normal")
    lengths = np.ones(T * B, dtype=np.int64)
    offsets = np.arange(T * B + 1, dtype=np.int64)
    indices = np.concatenate([np.arange(B), np.arange(B)]).astype(np.int32)
    weights = np.ones(T * B, dtype=np.float32) if weighted else None
    inp = Inputs(w, lengths, offsets, indices, weights, host_tables=host)
    dev = sdev.to_device(inp)
    plan = make_plan(w)
    send, _, flags = new_buffers(w)
    for fused in (True, False):
        send.fill_(float("nan"))
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        got = send.cpu().numpy()
        want0 = (np.float32(0.0) + wide).reshape(rows, D)
        want1 = want0[::-1]
        # send row of sample b is b (destinations are contiguous blocks of the batch)
        assert np.array_equal(got[:, :D].view(np.uint32), want0.view(np.uint32)), "table 0"
        assert np.array_equal(got[:, D:].view(np.uint32), want1.view(np.uint32)), "table 1"
