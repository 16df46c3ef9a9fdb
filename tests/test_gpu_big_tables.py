"""Tables at the 4 GiB boundary of the fast kernels' 32-bit buffer offsets.

A table of at most 4 GiB - 1 byte is gathered through one buffer resource
with 32-bit row offsets; a larger one goes through the general kernels with
64-bit addresses.  Each case puts lookups on the first row, on the table's
last rows and on the rows around byte 2^32, and checks every bag of the batch
against the per-bag oracle, fused and unfused, with every flag."""
import numpy as np
import pytest

import oracle
import synth
from oracle import sampled
from synth import device as sdev
from tests.gpu_util import flags_np, make_plan, new_buffers, run, say

pytestmark = pytest.mark.gpu

# name: (dtype, big table dim, big table rows, weighted)
CASES = {
    "f32_just_below_4GiB": (synth.F32, 256, (1 << 22) - 1, False),
    "f32_just_above_4GiB": (synth.F32, 256, (1 << 22) + 1, True),
    "bf16_above_4GiB": (synth.BF16, 512, (1 << 22) + 96, True),
}


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _inputs(dtype, dim, rows, weighted):
    w = synth.Workload("big", 7, 2, (rows, 1000), (dim, 64), dtype, 64, 2, 4, "uniform:0:40", "uniform",
                       weighted, "uniform")
    inp = synth.make_inputs(w)
    # Steer lookups of table 0 onto its edges: the first row, the last rows,
    # and the rows whose bytes straddle offset 2^32.
    seg = inp.indices[: int(inp.offsets[w.B])]
    boundary_row = (1 << 32) // (dim * w.elt)
    edges = np.array([0, rows - 1, rows - 2, boundary_row - 1, boundary_row, boundary_row + 1], dtype=np.int64)
    edges = edges[(edges >= 0) & (edges < rows)]
    rng = np.random.default_rng(99)
    pick = rng.random(seg.size) < 0.3
    seg[pick] = rng.choice(edges, size=int(pick.sum())).astype(np.int32)
    return inp


@pytest.mark.parametrize("name", sorted(CASES))
def test_table_at_4gib_boundary(name):
    import torch
    dtype, dim, rows, weighted = CASES[name]
    inp = _inputs(dtype, dim, rows, weighted)
    w = inp.w
    say("big table", name, "rows", rows, "bytes", rows * dim * w.elt)
    dev = sdev.to_device(inp)
    bags = [(t, b) for t in range(w.T) for b in range(w.B)]
    exp = sampled.pool_bags(inp, bags)
    plan = make_plan(w)
    send, _, flags = new_buffers(w)
    for fused in (True, False):
        flags.zero_()
        send.fill_(float("nan"))
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        say("big table", name, "fused" if fused else "unfused", "ran")
        got = send.cpu().numpy()
        for t, b, row, col, s, a in exp:
            ok, err, bound = oracle.within_tolerance(got[row, col:col + w.dims[t]], s, a)
            assert ok, f"bag (t={t}, b={b}) outside tolerance: max excess {(err - bound).max()}"
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))
    assert plan.status_ex() == (0, -1, 0, -1)
    plan.close()
    del dev, send, flags
    torch.cuda.empty_cache()
