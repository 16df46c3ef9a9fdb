"""The plan-free forward that allocates nothing (ebag_a2a_forward_noalloc),
called through the C ABI, against the plan's forward (ebag_a2a_forward) on
the same inputs: both run the same pooling kernel in the same order, so the
send buffers must agree bit for bit, and the flags must equal the epoch.
Each case makes two calls in a row on the device's one scratch array, the
second with a smaller input (fewer tables, a smaller batch), so leftovers of
the first call would show in the second.  The results are also checked
against the oracle."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, flags_np, make_plan, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2305_06942_amd as ebag
    ebag.load()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _pair(base, rows, T1, B1, T2, B2):
    big = synth.scaled(base, rows=rows, T=T1, B=B1, name=base.name + "_noalloc_a")
    small = synth.scaled(base, rows=rows, T=T2, B=B2, name=base.name + "_noalloc_b")
    return big, small


CASES = {
    # (first call, second call), plan options
    "tiny": (_pair(synth.TINY, 10_000, 4, 256, 2, 64), {}),
    "dlrm": (_pair(synth.DLRM, 4000, 70, 1024, 9, 512), {}),
    "skewed_table_major": (_pair(synth.SKEWED, 3000, 16, 1024, 8, 512),
                           {"stream_rows": 0, "table_major": 1, "slice_granule": 1}),
    "mixed_weighted_persistent": (_pair(synth.MIXED, 3000, 12, 4096, 4, 2048),
                                  {"persistent_wgs_per_cu": 2, "table_major": 2, "slice_granule": 1}),
    "large_comm_aware": (_pair(synth.LARGE, 3000, 16, 4096, 8, 2048), {"chunk_order": 1, "self_rank": 3}),
    "mean": (_pair(synth.DLRM.with_(lengths="uniform:0:40"), 2000, 8, 1024, 3, 512), {"pooling_mode": 1}),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_noalloc_matches_plan_forward(name):
    import torch
    import paper_2305_06942_amd as ebag
    (first, second), opts = CASES[name]
    for call, w in enumerate((first, second)):
        mean = opts.get("pooling_mode", 0) == 1
        if mean:
            w = w.with_(weighted=False)
        say("noalloc", name, "call", call, "T", w.T, "B", w.B, "R", w.R, "C", w.C, opts)
        inp = synth.make_inputs(w)
        dev = sdev.to_device(inp)
        n_flags = w.n_chunks * (w.T if opts.get("slice_granule", 0) == 1 else 1)
        want = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
        got = torch.full_like(want, float("nan"))
        f_want = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
        f_got = torch.zeros_like(f_want)
        plan = make_plan(w, **opts)
        for epoch in (1, 2):
            plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, want, f_want)
            ebag.forward_noalloc(w.rows, w.dims, w.dtype, w.C, dev.tables, dev.indices, dev.offsets, dev.weights,
                                 w.B, w.R, got, f_got, **opts)
            torch.cuda.synchronize()
            assert torch.equal(got.view(torch.int32), want.view(torch.int32)), "differs from the plan's forward"
            assert np.all(flags_np(f_got) == epoch) and np.all(flags_np(f_want) == epoch)
        plan.close()
        if mean:
            s64, a64, _ = oracle.pool_inputs(inp, mean=True)
        else:
            s64, a64, _ = oracle.pool_inputs(inp)
        check_full(inp, got.cpu().numpy(), s64, a64)
        want_flags = oracle.flags(w.B, w.R, w.C, 2, per_slice=w.T if opts.get("slice_granule", 0) == 1 else 1)
        assert np.array_equal(flags_np(f_got), want_flags)


def test_noalloc_integer_tables_bit_exact():
    """Integer-valued tables have exactly one correct fp32 result."""
    import torch
    import paper_2305_06942_amd as ebag
    for w in (synth.TINY_INT, synth.scaled(synth.TINY_INT, rows=10_000, T=3, B=64, name="tiny_int_b")):
        say("noalloc integer", w.T, w.B)
        inp = synth.make_inputs(w)
        dev = sdev.to_device(inp)
        got = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
        flags = torch.zeros(w.n_chunks, dtype=torch.int32, device="cuda")
        ebag.forward_noalloc(w.rows, w.dims, w.dtype, w.C, dev.tables, dev.indices, dev.offsets, dev.weights,
                             w.B, w.R, got, flags)
        torch.cuda.synchronize()
        check_full(inp, got.cpu().numpy(), exact=True)
        assert np.all(flags_np(flags) == 1)


def test_noalloc_at_its_limits():
    """The stated maxima: 1024 tables (16 install launches), then 65,536
    flags (one-sample slices); each call against the plan's forward bit for
    bit and against the oracle."""
    import torch
    import paper_2305_06942_amd as ebag
    cases = [
        (synth.scaled(synth.TINY, rows=64, T=1024, B=64, R=2, C=32, name="noalloc_1024_tables").with_(dims=(16,) * 1024),
         {}),
        (synth.scaled(synth.TINY, rows=1000, T=1, B=65536, R=1, C=1, name="noalloc_65536_flags"), {}),
        (synth.scaled(synth.TINY, rows=1000, T=2, B=32768, R=2, C=1, name="noalloc_65536_table_flags"),
         {"slice_granule": 1}),
    ]
    for w, opts in cases:
        n_flags = w.n_chunks * (w.T if opts.get("slice_granule", 0) == 1 else 1)
        say("noalloc limits", w.name, "T", w.T, "B", w.B, "flags", n_flags)
        assert n_flags <= ebag.abi.NOALLOC_MAX_FLAGS and w.T <= ebag.abi.NOALLOC_MAX_TABLES
        inp = synth.make_inputs(w)
        dev = sdev.to_device(inp)
        want = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
        got = torch.full_like(want, float("nan"))
        f_want = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
        f_got = torch.zeros_like(f_want)
        plan = make_plan(w, **opts)
        plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, want, f_want)
        ebag.forward_noalloc(w.rows, w.dims, w.dtype, w.C, dev.tables, dev.indices, dev.offsets, dev.weights,
                             w.B, w.R, got, f_got, **opts)
        torch.cuda.synchronize()
        plan.close()
        assert torch.equal(got.view(torch.int32), want.view(torch.int32)), "differs from the plan's forward"
        assert np.all(flags_np(f_got) == 1) and np.all(flags_np(f_want) == 1)
        check_full(inp, got.cpu().numpy())


def test_noalloc_headline_workload_full_size():
    """The large workload at full size in the benchmark's launch options
    (128 tables, per-table slices: 512 x 128 = 65,536 flags, the stated
    maximum): the whole send buffer equals the plan's forward bit for bit,
    every element is written, and sampled bags match the oracle."""
    import torch
    import bench
    import paper_2305_06942_amd as ebag
    from tests.gpu_util import check_sampled
    w = synth.FULL["large"]
    opts = {k: v for k, v in bench.PLAN_OPTS["large"].items() if not k.startswith(("consume", "deliver", "backward"))}
    n_flags = w.n_chunks * w.T
    assert n_flags == ebag.abi.NOALLOC_MAX_FLAGS and opts.get("slice_granule") == 1
    say("noalloc full size large", opts)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    want = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
    got = torch.full_like(want, float("nan"))
    f_want = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    f_got = torch.zeros_like(f_want)
    plan = make_plan(w, **opts)
    plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, want, f_want)
    ebag.forward_noalloc(w.rows, w.dims, w.dtype, w.C, dev.tables, dev.indices, dev.offsets, dev.weights,
                         w.B, w.R, got, f_got, **opts)
    torch.cuda.synchronize()
    plan.close()
    assert not torch.isnan(got).any().item(), "some output element was never written"
    assert torch.equal(got.view(torch.int32), want.view(torch.int32)), "differs from the plan's forward"
    assert np.all(flags_np(f_got) == 1)
    say("noalloc full size large: checked", check_sampled(inp, got, n_bags=200), "bags")
    del dev, want, got
    torch.cuda.empty_cache()


def test_noalloc_graph_replays():
    """Under HIP graph capture, one of the uses this entry point exists for:
    captured once and replayed three times.  Between replays an eager
    plan-free call on another input leaves its own state in the device's
    scratch array, and eager work and synchronizations run too.  Every replay
    re-installs its descriptors and clears the counters, so each gives the
    plan's forward result bit for bit, and the flags advance by one per
    replay (capture itself runs nothing)."""
    import torch
    import paper_2305_06942_amd as ebag
    w = synth.scaled(synth.MIXED, rows=3000, T=12, B=2048, name="mixed_noalloc_graph")
    other = synth.scaled(synth.DLRM, rows=2000, T=5, B=512, name="dlrm_noalloc_graph_other")
    opts = {"table_major": 2, "slice_granule": 1}
    say("noalloc graph", w.T, w.B, opts)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    o_inp = synth.make_inputs(other)
    o_dev = sdev.to_device(o_inp)
    n_flags = w.n_chunks * w.T
    want = torch.full((w.B, w.sum_dim), float("nan"), device="cuda")
    f_want = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    plan = make_plan(w, **opts)
    plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, want, f_want)
    torch.cuda.synchronize()
    check_full(inp, want.cpu().numpy())
    plan.close()
    got = torch.full_like(want, float("nan"))
    f_got = torch.zeros_like(f_want)
    o_send = torch.empty((other.B, other.sum_dim), device="cuda")
    o_flags = torch.zeros(other.n_chunks, dtype=torch.int32, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ebag.forward_noalloc(w.rows, w.dims, w.dtype, w.C, dev.tables, dev.indices, dev.offsets, dev.weights,
                             w.B, w.R, got, f_got, **opts)
    torch.cuda.synchronize()
    assert np.all(flags_np(f_got) == 0), "capture must not execute"
    for k in range(1, 4):
        ebag.forward_noalloc(other.rows, other.dims, other.dtype, other.C, o_dev.tables, o_dev.indices,
                             o_dev.offsets, o_dev.weights, other.B, other.R, o_send, o_flags)
        torch.cuda.synchronize()
        got.fill_(float("nan"))
        g.replay()
        (torch.randn(256, 256, device="cuda") @ torch.randn(256, 256, device="cuda")).sum().item()
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int32), want.view(torch.int32)), f"replay {k}"
        assert np.all(flags_np(f_got) == k), f"replay {k}"
    assert np.all(flags_np(o_flags) == 3)
