"""Parity of the HIP path (through the C ABI) with the CPU oracle."""
import numpy as np
import pytest

import oracle
import synth
from synth import device as sdev
from tests.gpu_util import check_full, check_sampled, flags_np, make_plan, new_buffers, run, say

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


@pytest.mark.parametrize("dtype", [synth.F32, synth.F16, synth.BF16])
@pytest.mark.parametrize("kind", [0, 1])
def test_device_fill_matches_host(dtype, kind):
    import torch
    rows, dim = 1000, 64
    x = torch.empty((rows, dim), dtype=sdev.torch_dtype(dtype), device="cuda")
    seed = synth.table_seed(7, 3)
    sdev.fill_table(x, seed, kind, dtype)
    torch.cuda.synchronize()
    got = x.cpu()
    got = got.view(torch.int16).numpy().view(np.uint16) if dtype != synth.F32 else got.numpy()
    want = synth.counter_values(seed, dim, np.arange(rows), kind, dtype)
    assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(want).view(np.uint8))


def test_tiny_integer_tables_bit_exact():
    """Integer-valued tables: exactly one correct fp32 result, in any order."""
    w = synth.TINY_INT
    say("tiny_int", w)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    for fused in (True, False):
        plan = make_plan(w)
        send, _, flags = new_buffers(w)
        for epoch in (1, 2, 3):
            run(plan, w, dev, send, flags, fused=fused)
            import torch
            torch.cuda.synchronize()
            check_full(inp, send.cpu().numpy(), s64, a64, exact=True)
            assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, epoch))
        assert plan.status_ex() == (0, -1, 0, -1)


def _small(base):
    return synth.scaled(base, rows=5000, B=base.R * base.C * 2, T=min(base.T, 12))


SMALL = {"tiny": synth.TINY, "dlrm_small": _small(synth.DLRM), "skewed_small": _small(synth.SKEWED),
         "large_small": _small(synth.LARGE), "mixed_small": _small(synth.MIXED)}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_parity_small_every_element(name):
    """Every element of fused and unfused results within the tolerance of the
    oracle, flags bit-exact; both paths produce identical bits."""
    import torch
    w = SMALL[name]
    say("parity", name, w.T, w.B, w.R, w.C)
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    plan = make_plan(w)
    outs = []
    for fused in (True, False):
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        got = send.cpu().numpy()
        check_full(inp, got, s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))
        outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


VARIANTS = [
    dict(waves_per_wg=1), dict(waves_per_wg=16), dict(rows_in_flight=4), dict(rows_in_flight=16),
    dict(bags_per_run=1), dict(bags_per_run=1000), dict(bags_per_run=5), dict(persistent_wgs_per_cu=2),
    dict(persistent_wgs_per_cu=-1), dict(release_mode=0), dict(release_mode=0, bags_per_run=64, waves_per_wg=8), dict(chunk_order=1, self_rank=1),
    dict(check_indices=1), dict(stream_rows=0),
]


@pytest.mark.parametrize("opts", VARIANTS, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_launch_variants(opts):
    import torch
    w = SMALL["mixed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    plan = make_plan(w, **opts)
    for fused in (True, False):
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        check_full(inp, send.cpu().numpy(), s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))
    assert plan.status_ex() == (0, -1, 0, -1)


def _custom_inputs(dtype, dims, rows, B, R, C, lengths, weighted, seed):
    rng = np.random.default_rng(seed)
    w = synth.Workload("custom", 9, len(dims), tuple(rows), tuple(dims), dtype, B, R, C, "fixed:1", "uniform",
                       weighted, "normal")
    T = len(dims)
    L = np.asarray(lengths(rng, T * B), dtype=np.int64)
    off = np.zeros(T * B + 1, dtype=np.int64)
    off[1:] = np.cumsum(L)
    idx = np.concatenate([rng.integers(0, rows[t], size=int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)]).astype(np.int32) if off[-1] else np.zeros(0, np.int32)
    tabs = []
    for t in range(T):
        v = rng.standard_normal((rows[t], dims[t])).astype(np.float32)
        if dtype == synth.F16:
            v = v.astype(np.float16)
        elif dtype == synth.BF16:
            v = synth.gen.f32_to_bf16_bits(v)
        tabs.append(v)
    wts = rng.random(int(off[-1]), dtype=np.float32) if weighted else None
    return synth.Inputs(w, L, off, idx, wts, tabs)


EDGE = {
    "single_sample": (synth.F32, [4], [3], 1, 1, 1, lambda r, n: r.integers(1, 3, n), False),
    "empty_bags": (synth.F32, [64, 32], [50, 40], 8, 2, 2, lambda r, n: r.integers(0, 2, n) * r.integers(0, 5, n), False),
    "long_bags_cross_stage": (synth.BF16, [128], [300], 8, 2, 4, lambda r, n: r.integers(120, 400, n), True),
    "odd_vector_count": (synth.F32, [12, 20, 4], [30, 30, 30], 16, 4, 2, lambda r, n: r.integers(1, 20, n), True),
    "wide_rows_512": (synth.F32, [512, 1024], [20, 10], 8, 2, 2, lambda r, n: r.integers(1, 40, n), False),
    "fp16_wide_ragged": (synth.F16, [8, 24, 256, 72], [100, 7, 60, 9], 12, 3, 2, lambda r, n: r.integers(0, 70, n), True),
    "many_tables": (synth.BF16, [32] * 70, [64] * 70, 4, 2, 1, lambda r, n: r.integers(1, 9, n), False),
    "all_bags_empty": (synth.F16, [64, 32], [50, 40], 8, 2, 2, lambda r, n: np.zeros(n, dtype=np.int64), True),
}


@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_cases(name):
    import torch
    inp = _custom_inputs(*EDGE[name], seed=len(name))
    w = inp.w
    say("edge", name, w.dims, w.B, w.R, w.C)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    plan = make_plan(w)
    for fused in (True, False):
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=fused)
        torch.cuda.synchronize()
        check_full(inp, send.cpu().numpy(), s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))


# Full-size workloads whose tables fit comfortably in host memory are checked
# element by element over the whole batch; for the large workload (131 GB of
# tables) every element of the column stripes of its first and last four
# tables is checked, next to the sampled bags of every table.
FULL_HOST_TABLE_BYTES = 20 << 30


def _full_oracle(inp):
    """(column ranges, sum64, abs64) of the oracle over whole tables: every
    table when they fit in host memory, else the first and last four."""
    w = inp.w
    if w.table_bytes() <= FULL_HOST_TABLE_BYTES:
        s64, a64, _ = oracle.pool_inputs(inp, want_send=False)
        return [((0, w.T), s64, a64)]
    out = []
    for t0, t1 in ((0, 4), (w.T - 4, w.T)):
        B = w.B
        lo, hi = int(inp.offsets[t0 * B]), int(inp.offsets[t1 * B])
        s64, a64, _ = oracle.pool([inp.table(t) for t in range(t0, t1)], w.dtype, w.dims[t0:t1],
                                  inp.indices[lo:hi], inp.offsets[t0 * B:t1 * B + 1] - lo,
                                  None if inp.weights is None else inp.weights[lo:hi], B, w.R, w.C, want_send=False)
        out.append(((t0, t1), s64, a64))
    return out


def _check_columns(inp, send_np, parts):
    w = inp.w
    for (t0, t1), s64, a64 in parts:
        c0, c1 = w.col_off[t0], w.col_off[t1 - 1] + w.dims[t1 - 1]
        got = send_np[:, c0:c1]
        ok, err, bound = oracle.within_tolerance(got, s64, a64)
        if not ok:
            i = np.unravel_index(np.argmax(err - bound), err.shape)
            raise AssertionError(f"tables {t0}..{t1 - 1}: outside tolerance at {i}: gpu={got[i]} oracle={s64[i]}")


@pytest.mark.parametrize("name", ["tiny", "dlrm", "skewed", "mixed", "large"])
def test_full_size_sampled(name):
    """Full workload sizes, in the launch configuration the benchmark times
    (and in the default one where they differ), fused and unfused: every
    element written, every flag equal to the epoch, sampled bags of every
    table element by element against the per-bag oracle, and every element
    against the C oracle over whole tables (all of them where they fit in host
    memory; the first and last four of the large workload)."""
    import torch
    import bench
    w = synth.FULL[name]
    say("full", name, "generating inputs")
    inp = synth.make_inputs(w)
    say("full", name, "nnz", inp.nnz, "to device")
    dev = sdev.to_device(inp)
    launches = [dict(bench.PLAN_OPTS.get(name, {}))]
    if launches[0]:
        launches.append({})
    send, _, _ = new_buffers(w)
    parts = None
    for opts in launches:
        plan = make_plan(w, **opts)
        per_slice = w.T if opts.get("slice_granule") == 1 else 1
        flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
        for fused in (True, False):
            flags.zero_()
            send.fill_(float("nan"))
            run(plan, w, dev, send, flags, fused=fused)
            torch.cuda.synchronize()
            say("full", name, opts, "fused" if fused else "unfused", "ran; checking")
            assert not torch.isnan(send).any().item(), "some output element was never written"
            assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1, per_slice=per_slice))
            n = check_sampled(inp, send, n_bags=200)
            if parts is None:
                say("full", name, "oracle over whole tables")
                parts = _full_oracle(inp)
            _check_columns(inp, send.cpu().numpy(), parts)
            say("full", name, "checked", n, "sampled bags and", sum(p[1].size for p in parts), "elements")
        assert plan.status_ex() == (0, -1, 0, -1)
        plan.close()
    del dev, send, flags, parts
    torch.cuda.empty_cache()


def test_occupancy_query_and_full_persistent_grid():
    """ebag_a2a_occupancy reports the launch shape; a persistent grid of
    exactly that many workgroups per CU (weighted kernel) gives the same
    result as the one-workgroup-per-run grid."""
    import torch
    w = SMALL["mixed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    for waves in (2, 4):
        probe = make_plan(w, waves_per_wg=waves)
        max_wgs, cus, block, K = probe.occupancy(True)
        probe.close()
        assert cus == torch.cuda.get_device_properties(0).multi_processor_count
        assert block == 64 * waves and 1 <= K <= w.C and max_wgs >= 1
        plan = make_plan(w, waves_per_wg=waves, persistent_wgs_per_cu=max_wgs)
        send, _, flags = new_buffers(w)
        run(plan, w, dev, send, flags, fused=True)
        torch.cuda.synchronize()
        check_full(inp, send.cpu().numpy(), s64, a64)
        assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, 1))


def test_gather_probe_reads_in_bounds_rows():
    """The random-row probe used by the benchmark: a buffer of identical
    16-byte words folds to zero in every thread (an even number of loads per
    lane), for every supported row width."""
    import torch
    buf = torch.full((1 << 22,), 0x01020304, dtype=torch.int32, device="cuda")
    grid = 16
    out = torch.full((grid * 256,), -1, dtype=torch.int32, device="cuda")
    for rb in (16, 64, 128, 256, 512, 1024):
        out.fill_(-1)
        n = sdev.gather_probe(buf, rb, 16, grid, out, nt=(rb % 128 == 0))
        torch.cuda.synchronize()
        assert n == grid * 4 * 16 * 1024
        assert int(out.abs().sum()) == 0


@pytest.mark.parametrize("per_cu", [1, 3, -1])
def test_persistent_ticket_rearms_every_launch(per_cu):
    """Persistent grids claim runs from a ticket that the last workgroup out
    re-arms: several launches in a row (fused and unfused, both granules)
    each pool every bag and publish every flag once."""
    import torch
    w = SMALL["skewed_small"]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    s64, a64, _ = oracle.pool_inputs(inp)
    for granule in (0, 1):
        plan = make_plan(w, persistent_wgs_per_cu=per_cu, slice_granule=granule, bags_per_run=4)
        per_slice = w.T if granule else 1
        send, _, _ = new_buffers(w)
        flags = torch.zeros(w.n_chunks * per_slice, dtype=torch.int32, device="cuda")
        for epoch in range(1, 5):
            send.fill_(float("nan"))
            run(plan, w, dev, send, flags, fused=epoch % 2 == 1)
            torch.cuda.synchronize()
            check_full(inp, send.cpu().numpy(), s64, a64)
            assert np.array_equal(flags_np(flags), oracle.flags(w.B, w.R, w.C, epoch, per_slice=per_slice))
        assert plan.status_ex() == (0, -1, 0, -1)
