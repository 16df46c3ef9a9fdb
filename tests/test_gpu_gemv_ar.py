"""Fused GEMV + AllReduce (Sec. III-B) through the C ABI against the oracle.

Tolerance, from the kernel's arithmetic: every output is a tree of fp32
operations whose longest path has N fused multiply-adds inside one 16-byte
vector (N = 4 fp32, 8 fp16/bf16 elements), ceil(V / 64) per-lane vector
accumulations (V = K_r * elt / 16), 6 cross-lane butterfly levels and R
rank additions; each rounds once, so |gpu - y64| <= depth * 2^-24 * sum|terms|
to first order.  Integer-valued inputs are exact and compared bitwise."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _encode(v, dtype):
    if dtype == synth.F32:
        return v.astype(np.float32)
    if dtype == synth.F16:
        return v.astype(np.float16)
    return synth.gen.f32_to_bf16_bits(v.astype(np.float32))


def _to_dev(a, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == synth.BF16:
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.cuda()


def _inputs(R, M, Ks, dtype, seed, integer=False):
    rng = np.random.default_rng([2305, 6942, 311, seed])
    if integer:
        A = [_encode(rng.integers(-8, 9, size=(M, K)), dtype) for K in Ks]
        x = [_encode(rng.integers(-8, 9, size=K), dtype) for K in Ks]
    else:
        A = [_encode(rng.standard_normal((M, K)), dtype) for K in Ks]
        x = [_encode(rng.standard_normal(K), dtype) for K in Ks]
    return A, x


def _depth(R, Ks, dtype):
    N = 4 if dtype == synth.F32 else 8
    elt = 4 if dtype == synth.F32 else 2
    return N + max(-(-(K * elt // 16) // 64) for K in Ks) + 6 + R


def _run(R, M, Ks, dtype, seed, integer=False, epochs=2, **opts):
    import torch
    import paper_2305_06942_amd as ebag
    A, x = _inputs(R, M, Ks, dtype, seed, integer)
    y64, abs64, yf = oracle.gemv_ar(A, x, dtype)
    dA = [_to_dev(a, dtype) for a in A]
    dx = [_to_dev(v, dtype) for v in x]
    plan = ebag.GemvAR(R, M, Ks, dtype, **opts)
    P, block, n_tiles, resident, tile_rows = plan.launch_info()
    assert n_tiles == -(-M // tile_rows)
    assert 1 <= P <= n_tiles and (opts.get("reduce_mode", 0) == 0 or R * P <= resident)
    rel = _depth(R, Ks, dtype) * 2.0 ** -24
    outs = []
    for fused in (True, False):
        y = [torch.full((M,), float("nan"), device="cuda") for _ in range(R)]
        flags = torch.zeros(R * P, dtype=torch.int32, device="cuda")
        for e in range(1, epochs + 1):
            (plan.forward if fused else plan.unfused_forward)(dA, dx, y, flags)
            torch.cuda.synchronize()
            assert np.all(flags.cpu().numpy() == e)
        assert plan.status() == (0, -1)
        got = [v.cpu().numpy() for v in y]
        for r in range(1, R):
            assert np.array_equal(got[r].view(np.uint32), got[0].view(np.uint32)), f"rank {r} differs from rank 0"
        if integer:
            assert np.array_equal(got[0].view(np.uint32), yf.view(np.uint32))
        else:
            err = np.abs(got[0].astype(np.float64) - y64)
            bound = rel * abs64 + 1e-30
            assert np.all(err <= bound), f"max excess {(err - bound).max()} at {int(np.argmax(err - bound))}"
        outs.append(got[0])
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32)), "fused and unfused differ"
    plan.close()


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("dtype", [synth.F32, synth.F16, synth.BF16])
@pytest.mark.parametrize("R", [1, 2, 4, 8])
def test_gemv_ar_parity(dtype, R, mode):
    elt = 4 if dtype == synth.F32 else 2
    Ks = [(16 // elt) * k for k in ([37, 64, 5, 129, 256, 16, 3, 200][:R])]
    _run(R, 3000 + 37, Ks, dtype, seed=R * 3 + dtype, reduce_mode=mode)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("dtype", [synth.F32, synth.F16, synth.BF16])
def test_gemv_ar_integer_exact(dtype, mode):
    elt = 4 if dtype == synth.F32 else 2
    _run(4, 2048 + 5, [(16 // elt) * k for k in (64, 32, 100, 8)], dtype, seed=7, integer=True, reduce_mode=mode)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("opts", [dict(tile_rows=1), dict(tile_rows=16), dict(tile_rows=1000),
                                  dict(wgs_per_rank=1), dict(wgs_per_rank=3), dict(comm_aware=0),
                                  dict(waves_per_wg=1), dict(waves_per_wg=16)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_gemv_ar_launch_options(opts, mode):
    _run(4, 1500, [512, 256, 1024, 128], synth.F16, seed=11, reduce_mode=mode, **opts)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("M", [16384, 32768, 65536])
def test_gemv_ar_benchmark_shapes(M, mode):
    """The benchmarked shapes: M outputs, K = 8192 over 4 ranks, fp16."""
    _run(4, M, [2048] * 4, synth.F16, seed=13, epochs=2, reduce_mode=mode)


def test_gemv_ar_suppressed_peer_flag_times_out():
    """A peer flag that is never set makes its owner workgroup give up after
    the timeout and name the flag; exactly that workgroup's tiles stay
    unwritten in every rank's output, every other row is reduced."""
    import torch
    import paper_2305_06942_amd as ebag
    R, M, Ks, dtype, P = 2, 1024, [256, 256], synth.F32, 4
    A, x = _inputs(R, M, Ks, dtype, seed=17)
    y64, abs64, _ = oracle.gemv_ar(A, x, dtype)
    dA = [_to_dev(a, dtype) for a in A]
    dx = [_to_dev(v, dtype) for v in x]
    f = (1 * R + 0) * P + 0  # owner 1, source rank 0, workgroup 0
    plan = ebag.GemvAR(R, M, Ks, dtype, tile_rows=64, wgs_per_rank=P, debug_suppress_flag=f, timeout_us=20000,
                       reduce_mode=1)
    assert plan.launch_info()[0] == P and plan.launch_info()[2] == 16
    y = [torch.full((M,), float("nan"), device="cuda") for _ in range(R)]
    plan.forward(dA, dx, y)
    assert plan.status() == (1, f)
    plan.reset()
    assert plan.status() == (0, -1)
    # owner 1 holds tiles 8..15; its workgroup 0 handles tiles 8 and 12
    missing = np.zeros(M, dtype=bool)
    for t in (8, 12):
        missing[t * 64:(t + 1) * 64] = True
    rel = _depth(R, Ks, dtype) * 2.0 ** -24
    for r in range(R):
        got = y[r].cpu().numpy()
        assert np.all(np.isnan(got[missing]))
        assert np.all(np.abs(got[~missing] - y64[~missing]) <= rel * abs64[~missing] + 1e-30)


@pytest.mark.parametrize("seed", range(32))
def test_gemv_ar_random(seed):
    """Seeded random shapes and launches: ranks 1..16, ragged M, per-rank K
    (16-byte multiples, up to the 64 KiB LDS limit), every storage type,
    integer or normal values, tile height, waves, workgroups per rank, order
    and reduction mode; two epochs each, fused and unfused."""
    rng = np.random.default_rng([2305, 6942, 5, seed])
    dtype = int(rng.integers(0, 3))
    elt = 4 if dtype == synth.F32 else 2
    R = int(rng.choice([1, 2, 3, 4, 7, 8, 16]))
    M = int(rng.integers(1, 5000))
    Ks = [(16 // elt) * int(rng.integers(1, 300)) for _ in range(R)]
    opts = dict(tile_rows=int(rng.choice([0, 1, 7, 32, 64, 128, 300])), waves_per_wg=int(rng.choice([1, 2, 4, 16])),
                comm_aware=int(rng.integers(0, 2)), reduce_mode=int(rng.integers(0, 2)))
    if rng.random() < 0.3:
        opts["wgs_per_rank"] = int(rng.integers(1, 9))
    _run(R, M, Ks, dtype, seed=1000 + seed, integer=bool(rng.integers(0, 2)), **opts)


def test_overlapping_forwards_on_two_streams_refused():
    """A forward (fused or not) enqueued on another stream while the plan's
    last forward has not completed returns EBAG_EBUSY and enqueues nothing;
    on the same stream it runs, ordered after the first.  The first forward
    is held back by a bounded spin kernel queued ahead of it; every output
    and flag is then checked against the oracle and the two forwards."""
    import torch
    import paper_2305_06942_amd as ebag
    if not hasattr(torch.cuda, "_sleep"):
        pytest.skip("torch.cuda._sleep is not available")
    R, M, Ks, dtype = 4, 4096 + 37, [1024, 512, 2048, 256], synth.F16
    A, x = _inputs(R, M, Ks, dtype, 77)
    y64, abs64, _ = oracle.gemv_ar(A, x, dtype)
    dA = [_to_dev(a, dtype) for a in A]
    dx = [_to_dev(v, dtype) for v in x]
    plan = ebag.GemvAR(R, M, Ks, dtype)
    P = plan.launch_info()[0]
    y = [torch.full((M,), float("nan"), device="cuda") for _ in range(R)]
    flags = torch.zeros(R * P, dtype=torch.int32, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        torch.cuda._sleep(200_000_000)
        plan.forward(dA, dx, y, flags)
    for call in (plan.forward, plan.unfused_forward):
        with pytest.raises(ebag.EbagError) as e:
            call(dA, dx, y, flags, stream=s2)
        assert e.value.code == ebag.abi.EBAG_EBUSY
    with torch.cuda.stream(s1):
        plan.unfused_forward(dA, dx, y, flags)  # same stream: ordered after the first
    torch.cuda.synchronize()
    assert np.all(flags.cpu().numpy() == 2), "two forwards ran, the refused ones enqueued nothing"
    assert plan.status() == (0, -1)
    bound = _depth(R, Ks, dtype) * 2.0 ** -24 * abs64 + 1e-30
    for r in range(R):
        err = np.abs(y[r].cpu().numpy().astype(np.float64) - y64)
        assert np.all(err <= bound), f"rank {r}"
    plan.forward(dA, dx, y, flags, stream=s2)  # the first has completed: another stream is accepted
    torch.cuda.synchronize()
    assert np.all(flags.cpu().numpy() == 3)
    plan.close()
