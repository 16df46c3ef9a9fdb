"""Seeded input generator: determinism, distributions and value function (no GPU)."""
import hashlib

import numpy as np
import pytest

import synth
from synth import gen


def _digest(inp):
    h = hashlib.sha256()
    for a in (inp.lengths, inp.offsets, inp.indices, inp.weights):
        if a is not None:
            h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_splitmix64_known_answers():
    # SplitMix64 seeded with 0 (Steele, Lea, Flood 2014): first two outputs.
    assert int(gen.splitmix64(np.uint64(0))) == 0xE220A8397B1DCDAF
    assert int(gen.splitmix64(np.uint64(0x9E3779B97F4A7C15))) == 0x6E789E6AA1B965F4


@pytest.mark.parametrize("name", ["tiny", "tiny_int", "dlrm", "mixed"])
def test_deterministic(name):
    w = synth.ALL[name]
    w = synth.scaled(w, rows=w.rows[0], B=w.R * w.C) if name in ("dlrm", "mixed") else w
    a, b = synth.make_inputs(w), synth.make_inputs(w)
    assert _digest(a) == _digest(b)
    if a.host_tables is not None:
        assert all(np.array_equal(x, y) for x, y in zip(a.host_tables, b.host_tables))


def test_lengths_and_offsets():
    for base in (synth.SKEWED, synth.LARGE, synth.MIXED):
        w = synth.scaled(base, rows=1000, B=base.R * base.C * 2, T=4)
        inp = synth.make_inputs(w)
        L = inp.lengths
        kind, *p = w.lengths.split(":")
        lo, hi = (int(p[0]), int(p[1])) if kind == "uniform" else (int(p[1]), int(p[2]))
        assert L.min() >= lo and L.max() <= hi
        assert inp.offsets[0] == 0 and np.all(np.diff(inp.offsets) == L)
        assert inp.indices.min() >= 0 and inp.indices.max() < w.rows[0]
        if kind == "poisson":
            assert abs(L.mean() - 40) < 1.0
        else:
            assert abs(L.mean() - (lo + hi) / 2) < 0.05 * hi


def test_zipf_head_share():
    w = synth.scaled(synth.SKEWED, rows=20000, B=synth.SKEWED.R * synth.SKEWED.C * 4, T=2)
    inp = synth.make_inputs(w)
    n = w.rows[0]
    H = np.sum(np.arange(1, n + 1, dtype=np.float64) ** -1.05)
    idx = inp.indices[inp.offsets[0]:inp.offsets[w.B]]
    top = np.bincount(idx).max() / idx.size
    assert abs(top - 1.0 / H) < 0.01  # rank 1 carries 1/H of the mass


def test_counter_values_range_and_storage():
    rows = np.arange(0, 5000, 7)
    v = gen.counter_values(12345, 64, rows, 0, synth.F32)
    assert v.dtype == np.float32 and v.shape == (rows.size, 64)
    assert np.all(np.abs(v) < 0.05) and abs(float(v.mean())) < 1e-3
    c = gen.counter_values(12345, 64, rows, 1, synth.F32)
    assert set(np.unique(c).tolist()) <= set(range(-8, 9))
    h = gen.counter_values(12345, 64, rows, 0, synth.F16)
    assert h.dtype == np.float16 and np.array_equal(h, v.astype(np.float16))


def test_bf16_rounding_matches_torch():
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 0.0, 3.0e-39], dtype=np.float32)])
    ours = gen.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("dtype", [synth.F32, synth.F16, synth.BF16])
@pytest.mark.parametrize("kind", [0, 1])
def test_host_fill_matches_numpy(dtype, kind):
    from synth import host
    seed = gen.table_seed(4, 9)
    x = host.fill(777, 24, dtype, seed, kind, nthreads=3)
    want = gen.counter_values(seed, 24, np.arange(777), kind, dtype)
    assert np.array_equal(np.ascontiguousarray(x).view(np.uint8), np.ascontiguousarray(want).view(np.uint8))


def test_host_half_rounding_matches_numpy():
    from synth import host
    lib = host.load()
    rng = np.random.default_rng(2)
    xs = np.concatenate([rng.standard_normal(20000).astype(np.float32) * np.float32(0.05),
                         (rng.standard_normal(20000) * 1e-5).astype(np.float32),
                         np.array([6.1035156e-05, 6.0975552e-05, 5.96e-08, 2.98e-08, 2.99e-08, 65504.0, 1.0009766,
                                   1.00048828125, 1.00146484375, -0.0, 0.0], dtype=np.float32)])
    got = np.array([lib.synth_half_rne(float(v)) for v in xs], dtype=np.uint16)
    assert np.array_equal(got, xs.astype(np.float16).view(np.uint16))
