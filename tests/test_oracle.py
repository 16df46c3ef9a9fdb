"""The CPU oracle against what the paper and mathematics fix (no GPU)."""
import numpy as np
import pytest

import oracle
from oracle import brute, sampled
from synth import DLRM, LARGE, MIXED, SKEWED, make_inputs, scaled
from tests import oracle_pins
from tests.golden import hand


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(oracle_lib, pin):
    pin(oracle_lib)


def test_brute_matches_hand():
    d = hand.load()
    for key, w, mean in (("sum", None, False), ("wsum", d["weights"], False), ("mean", None, True)):
        got = brute.pool(d["tables"], d["indices"], d["offsets"], w, d["B"], d["R"], mean=mean)
        assert np.array_equal(np.array(got), d[key])
    assert [f for row in brute.flags(d["B"], d["R"], d["C"], 1) for f in row] == d["flags"]


def test_brute_matches_c_random(oracle_lib):
    rng = np.random.default_rng(21)
    T, B, R, C = 3, 12, 3, 2
    rows, dims = [11, 5, 20], [4, 8, 4]
    tabs = [rng.standard_normal((rows[t], dims[t])).astype(np.float32) for t in range(T)]
    off, idx = oracle_pins._random_bags(rng, T, B, rows, 9, allow_empty=True)
    w = rng.random(off[-1], dtype=np.float32)
    for weights, mean in ((None, False), (w, False), (None, True)):
        s64, _, send = oracle.pool(tabs, 0, dims, idx, off, weights, B, R, C, lib=oracle_lib, mean=mean)
        ref = np.array(brute.pool([t.tolist() for t in tabs], idx.tolist(), off.tolist(),
                                  None if weights is None else weights.tolist(), B, R, mean=mean))
        assert np.array_equal(s64, ref.reshape(B, -1))


@pytest.mark.parametrize("base", [DLRM, SKEWED, LARGE, MIXED], ids=lambda w: w.name)
def test_sampled_matches_c(oracle_lib, base):
    """The numpy per-bag oracle and the C oracle agree bit for bit (same
    operations in the same order) on small versions of every workload."""
    w = scaled(base, rows=300, B=base.R * base.C, T=min(base.T, 8))
    inp = make_inputs(w)
    bags = sampled.sample_bags(w, 40)
    for mean in ((False, True) if inp.weights is None else (False,)):
        s64, a64, send = oracle.pool_inputs(inp, lib=oracle_lib, mean=mean)
        for t, b, row, col, s, a in sampled.pool_bags(inp, bags, mean=mean):
            D = w.dims[t]
            assert np.array_equal(s64[row, col:col + D], s), (t, b)
            assert np.array_equal(a64[row, col:col + D], a), (t, b)


def test_fp32_summation_within_tolerance():
    """Reading of the tolerance: recursive fp32 summation (any order) of up to
    128 terms stays within 1e-5 * sum|terms| + 1e-6 of the fp64 sum, since
    its error is at most (L - 1) * 2^-24 * sum|terms|."""
    rng = np.random.default_rng(1)
    for L in (1, 8, 32, 64, 128):
        terms = rng.standard_normal((2000, L)).astype(np.float32)
        acc = np.zeros(2000, dtype=np.float32)
        for k in rng.permutation(L):
            acc = (acc + terms[:, k]).astype(np.float32)
        s64 = terms.astype(np.float64).sum(1)
        a64 = np.abs(terms.astype(np.float64)).sum(1)
        ok, _, _ = oracle.within_tolerance(acc, s64, a64)
        assert ok
        assert np.all(np.abs(acc - s64) <= (L - 1) * 2.0 ** -24 * a64 + 1e-30)


def test_flags_shape():
    f = oracle.flags(4096, 8, 64, 5)
    assert f.shape == (64,) and np.all(f == 5)
    with pytest.raises(oracle.OracleError):
        oracle.flags(4096, 8, 100, 1)


@pytest.mark.parametrize("base", [DLRM, SKEWED, LARGE, MIXED], ids=lambda w: w.name)
def test_sampled_backward_matches_c(oracle_lib, base):
    """The numpy per-bag backward (values and their position) and the C
    oracle's whole backward agree bit for bit on small versions of every
    workload, for sum / weighted sum and mean."""
    w = scaled(base, rows=300, B=base.R * base.C, T=min(base.T, 8))
    inp = make_inputs(w)
    grad = np.random.default_rng(3).standard_normal((w.B, w.sum_dim)).astype(np.float32)
    for mean in ((False, True) if inp.weights is None else (False,)):
        full = oracle.backward(w.dims, inp.offsets, inp.weights, grad, w.B, w.R, mean=mean, lib=oracle_lib)
        for t, b in sampled.sample_bags(w, 60, seed=1):
            want = sampled.backward_bag(inp, grad, t, b, mean=mean).reshape(-1)
            o = sampled.backward_value_offset(inp, t, b)
            assert np.array_equal(full[o:o + want.size].view(np.uint32), want.view(np.uint32)), (t, b, mean)
