"""Pins of the CPU oracle to facts fixed outside the oracle itself.

Each ``pin_*`` takes a loaded oracle library (ctypes) and raises
AssertionError when the oracle disagrees with:
  * values worked out by hand (tests/golden/hand_example.txt),
  * exact integer arithmetic (Python ints) on integer-valued tables,
  * closed forms (all-ones tables, row-coded tables, single-row bags),
  * a library routine on a special case (torch.nn.functional.embedding_bag),
  * IEEE binary16 / bfloat16 decoding as done by numpy / torch,
  * the placement rule of Sec. III-A (first B/R samples to destination 0,
    {local batch, numTables x D} per destination, one flag per slice).
The mutation test runs every pin against deliberately broken copies of the
oracle and requires each copy to fail at least one pin.
"""
from __future__ import annotations

import ctypes
import fractions

import numpy as np

import oracle
from tests.golden import hand


def _pool(lib, tables, dtype, dims, indices, offsets, weights, B, R, C, nthreads=2, mean=False):
    return oracle.pool(tables, dtype, dims, indices, offsets, weights, B, R, C, nthreads=nthreads, lib=lib,
                       mean=mean)


def pin_hand(lib):
    d = hand.load()
    tabs = [np.array(t, dtype=np.float32) for t in d["tables"]]
    dims = [t.shape[1] for t in tabs]
    idx = np.array(d["indices"], dtype=np.int32)
    off = np.array(d["offsets"], dtype=np.int64)
    B, R, C = d["B"], d["R"], d["C"]
    S = B // R
    s64, a64, send = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C)
    assert np.array_equal(send.reshape(R, S, -1), d["sum"].astype(np.float32)), "hand sum"
    assert np.array_equal(s64.reshape(R, S, -1), d["sum"]), "hand sum64"
    w = np.array(d["weights"], dtype=np.float32)
    s64, a64, send = _pool(lib, tabs, 0, dims, idx, off, w, B, R, C)
    assert np.array_equal(s64.reshape(R, S, -1), d["wsum"]), "hand weighted sum"
    assert np.array_equal(send.reshape(R, S, -1), d["wsum"].astype(np.float32)), "hand weighted send"
    s64, a64, send = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C, mean=True)
    assert np.array_equal(s64.reshape(R, S, -1), d["mean"]), "hand mean64"
    assert np.array_equal(send.reshape(R, S, -1), d["mean"].astype(np.float32)), "hand mean"
    fl = oracle.flags(B, R, C, 1, lib=lib)
    assert fl.tolist() == d["flags"], "hand flags"
    fl = oracle.flags(B, R, C, 1, lib=lib, per_slice=len(tabs))
    assert fl.tolist() == d["flags_per_table"], "hand per-table flags"


def _random_bags(rng, T, B, rows, max_len, allow_empty=False):
    lo = 0 if allow_empty else 1
    lengths = rng.integers(lo, max_len + 1, size=T * B)
    off = np.zeros(T * B + 1, dtype=np.int64)
    off[1:] = np.cumsum(lengths)
    idx = np.empty(off[-1], dtype=np.int32)
    for t in range(T):
        a, b = off[t * B], off[(t + 1) * B]
        idx[a:b] = rng.integers(0, rows[t], size=b - a)
    # force some repeated indices inside bags
    for q in range(0, T * B, 7):
        if off[q + 1] - off[q] >= 2:
            idx[off[q] + 1] = idx[off[q]]
    return off, idx


def pin_integer_exact(lib):
    """Integer-valued tables: sums are exact, so every correct order gives the
    same bits; compare against Python integer arithmetic."""
    rng = np.random.default_rng(11)
    T, B, R, C = 3, 24, 4, 3
    rows = [17, 40, 9]
    dims = [4, 8, 12]
    for dtype in (0, 1, 2):
        ints = [rng.integers(-8, 9, size=(rows[t], dims[t])) for t in range(T)]
        if dtype == 0:
            tabs = [x.astype(np.float32) for x in ints]
        elif dtype == 1:
            tabs = [x.astype(np.float16) for x in ints]
        else:
            tabs = [(x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16) for x in ints]
        off, idx = _random_bags(rng, T, B, rows, 128, allow_empty=True)
        s64, a64, send = _pool(lib, tabs, dtype, dims, idx, off, None, B, R, C)
        col = 0
        S = B // R
        for t in range(T):
            for b in range(B):
                r, s = b // S, b % S
                ks = range(off[t * B + b], off[t * B + b + 1])
                exact = [sum(int(ints[t][idx[k]][j]) for k in ks) for j in range(dims[t])]
                mags = [sum(abs(int(ints[t][idx[k]][j])) for k in ks) for j in range(dims[t])]
                row = r * S + s
                assert s64[row, col:col + dims[t]].tolist() == [float(v) for v in exact], (dtype, t, b)
                assert a64[row, col:col + dims[t]].tolist() == [float(v) for v in mags], (dtype, t, b)
                assert np.array_equal(send[row, col:col + dims[t]], np.array(exact, dtype=np.float32))
            col += dims[t]


def pin_ones_and_weights(lib):
    """All-ones tables: plain sum = L, weighted sum = sum of weights (exact:
    float32 U[0,1) weights are multiples of 2^-24, so the fp64 sum is exact)."""
    rng = np.random.default_rng(5)
    T, B, R, C = 2, 16, 2, 4
    rows, dims = [30, 7], [8, 16]
    tabs = [np.ones((rows[t], dims[t]), dtype=np.float32) for t in range(T)]
    off, idx = _random_bags(rng, T, B, rows, 100, allow_empty=True)
    w = rng.random(off[-1], dtype=np.float32)
    s64, _, _ = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C)
    s64w, a64w, _ = _pool(lib, tabs, 0, dims, idx, off, w, B, R, C)
    col = 0
    for t in range(T):
        for b in range(B):
            L = off[t * B + b + 1] - off[t * B + b]
            assert np.all(s64[b, col:col + dims[t]] == L)
            exact = sum(fractions.Fraction(float(x)) for x in w[off[t * B + b]:off[t * B + b + 1]])
            assert np.all(s64w[b, col:col + dims[t]] == float(exact))
            assert np.all(a64w[b, col:col + dims[t]] == float(exact))
        col += dims[t]


def pin_row_coded(lib):
    """table_t[r][j] = r + 4096 t  =>  bag sum = sum(indices) + L * 4096 t
    (exact: every bag sum stays below 2^24)."""
    rng = np.random.default_rng(7)
    T, B, R, C = 4, 32, 2, 8
    N, D = 1000, 8
    tabs = [np.repeat((np.arange(N) + 4096 * t).astype(np.float32)[:, None], D, axis=1) for t in range(T)]
    off, idx = _random_bags(rng, T, B, [N] * T, 8)
    _, _, send = _pool(lib, tabs, 0, [D] * T, idx, off, None, B, R, C)
    for t in range(T):
        for b in range(B):
            ks = slice(off[t * B + b], off[t * B + b + 1])
            L = off[t * B + b + 1] - off[t * B + b]
            want = int(idx[ks].astype(np.int64).sum()) + L * 4096 * t
            assert np.all(send[b, t * D:(t + 1) * D] == want), (t, b)


def pin_placement(lib):
    """Single-row bags on tables whose element (t, r, j) stores the code
    (t * N + r) * D + j: every output element names its source, so the
    placement send[r][s][off_t + j], b = r * S + s, is checked element by
    element.  Also the worked example's shape (B = 4, two destinations, four
    tables, slices of two samples)."""
    for (T, N, dims, B, R, C) in [(3, 50, [4, 8, 12], 12, 3, 2), (4, 16, [4, 4, 4, 4], 4, 2, 2)]:
        D_max = max(dims)
        tabs = []
        for t in range(T):
            rr = np.arange(N)[:, None]
            jj = np.arange(dims[t])[None, :]
            tabs.append(((t * N + rr) * D_max + jj).astype(np.float32))
        rng = np.random.default_rng(T)
        off = np.arange(T * B + 1, dtype=np.int64)
        idx = rng.integers(0, N, size=T * B).astype(np.int32)
        _, _, send = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C)
        S = B // R
        view = send.reshape(R, S, sum(dims))
        col = 0
        for t in range(T):
            for b in range(B):
                r, s = b // S, b % S
                got = view[r, s, col:col + dims[t]].astype(np.int64)
                src_t, rem = divmod(got // D_max, N)
                assert np.all(src_t == t) and np.all(rem == idx[t * B + b]), (t, b)
                assert np.array_equal(got % D_max, np.arange(dims[t])), (t, b)
            col += dims[t]
        fl = oracle.flags(B, R, C, 3, lib=lib)
        assert fl.size == R * (S // C) and np.all(fl == 3)


def pin_fp16_decode(lib):
    """All 65536 binary16 patterns decode exactly as numpy's float16 does."""
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = pats.view(np.float16).astype(np.float64)
    f = lib.oracle_half_to_double
    got = np.array([f(int(p)) for p in pats])
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def pin_bf16_decode(lib):
    """All 65536 bfloat16 patterns decode exactly as torch's bfloat16 does."""
    import torch
    pats = np.arange(65536, dtype=np.int64)
    want = torch.from_numpy(pats.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    f = lib.oracle_bf16_to_double
    got = np.array([f(int(p)) for p in pats])
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def pin_fp16_pool(lib):
    """fp16 tables with subnormal and extreme values: pooled sums equal the
    numpy-decoded fp64 sums of the same rows (single-row and multi-row bags)."""
    rng = np.random.default_rng(3)
    pats = np.array([0x0001, 0x03FF, 0x0400, 0x3C00, 0xBC00, 0x7BFF, 0xFBFF, 0x8001, 0x3555], dtype=np.uint16)
    N, D, T, B, R, C = 9, 8, 1, 6, 1, 2
    tab = rng.choice(pats, size=(N, D)).view(np.float16)
    off = np.array([0, 1, 3, 6, 7, 9, 12], dtype=np.int64)
    idx = rng.integers(0, N, size=12).astype(np.int32)
    s64, _, _ = _pool(lib, [tab], 1, [D], idx, off, None, B, R, C)
    for b in range(B):
        want = np.zeros(D)
        for k in range(off[b], off[b + 1]):
            want = want + tab[idx[k]].astype(np.float64)
        assert np.array_equal(s64[b], want)


def pin_torch_embedding_bag(lib):
    """Special case that reduces to a library routine: per table,
    F.embedding_bag(mode='sum', per_sample_weights=w) in fp64, concatenated
    along the feature axis, is the [B][sum D] send buffer."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(13)
    T, B, R, C = 3, 40, 4, 5
    rows, dims = [100, 37, 64], [16, 8, 32]
    tabs = [rng.standard_normal((rows[t], dims[t])).astype(np.float32) for t in range(T)]
    off, idx = _random_bags(rng, T, B, rows, 50)
    w = rng.random(off[-1], dtype=np.float32)
    for weights in (None, w):
        s64, _, send = _pool(lib, tabs, 0, dims, idx, off, weights, B, R, C)
        parts = []
        for t in range(T):
            a, b = off[t * B], off[(t + 1) * B]
            inp = torch.from_numpy(idx[a:b].astype(np.int64))
            offs = torch.from_numpy((off[t * B:(t + 1) * B] - a).astype(np.int64))
            psw = None if weights is None else torch.from_numpy(weights[a:b].astype(np.float64))
            parts.append(F.embedding_bag(inp, torch.from_numpy(tabs[t].astype(np.float64)), offs,
                                         mode="sum", per_sample_weights=psw).numpy())
        ref = np.concatenate(parts, axis=1)
        assert np.allclose(s64, ref, rtol=1e-12, atol=1e-12)
        # fp32 output is the fp64 sum rounded to nearest: within half an ulp
        assert np.all(np.abs(send.astype(np.float64) - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12)


def pin_mean_closed_forms(lib):
    """Mean pooling: a bag of identical rows has that row as its mean for any
    length; a single-row bag is the row itself; an empty bag is zero;
    integer tables give the exact rational sum / L rounded once (compared
    with Python fractions)."""
    rng = np.random.default_rng(17)
    T, B, R, C = 2, 24, 3, 4
    rows, dims = [6, 50], [4, 12]
    const = [np.repeat(rng.standard_normal((1, dims[t])).astype(np.float32), rows[t], axis=0) for t in range(T)]
    off, idx = _random_bags(rng, T, B, rows, 60, allow_empty=True)
    s64, a64, send = _pool(lib, const, 0, dims, idx, off, None, B, R, C, mean=True)
    col = 0
    for t in range(T):
        for b in range(B):
            L = off[t * B + b + 1] - off[t * B + b]
            want = const[t][0].astype(np.float64) if L else np.zeros(dims[t])
            assert np.array_equal(s64[b, col:col + dims[t]], want), (t, b, L)
            assert np.array_equal(send[b, col:col + dims[t]], want.astype(np.float32))
            assert np.array_equal(a64[b, col:col + dims[t]], np.abs(want))
        col += dims[t]
    ints = [rng.integers(-8, 9, size=(rows[t], dims[t])) for t in range(T)]
    tabs = [x.astype(np.float32) for x in ints]
    s64, _, send = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C, mean=True)
    col = 0
    for t in range(T):
        for b in range(B):
            ks = range(off[t * B + b], off[t * B + b + 1])
            for j in range(dims[t]):
                want = (fractions.Fraction(sum(int(ints[t][idx[k]][j]) for k in ks), len(ks)) if len(ks)
                        else fractions.Fraction(0))
                assert s64[b, col + j] == float(want), (t, b, j)
        col += dims[t]
    single = np.arange(T * B + 1, dtype=np.int64)
    sidx = np.concatenate([rng.integers(0, rows[t], size=B) for t in range(T)]).astype(np.int32)
    _, _, send = _pool(lib, tabs, 0, dims, sidx, single, None, B, R, C, mean=True)
    col = 0
    for t in range(T):
        assert np.array_equal(send[:, col:col + dims[t]], tabs[t][sidx[t * B:(t + 1) * B]])
        col += dims[t]


def pin_torch_embedding_bag_mean(lib):
    """F.embedding_bag(mode='mean') per table in fp64, concatenated along the
    feature axis (PyTorch also returns zeros for an empty bag)."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(19)
    T, B, R, C = 3, 30, 5, 3
    rows, dims = [80, 33, 64], [8, 16, 4]
    tabs = [rng.standard_normal((rows[t], dims[t])).astype(np.float32) for t in range(T)]
    off, idx = _random_bags(rng, T, B, rows, 40, allow_empty=True)
    s64, _, _ = _pool(lib, tabs, 0, dims, idx, off, None, B, R, C, mean=True)
    parts = []
    for t in range(T):
        a, b = off[t * B], off[(t + 1) * B]
        inp = torch.from_numpy(idx[a:b].astype(np.int64))
        offs = torch.from_numpy((off[t * B:(t + 1) * B] - a).astype(np.int64))
        parts.append(F.embedding_bag(inp, torch.from_numpy(tabs[t].astype(np.float64)), offs, mode="mean").numpy())
    assert np.allclose(s64, np.concatenate(parts, axis=1), rtol=1e-12, atol=1e-12)


def pin_validation(lib):
    """Inputs outside the definition are rejected with the documented code."""
    tabs = [np.zeros((4, 4), dtype=np.float32)]
    off = np.array([0, 1, 2, 3, 4], dtype=np.int64)
    idx = np.array([0, 1, 2, 3], dtype=np.int32)
    cases = [
        (dict(B=4, R=3, C=1), "B % R"),
        (dict(B=4, R=2, C=3), "S % C"),
    ]
    for kw, _ in cases:
        try:
            _pool(lib, tabs, 0, [4], idx, off, None, **kw)
        except oracle.OracleError as e:
            assert "not zero" in str(e)
        else:
            raise AssertionError(kw)
    for bad_off, bad_idx, msg in [
        (np.array([0, 2, 1, 3, 4]), idx, "bad offsets"),
        (np.array([1, 1, 2, 3, 4]), idx, "bad offsets"),
        (np.array([0, 1, 2, 3, 3]), idx, "bad offsets"),
        (off, np.array([0, 1, 4, 3]), "index out of range"),
        (off, np.array([0, -1, 2, 3]), "index out of range"),
    ]:
        try:
            _pool(lib, tabs, 0, [4], bad_idx, bad_off, None, 4, 2, 1)
        except oracle.OracleError as e:
            assert msg in str(e), (msg, e)
        else:
            raise AssertionError(msg)
    try:
        _pool(lib, tabs, 0, [4], idx, off, np.ones(4, dtype=np.float32), 4, 2, 1, mean=True)
    except oracle.OracleError as e:
        assert "bad arguments" in str(e)
    else:
        raise AssertionError("mean pooling with weights accepted")


# ---- GEMV + AllReduce (Sec. III-B) -----------------------------------------


def pin_gemv_hand(lib):
    d = hand.load_gemv()
    A = [a.astype(np.float32) for a in d["A"]]
    x = [v.astype(np.float32) for v in d["x"]]
    y64, abs64, y = oracle.gemv_ar(A, x, 0, nthreads=2, lib=lib)
    assert np.array_equal(y64, d["y"]) and np.array_equal(abs64, d["abs"]), (y64, abs64)
    assert np.array_equal(y, d["y"].astype(np.float32))


def pin_gemv_integer_exact(lib):
    """Integer matrices and vectors: exact, compared with Python integers, for
    every storage type."""
    rng = np.random.default_rng(31)
    R, M = 3, 37
    Ks = [5, 64, 17]
    for dtype in (0, 1, 2):
        ia = [rng.integers(-8, 9, size=(M, K)) for K in Ks]
        ix = [rng.integers(-8, 9, size=K) for K in Ks]

        def enc(v):
            if dtype == 0:
                return v.astype(np.float32)
            if dtype == 1:
                return v.astype(np.float16)
            return (v.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        y64, abs64, y = oracle.gemv_ar([enc(a) for a in ia], [enc(v) for v in ix], dtype, nthreads=2, lib=lib)
        for i in range(M):
            terms = [int(ia[r][i, k]) * int(ix[r][k]) for r in range(R) for k in range(Ks[r])]
            assert y64[i] == float(sum(terms)) and abs64[i] == float(sum(abs(t) for t in terms)), (dtype, i)
            assert y[i] == np.float32(sum(terms))


def pin_gemv_matmul(lib):
    """Special case that reduces to a library routine: the column blocks
    concatenate to A = [A_0 | ... | A_{R-1}], x to their stacked parts, and the
    result is numpy's fp64 A @ x."""
    rng = np.random.default_rng(37)
    Ks = [40, 7, 128, 33]
    M = 90
    A = [rng.standard_normal((M, K)).astype(np.float32) for K in Ks]
    x = [rng.standard_normal(K).astype(np.float32) for K in Ks]
    y64, abs64, y = oracle.gemv_ar(A, x, 0, nthreads=3, lib=lib)
    full = np.concatenate([a.astype(np.float64) for a in A], axis=1)
    xv = np.concatenate([v.astype(np.float64) for v in x])
    assert np.allclose(y64, full @ xv, rtol=1e-12, atol=1e-12)
    assert np.allclose(abs64, np.abs(full) @ np.abs(xv), rtol=1e-12, atol=1e-12)
    assert np.all(np.abs(y.astype(np.float64) - y64) <= 2.0 ** -24 * np.abs(y64) + 1e-300)


def pin_gemv_closed_forms(lib):
    """All-ones matrices give the sum of every rank's x in each row; an
    identity block on rank 0 with zero blocks elsewhere returns x_0."""
    rng = np.random.default_rng(41)
    Ks = [6, 10]
    M = 6
    x = [rng.integers(-100, 100, size=K).astype(np.float32) for K in Ks]
    y64, _, _ = oracle.gemv_ar([np.ones((M, K), np.float32) for K in Ks], x, 0, nthreads=1, lib=lib)
    assert np.all(y64 == float(sum(v.astype(np.int64).sum() for v in x)))
    A = [np.eye(M, Ks[0], dtype=np.float32), np.zeros((M, Ks[1]), np.float32)]
    y64, _, y = oracle.gemv_ar(A, x, 0, nthreads=1, lib=lib)
    assert np.array_equal(y, x[0])


def pin_gemv_validation(lib):
    A = [np.zeros((4, 3), np.float32)]
    for bad in ([np.zeros(4, np.float32)], [np.zeros(3, np.float32), np.zeros(3, np.float32)]):
        try:
            oracle.gemv_ar(A, bad, 0, lib=lib)
        except oracle.OracleError:
            pass
        else:
            raise AssertionError("shape mismatch accepted")


# ---- Embedding backward -----------------------------------------------------


def pin_backward_hand(lib):
    d = hand.load()
    bw = hand.load_backward()
    off = np.array(d["offsets"], dtype=np.int64)
    w = np.array(d["weights"], dtype=np.float32)
    dims = [4, 4]
    for key, weights, mean in (("sum", None, False), ("wsum", w, False), ("mean", None, True)):
        got = oracle.backward(dims, off, weights, bw["grad"], d["B"], d["R"], mean=mean, lib=lib)
        assert np.array_equal(got.reshape(-1, 4), bw[key]), key


def pin_backward_torch(lib):
    """Special case that reduces to a library routine: scattering the
    per-lookup rows onto their table rows gives the dense gradient that
    torch's autograd computes for F.embedding_bag (sum, weighted sum, mean)."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(43)
    T, B, R = 3, 24, 4
    rows, dims = [50, 9, 70], [8, 16, 4]
    off, idx = _random_bags(rng, T, B, rows, 30, allow_empty=True)
    grad = rng.standard_normal((B, sum(dims))).astype(np.float32)
    w = rng.random(off[-1], dtype=np.float32)
    for weights, mean in ((None, False), (w, False), (None, True)):
        vals = oracle.backward(dims, off, weights, grad, B, R, mean=mean, lib=lib).astype(np.float64)
        base, col = 0, 0
        for t in range(T):
            a, b = off[t * B], off[(t + 1) * B]
            tab = torch.zeros((rows[t], dims[t]), dtype=torch.float64, requires_grad=True)
            psw = None if weights is None else torch.from_numpy(weights[a:b].astype(np.float64))
            out = F.embedding_bag(torch.from_numpy(idx[a:b].astype(np.int64)), tab,
                                  torch.from_numpy((off[t * B:(t + 1) * B] - a).astype(np.int64)),
                                  mode="mean" if mean else "sum", per_sample_weights=psw)
            out.backward(torch.from_numpy(grad[:, col:col + dims[t]].astype(np.float64)))
            mine = np.zeros((rows[t], dims[t]))
            np.add.at(mine, idx[a:b], vals[base:base + (b - a) * dims[t]].reshape(b - a, dims[t]))
            assert np.allclose(mine, tab.grad.numpy(), rtol=1e-6, atol=1e-6), (t, mean, weights is None)
            base += (b - a) * dims[t]
            col += dims[t]


def pin_backward_closed_forms(lib):
    """A constant pooled gradient c: every plain row is c, every mean row c/L,
    every weighted row c * w_k (single fp32 rounding each)."""
    rng = np.random.default_rng(47)
    T, B, R = 2, 12, 3
    rows, dims = [20, 20], [8, 4]
    off, idx = _random_bags(rng, T, B, rows, 20, allow_empty=True)
    c = np.float32(0.7)
    grad = np.full((B, sum(dims)), c, dtype=np.float32)
    w = rng.random(off[-1], dtype=np.float32)
    plain = oracle.backward(dims, off, None, grad, B, R, lib=lib)
    assert np.all(plain == c)
    wv = oracle.backward(dims, off, w, grad, B, R, lib=lib)
    mv = oracle.backward(dims, off, None, grad, B, R, mean=True, lib=lib)
    base = 0
    for t in range(T):
        for b in range(B):
            lo, hi = off[t * B + b], off[t * B + b + 1]
            for k in range(lo, hi):
                seg = slice(base + (k - off[t * B]) * dims[t], base + (k - off[t * B] + 1) * dims[t])
                assert np.all(wv[seg] == np.float32(np.float64(w[k]) * np.float64(c)))
                assert np.all(mv[seg] == np.float32(np.float64(c) / (hi - lo)))
        base += (off[(t + 1) * B] - off[t * B]) * dims[t]


ALL_PINS = [pin_hand, pin_integer_exact, pin_ones_and_weights, pin_row_coded, pin_placement,
            pin_fp16_decode, pin_bf16_decode, pin_fp16_pool, pin_torch_embedding_bag, pin_mean_closed_forms,
            pin_torch_embedding_bag_mean, pin_validation, pin_gemv_hand, pin_gemv_integer_exact, pin_gemv_matmul,
            pin_gemv_closed_forms, pin_gemv_validation, pin_backward_hand, pin_backward_torch,
            pin_backward_closed_forms]
