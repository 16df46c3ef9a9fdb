"""Per-bag oracle in numpy for workloads whose tables do not fit on the host.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Rows are fetched on demand through ``inputs.table_rows(t, rows)`` (the seeded
generator recomputes them from its counter-based value function), widened to
fp64 exactly and summed in index order -- the same definition as ``oracle.c``
(Sec. III-A: one pooled vector per logical workgroup), written independently.
"""
from __future__ import annotations

import numpy as np

F32, F16, BF16 = 0, 1, 2


def widen(stored: np.ndarray, dtype: int) -> np.ndarray:
    """Storage values -> exact fp64."""
    if dtype == F32:
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    if dtype == F16:
        return np.asarray(stored, dtype=np.float16).astype(np.float64)
    bits = np.asarray(stored, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return bits.view(np.float32).astype(np.float64)


def column_offsets(dims):
    off = np.zeros(len(dims), dtype=np.int64)
    off[1:] = np.cumsum(dims)[:-1]
    return off


def placement(B, R, dims, t, b):
    """(destination r, local row s, first column) of pooled vector (t, b) in
    the send layout [R][B/R][sum D]: the first B/R samples go to destination 0."""
    S = B // R
    return b // S, b % S, int(column_offsets(dims)[t])


def flat_row(B, R, b):
    """Row of the [B][sum D] view of the send buffer that holds sample b."""
    S = B // R
    r, s = b // S, b % S
    return r * S + s


def pool_bag(inputs, t, b, mean=False):
    """fp64 (sum, sum of |terms|) of bag (t, b), each of length D_t; with
    mean=True both divided by the bag length (zeros for an empty bag)."""
    w = inputs.w
    lo, hi = int(inputs.offsets[t * w.B + b]), int(inputs.offsets[t * w.B + b + 1])
    D = w.dims[t]
    if hi == lo:
        return np.zeros(D), np.zeros(D)
    rows = widen(inputs.table_rows(t, inputs.indices[lo:hi]), w.dtype)  # (L, D)
    if inputs.weights is not None:
        rows = rows * inputs.weights[lo:hi].astype(np.float64)[:, None]
    s = np.zeros(D)
    a = np.zeros(D)
    for k in range(rows.shape[0]):      # index order, like the definition
        s += rows[k]
        a += np.abs(rows[k])
    if mean:
        s /= rows.shape[0]
        a /= rows.shape[0]
    return s, a


def pool_bags(inputs, bags, mean=False):
    """Expected values for a list of (t, b) bags.

    Returns a list of (t, b, flat_row, col0, sum64, abs64)."""
    w = inputs.w
    off = column_offsets(w.dims)
    out = []
    for t, b in bags:
        s, a = pool_bag(inputs, int(t), int(b), mean)
        out.append((int(t), int(b), flat_row(w.B, w.R, int(b)), int(off[t]), s, a))
    return out


def sample_bags(w, n, seed=0):
    """A deterministic spread of bags over every chunk, table and the last
    sample of each destination (ragged edges)."""
    rng = np.random.default_rng(seed)
    bags = set()
    S = w.B // w.R
    for r in range(w.R):
        for b in (r * S, r * S + S - 1):
            bags.add((int(rng.integers(0, w.T)), b))
    for t in range(w.T):
        bags.add((t, int(rng.integers(0, w.B))))
    for g in range(w.B // w.C):
        bags.add((int(rng.integers(0, w.T)), g * w.C + int(rng.integers(0, w.C))))
    while len(bags) < n:
        bags.add((int(rng.integers(0, w.T)), int(rng.integers(0, w.B))))
    return sorted(bags)


def backward_bag(inputs, grad, t, b, mean=False):
    """Per-lookup gradient rows of bag (t, b), fp32 [L, D_t]: lookup k gets
    w_k * g (sum and weighted sum; w_k = 1 without weights) or g / L (mean),
    g = grad[b, off_t : off_t + D_t] -- the derivative of the pooled value
    with respect to each gathered row (Sec. III-A pooling, run backwards as
    in the training pass of Sec. IV-D), each value one fp32 operation."""
    w = inputs.w
    lo, hi = int(inputs.offsets[t * w.B + b]), int(inputs.offsets[t * w.B + b + 1])
    D = w.dims[t]
    col = int(column_offsets(w.dims)[t])
    g = np.asarray(grad[b, col:col + D], dtype=np.float32)
    L = hi - lo
    rows = np.empty((L, D), dtype=np.float32)
    for k in range(L):
        if mean:
            rows[k] = g / np.float32(L)
        elif inputs.weights is not None:
            rows[k] = np.float32(inputs.weights[lo + k]) * g
        else:
            rows[k] = g
    return rows


def backward_value_offset(inputs, t, b):
    """First value of bag (t, b) in the backward's output: the table blocks
    (nnz_t x D_t values each) follow each other in table order, lookups in
    order inside a block."""
    w = inputs.w
    base = 0
    for u in range(t):
        base += int(inputs.offsets[(u + 1) * w.B] - inputs.offsets[u * w.B]) * w.dims[u]
    return base + int(inputs.offsets[t * w.B + b] - inputs.offsets[t * w.B]) * w.dims[t]
