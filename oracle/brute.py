"""Pure-Python brute force of the pooled send layout, for tiny inputs.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Written with plain loops and Python floats (IEEE fp64) straight from the
definition in Sec. III-A: output vector (t, b) is the (weighted) sum of the
rows named by bag (t, b); the batch is split into R contiguous parts of
S = B / R samples (the first part to destination 0); destination r receives
{S, sum of D_t} with table t in columns off_t .. off_t + D_t; one ready flag
per (destination, slice of C samples), equal to the number of forwards.
"""
from __future__ import annotations


def pool(tables, indices, offsets, weights, B, R, mean=False):
    """tables: list of T lists of rows (each row a list of numbers).
    Returns send as a nested list send[r][s][col] of Python floats; mean=True
    divides each bag's sum by its length (an empty bag stays zero)."""
    T = len(tables)
    dims = [len(tab[0]) for tab in tables]
    S = B // R
    width = sum(dims)
    send = [[[0.0] * width for _ in range(S)] for _ in range(R)]
    col = 0
    for t in range(T):
        for b in range(B):
            r, s = b // S, b % S
            lo, hi = offsets[t * B + b], offsets[t * B + b + 1]
            for j in range(dims[t]):
                acc = 0.0
                for k in range(lo, hi):
                    w = 1.0 if weights is None else float(weights[k])
                    acc += w * float(tables[t][indices[k]][j])
                if mean and hi > lo:
                    acc /= hi - lo
                send[r][s][col + j] = acc
        col += dims[t]
    return send


def flags(B, R, C, epoch):
    S = B // R
    return [[epoch for _ in range(S // C)] for _ in range(R)]
