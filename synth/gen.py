"""Seeded synthetic inputs for pooled embedding-bag workloads.

This module is shared by the CPU oracle and by the GPU path, so it holds no
part of the pooling / placement / flag arithmetic: it only draws bag lengths,
indices, per-index weights and table values.

Randomness:
  * numpy ``SeedSequence([2305, 6942, cfg_id])`` spawns independent streams for
    bag lengths, indices, per-table permutations, weights and (Tiny only) table
    values.
  * Table values of the large workloads come from a counter-based function so
    that the GPU can fill 10^11-byte tables in place and the host can recompute
    any row without materialising the table:

        u   = splitmix64(seed_t ^ (row * D_t + j)) >> 40      (24-bit integer)
        x   = float32(u - 2^23) * 2^-24                       (exact)
        v   = x * float32(0.1)                                (one IEEE RNE multiply: U(-0.05, 0.05))
        cint variant: v = float32((u mod 17) - 8)             (integers in [-8, 8])

    then round-to-nearest-even to fp16 / bf16 storage.  SplitMix64 is the
    generator published by Steele, Lea and Flood (OOPSLA 2014).
"""
from __future__ import annotations

import dataclasses
import functools
from typing import List, Optional

import numpy as np

from .configs import BF16, F16, F32, Workload

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(x):
    """SplitMix64 finaliser applied to state ``x`` (the generator's output for
    state ``x``); vectorised over uint64 arrays, wrapping arithmetic."""
    with np.errstate(over="ignore"):
        z = np.asarray(x, dtype=np.uint64) + _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def table_seed(cfg_id: int, t: int) -> int:
    return int(splitmix64(np.uint64((cfg_id << 32) | t)))


VALUE_KIND = {"uniform": 0, "cint": 1}


def f32_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 (finite inputs), returned as uint16 bits."""
    bits = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (bits + np.uint64(0x7FFF) + ((bits >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def counter_values(seed: int, dim: int, rows: np.ndarray, kind: int, dtype: int) -> np.ndarray:
    """Values of rows ``rows`` (any int array) of a counter-based table, shape
    (len(rows), dim), in storage dtype (float32 / float16 / uint16 bf16 bits)."""
    rows = np.asarray(rows, dtype=np.uint64).reshape(-1, 1)
    e = rows * np.uint64(dim) + np.arange(dim, dtype=np.uint64).reshape(1, -1)
    u = splitmix64(np.uint64(seed) ^ e) >> np.uint64(40)
    if kind == 0:
        x = (u.astype(np.int64) - (1 << 23)).astype(np.float32) * np.float32(2.0 ** -24)
        v = x * np.float32(0.1)
    else:
        v = ((u % np.uint64(17)).astype(np.int64) - 8).astype(np.float32)
    v = v.astype(np.float32)
    if dtype == F32:
        return v
    if dtype == F16:
        return v.astype(np.float16)
    return f32_to_bf16_bits(v)


@functools.lru_cache(maxsize=8)
def _zipf_cdf(n: int, alpha: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-alpha)
    c = np.cumsum(w)
    return c / c[-1]


@dataclasses.dataclass
class Inputs:
    w: Workload
    lengths: np.ndarray            # int64 [T*B], table-major
    offsets: np.ndarray            # int64 [T*B + 1]
    indices: np.ndarray            # int32 [nnz]
    weights: Optional[np.ndarray]  # float32 [nnz] or None
    host_tables: Optional[List[np.ndarray]] = None  # only for host-valued workloads

    @property
    def nnz(self) -> int:
        return int(self.offsets[-1])

    def table_rows(self, t: int, rows: np.ndarray) -> np.ndarray:
        """Stored values of ``rows`` of table t (storage dtype)."""
        if self.host_tables is not None:
            return self.host_tables[t][np.asarray(rows, dtype=np.int64)]
        return counter_values(table_seed(self.w.cfg_id, t), self.w.dims[t], rows,
                              VALUE_KIND[self.w.values], self.w.dtype)

    def table(self, t: int) -> np.ndarray:
        """Whole table t materialised on the host."""
        if self.host_tables is not None:
            return self.host_tables[t]
        from . import host
        return host.fill(self.w.rows[t], self.w.dims[t], self.w.dtype, table_seed(self.w.cfg_id, t),
                         VALUE_KIND[self.w.values])

    def unique_rows(self) -> int:
        """Number of distinct (table, row) pairs touched: the DRAM lower bound."""
        tot = 0
        B = self.w.B
        for t in range(self.w.T):
            lo, hi = self.offsets[t * B], self.offsets[(t + 1) * B]
            tot += np.unique(self.indices[lo:hi]).size
        return tot

    def unique_row_bytes(self) -> int:
        B = self.w.B
        tot = 0
        for t in range(self.w.T):
            lo, hi = self.offsets[t * B], self.offsets[(t + 1) * B]
            tot += np.unique(self.indices[lo:hi]).size * self.w.dims[t] * self.w.elt
        return tot


def _lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    n = w.T * w.B
    kind, *p = w.lengths.split(":")
    if kind == "fixed":
        return np.full(n, int(p[0]), dtype=np.int64)
    if kind == "uniform":
        return rng.integers(int(p[0]), int(p[1]) + 1, size=n, dtype=np.int64)
    if kind == "poisson":
        return np.clip(rng.poisson(float(p[0]), size=n), int(p[1]), int(p[2])).astype(np.int64)
    raise ValueError(w.lengths)


def make_inputs(w: Workload) -> Inputs:
    """Draw every input of workload ``w`` deterministically from its seed."""
    ss = np.random.SeedSequence([2305, 6942, w.cfg_id])
    s_len, s_idx, s_perm, s_wt, s_val = ss.spawn(5)
    lengths = _lengths(w, np.random.default_rng(s_len))
    offsets = np.zeros(lengths.size + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    nnz = int(offsets[-1])
    indices = np.empty(nnz, dtype=np.int32)
    r_idx = np.random.default_rng(s_idx)
    r_perm = np.random.default_rng(s_perm)
    kind, *p = w.indices.split(":")
    for t in range(w.T):
        lo, hi = offsets[t * w.B], offsets[(t + 1) * w.B]
        n, N = hi - lo, w.rows[t]
        if kind == "uniform":
            indices[lo:hi] = r_idx.integers(0, N, size=n, dtype=np.int64)
        elif kind == "zipf":
            cdf = _zipf_cdf(N, float(p[0]))
            rank0 = np.searchsorted(cdf, r_idx.random(n), side="right")
            np.minimum(rank0, N - 1, out=rank0)
            perm = r_perm.permutation(N)
            indices[lo:hi] = perm[rank0]
        else:
            raise ValueError(w.indices)
    weights = np.random.default_rng(s_wt).random(nnz, dtype=np.float32) if w.weighted else None
    tables = None
    if w.values in ("normal", "int8"):
        r_val = np.random.default_rng(s_val)
        tables = []
        for t in range(w.T):
            shape = (w.rows[t], w.dims[t])
            if w.values == "normal":
                v = r_val.standard_normal(shape, dtype=np.float32)
            else:
                v = r_val.integers(-8, 9, size=shape).astype(np.float32)
            if w.dtype == F16:
                v = v.astype(np.float16)
            elif w.dtype == BF16:
                v = f32_to_bf16_bits(v)
            tables.append(v)
    return Inputs(w, lengths, offsets, indices, weights, tables)
