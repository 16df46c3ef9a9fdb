"""Workload shapes for pooled embedding-bag + all-to-all send layout.

The paper (Sec. IV-A, "Embedding + All-to-All") evaluates embedding pooling with
embedding dimension 256, global batches of 256..2048 and up to 256 tables per
GPU, inputs drawn by the public DLRM data generator, with an average pooling
size of 70 in the large scale-out study (Table II).  Those inputs are not
available here; these five seeded synthetic workloads stand in for them.

Nothing in this module computes anything the method computes: it only
describes shapes and distributions.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

F32, F16, BF16 = 0, 1, 2
DTYPE_NAMES = {F32: "f32", F16: "f16", BF16: "bf16"}
DTYPE_BYTES = {F32: 4, F16: 2, BF16: 2}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int                 # selects the seed stream
    T: int                      # tables on this GPU
    rows: Tuple[int, ...]       # rows per table
    dims: Tuple[int, ...]       # embedding dimension per table
    dtype: int                  # F32 / F16 / BF16 storage
    B: int                      # global batch
    R: int                      # logical destinations
    C: int                      # samples per flag chunk
    lengths: str                # "fixed:L" | "uniform:lo:hi" | "poisson:mean:lo:hi"
    indices: str                # "uniform" | "zipf:alpha"
    weighted: bool              # per-index fp32 weights U[0,1)
    values: str                 # "normal" (host) | "uniform" (counter-based) | "int8" (host ints in [-8,8]) | "cint" (counter-based ints)

    @property
    def S(self) -> int:
        return self.B // self.R

    @property
    def sum_dim(self) -> int:
        return int(sum(self.dims))

    @property
    def col_off(self) -> Tuple[int, ...]:
        off, acc = [], 0
        for d in self.dims:
            off.append(acc)
            acc += d
        return tuple(off)

    @property
    def n_chunks(self) -> int:
        return self.B // self.C

    @property
    def elt(self) -> int:
        return DTYPE_BYTES[self.dtype]

    def table_bytes(self) -> int:
        return sum(r * d * self.elt for r, d in zip(self.rows, self.dims))

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _uniform_tables(T, rows, dims):
    return (rows,) * T, tuple(dims[t % len(dims)] for t in range(T))


def _mk(name, cfg_id, T, rows, dims, dtype, B, R, C, lengths, indices, weighted, values):
    r, d = _uniform_tables(T, rows, dims)
    return Workload(name, cfg_id, T, r, d, dtype, B, R, C, lengths, indices, weighted, values)


# The five workloads.  The benchmark's headline line is "large", the largest
# that fits one GPU (131 GB of tables); the other four are reported beside it.
TINY = _mk("tiny", 0, 4, 10_000, [64], F32, 256, 2, 32, "fixed:8", "uniform", False, "normal")
TINY_INT = TINY.with_(name="tiny_int", values="int8")
DLRM = _mk("dlrm", 1, 32, 1_000_000, [128], F32, 4096, 8, 64, "fixed:32", "uniform", False, "uniform")
SKEWED = _mk("skewed", 2, 64, 500_000, [256], F16, 8192, 8, 64, "uniform:1:64", "zipf:1.05", False, "uniform")
LARGE = _mk("large", 3, 128, 2_000_000, [128], F32, 16384, 64, 32, "poisson:40:1:128", "zipf:0.9", False, "uniform")
MIXED = _mk("mixed", 4, 48, 1_000_000, [32, 64, 128, 256], BF16, 8192, 16, 128, "uniform:1:100", "uniform", True, "uniform")

FULL = {w.name: w for w in (TINY, DLRM, SKEWED, LARGE, MIXED)}
ALL = dict(FULL, tiny_int=TINY_INT)


def scaled(w: Workload, rows: int, B: Optional[int] = None, T: Optional[int] = None,
           R: Optional[int] = None, C: Optional[int] = None, name: Optional[str] = None) -> Workload:
    """Same structure (dtype, D pattern, length and index laws), smaller sizes.

    Used for element-by-element parity at sizes a CPU finishes in seconds.
    """
    T = T or w.T
    dims_pattern = list(dict.fromkeys(w.dims)) if len(set(w.dims)) > 1 else [w.dims[0]]
    if len(set(w.dims)) > 1:
        # keep the cycling pattern of the original
        period = next(p for p in range(1, w.T + 1) if all(w.dims[i] == w.dims[i % p] for i in range(w.T)))
        dims_pattern = list(w.dims[:period])
    r, d = _uniform_tables(T, rows, dims_pattern)
    return dataclasses.replace(w, name=name or (w.name + "_small"), T=T, rows=r, dims=d,
                               B=B or w.B, R=R or w.R, C=C or w.C)
