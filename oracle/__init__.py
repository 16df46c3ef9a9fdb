"""CPU oracle for pooled embedding-bag + All-to-All send layout + ready flags.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke``
and by the benchmark's CPU-baseline leg, never by the product package.  It
shares no code with the GPU path; the only thing both sides use is the seeded
input generator in ``synth``.

GEMV + AllReduce (Sec. III-B): :func:`gemv_ar` computes the reduced vector
every rank holds after the AllReduce, sum over ranks of A_r x_r, in fp64.

Three implementations of the same pooling definition (pooled sums in fp64, placed at
send[r][s][off_t + j] with r = b / S, s = b mod S; one flag per
(destination, slice) equal to the epoch), each usable as a check of the others:

* ``oracle.c`` (via :func:`pool`): plain C, threaded over samples, whole batch;
* :mod:`oracle.sampled`: numpy, any subset of bags, rows fetched on demand
  (used at full workload sizes where tables do not fit in host memory);
* :mod:`oracle.brute`: pure-Python loops for tiny hand-checkable inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

ERRORS = {0: "ok", -1: "bad arguments", -2: "B % R or S % C not zero", -3: "bad offsets", -4: "index out of range"}


def build(src: str = SRC, out: str = LIB) -> str:
    """Compile the C oracle (gcc -O2, no fast-math: IEEE fp64 as written)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib = None


def load(path: str = LIB):
    global _lib
    if path == LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.oracle_pool.argtypes = [i32, P, P, P, i32, P, i64, P, P, i32, i64, i32, i32, P, P, P, i32]
    lib.oracle_pool.restype = ctypes.c_int
    lib.oracle_validate.argtypes = [i32, P, P, P, i64, P, i64, i32, i32]
    lib.oracle_validate.restype = ctypes.c_int
    lib.oracle_flags.argtypes = [i64, i32, i32, i32, ctypes.c_uint32, P, i64]
    lib.oracle_flags.restype = ctypes.c_int
    lib.oracle_backward.argtypes = [i32, P, P, P, i32, i64, i32, P, P]
    lib.oracle_backward.restype = ctypes.c_int
    lib.oracle_gemv_ar.argtypes = [i32, i64, P, i32, P, P, P, P, P, i32]
    lib.oracle_gemv_ar.restype = ctypes.c_int
    lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_double.restype = ctypes.c_double
    lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_double.restype = ctypes.c_double
    if path == LIB:
        _lib = lib
    return lib


class OracleError(ValueError):
    pass


def _ptr(a):
    return None if a is None else a.ctypes.data


def pool(tables, dtype, dims, indices, offsets, weights, B, R, C, nthreads=None, lib=None,
         want_sum=True, want_abs=True, want_send=True, mean=False):
    """Pool one forward.  ``tables`` is a list of host arrays in storage dtype
    (float32, float16, or uint16 bf16 bits), shape (rows_t, dims[t]).
    ``mean``: mean pooling (sum / L, zeros for empty bags; no weights).

    Returns (sum64, abs64, send) with shape (B, sum(D)) each; ``send`` is the
    fp32 send buffer, whose memory order is [R][B/R][sum(D)].
    """
    lib = lib or load()
    T = len(tables)
    tabs = [np.ascontiguousarray(x) for x in tables]
    ptrs = (ctypes.c_void_p * T)(*[x.ctypes.data for x in tabs])
    rows = np.array([x.shape[0] for x in tabs], dtype=np.int64)
    dims = np.ascontiguousarray(dims, dtype=np.int32)
    indices = np.ascontiguousarray(indices, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    weights = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    sd = int(dims.sum())
    sum64 = np.empty((B, sd), dtype=np.float64) if want_sum else None
    abs64 = np.empty((B, sd), dtype=np.float64) if want_abs else None
    send = np.empty((B, sd), dtype=np.float32) if want_send else None
    if nthreads is None:
        nthreads = len(os.sched_getaffinity(0))
    rc = lib.oracle_pool(T, ctypes.cast(ptrs, ctypes.c_void_p), rows.ctypes.data, dims.ctypes.data, dtype,
                         _ptr(indices) if indices.size else None, indices.size, offsets.ctypes.data,
                         _ptr(weights), int(bool(mean)), B, R, C, _ptr(sum64), _ptr(abs64), _ptr(send), nthreads)
    if rc != 0:
        raise OracleError(f"oracle_pool: {ERRORS.get(rc, rc)}")
    return sum64, abs64, send


def pool_inputs(inp, nthreads=None, **kw):
    """Pool a whole :class:`synth.Inputs` (tables materialised on the host)."""
    w = inp.w
    tables = [inp.table(t) for t in range(w.T)]
    return pool(tables, w.dtype, w.dims, inp.indices, inp.offsets, inp.weights, w.B, w.R, w.C,
                nthreads=nthreads, **kw)


def flags(B, R, C, epoch, lib=None, per_slice=1):
    """Expected flags after ``epoch`` forwards; per_slice = T for per-table
    slices (flag (g, t) at g * T + t)."""
    lib = lib or load()
    if B <= 0 or R <= 0 or C <= 0 or B % R or (B // R) % C:
        raise OracleError("B % R or S % C not zero")
    n = R * ((B // R) // C) * per_slice
    out = np.empty(n, dtype=np.uint32)
    rc = lib.oracle_flags(B, R, C, per_slice, epoch, out.ctypes.data, n)
    if rc != 0:
        raise OracleError(f"oracle_flags: {ERRORS.get(rc, rc)}")
    return out


def backward(dims, offsets, weights, grad, B, R, mean=False, lib=None):
    """Embedding backward: per-lookup gradient rows (lookup order, table
    blocks one after the other) from the pooled-output gradient ``grad``
    ([B][sum D] fp32, the destination-partitioned layout).  Returns a flat
    fp32 array of sum over t of nnz_t * D_t values."""
    lib = lib or load()
    dims = np.ascontiguousarray(dims, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    weights = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    T = dims.size
    n = int(sum((offsets[(t + 1) * B] - offsets[t * B]) * dims[t] for t in range(T)))
    values = np.empty(max(n, 1), dtype=np.float32)
    rc = lib.oracle_backward(T, dims.ctypes.data, offsets.ctypes.data, _ptr(weights), int(bool(mean)), B, R,
                             grad.ctypes.data, values.ctypes.data)
    if rc != 0:
        raise OracleError(f"oracle_backward: {ERRORS.get(rc, rc)}")
    return values[:n]


def gemv_ar(A, x, dtype, nthreads=None, lib=None):
    """GEMV + AllReduce (Sec. III-B): A and x are lists of R host arrays in
    storage dtype, A[r] of shape (M, K_r), x[r] of K_r elements.  Returns
    (y64, abs64, y) -- the sum over ranks of A_r x_r in fp64, the sum of
    |terms|, and the fp32 result every rank holds after the AllReduce."""
    lib = lib or load()
    R = len(A)
    if R == 0 or len(x) != R:
        raise OracleError("bad arguments")
    As = [np.ascontiguousarray(a) for a in A]
    xs = [np.ascontiguousarray(v) for v in x]
    M = As[0].shape[0]
    for a, v in zip(As, xs):
        if a.ndim != 2 or a.shape[0] != M or v.shape != (a.shape[1],):
            raise OracleError("bad arguments")
    Ks = np.array([a.shape[1] for a in As], dtype=np.int64)
    pa = (ctypes.c_void_p * R)(*[a.ctypes.data for a in As])
    px = (ctypes.c_void_p * R)(*[v.ctypes.data for v in xs])
    y64 = np.empty(M, dtype=np.float64)
    abs64 = np.empty(M, dtype=np.float64)
    y = np.empty(M, dtype=np.float32)
    if nthreads is None:
        nthreads = len(os.sched_getaffinity(0))
    rc = lib.oracle_gemv_ar(R, M, Ks.ctypes.data, dtype, ctypes.cast(pa, ctypes.c_void_p),
                            ctypes.cast(px, ctypes.c_void_p), y64.ctypes.data, abs64.ctypes.data, y.ctypes.data,
                            nthreads)
    if rc != 0:
        raise OracleError(f"oracle_gemv_ar: {ERRORS.get(rc, rc)}")
    return y64, abs64, y


def within_tolerance(gpu, sum64, abs64, rel=1e-5, absol=1e-6):
    """Acceptance for floating-point outputs: |gpu - sum64| <= rel * abs64 + absol."""
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - sum64)
    bound = rel * abs64 + absol
    ok = err <= bound
    return bool(ok.all()), err, bound
