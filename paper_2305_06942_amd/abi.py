"""ctypes binding of include/ebag_a2a.h and include/gemv_ar.h (same names,
argument marshalling only).

Device buffers may be passed as torch tensors (their ``data_ptr()`` is used)
or as integer device addresses.  The stream defaults to torch's current
stream on the current device.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libebag_a2a.so")

EBAG_F32, EBAG_F16, EBAG_BF16 = 0, 1, 2
EBAG_OK, EBAG_EINVAL, EBAG_EUNSUPPORTED, EBAG_EHIP, EBAG_ETIMEOUT, EBAG_ENOMEM, EBAG_EBUSY = 0, -1, -2, -3, -4, -5, -6


class Opts(ctypes.Structure):
    _fields_ = [
        ("waves_per_wg", ctypes.c_int32),
        ("bags_per_run", ctypes.c_int32),
        ("rows_in_flight", ctypes.c_int32),
        ("persistent_wgs_per_cu", ctypes.c_int32),
        ("release_mode", ctypes.c_int32),
        ("chunk_order", ctypes.c_int32),
        ("self_rank", ctypes.c_int32),
        ("trace", ctypes.c_int32),
        ("check_indices", ctypes.c_int32),
        ("debug_suppress_flag", ctypes.c_int32),
        ("consumer_wgs", ctypes.c_int32),
        ("stream_rows", ctypes.c_int32),
        ("consume_timeout_us", ctypes.c_int64),
        ("pooling_mode", ctypes.c_int32),
        ("slice_granule", ctypes.c_int32),
        ("backward_bags_per_run", ctypes.c_int32),
        ("backward_waves_per_wg", ctypes.c_int32),
        ("table_major", ctypes.c_int32),
        ("consume_nontemporal", ctypes.c_int32),
        ("deliver_wgs", ctypes.c_int32),
        ("deliver_waves_per_wg", ctypes.c_int32),
    ]


class GemvOpts(ctypes.Structure):
    _fields_ = [
        ("tile_rows", ctypes.c_int32),
        ("wgs_per_rank", ctypes.c_int32),
        ("waves_per_wg", ctypes.c_int32),
        ("comm_aware", ctypes.c_int32),
        ("debug_suppress_flag", ctypes.c_int32),
        ("reduce_mode", ctypes.c_int32),
        ("timeout_us", ctypes.c_int64),
    ]


class EbagError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"ebag_a2a error {code}: {msg}")
        self.code = code


_lib = None

_P = ctypes.c_void_p
_SIGS = {
    "ebag_a2a_default_opts": ([_P], ctypes.c_int),
    "ebag_a2a_create": ([_P, ctypes.c_int32, _P, _P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, _P],
                        ctypes.c_int),
    "ebag_a2a_forward": ([_P, _P, _P, _P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "ebag_a2a_unfused_forward": ([_P, _P, _P, _P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "ebag_a2a_forward_noalloc": ([ctypes.c_int32, _P, _P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P, _P,
                                  ctypes.c_int64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "ebag_a2a_consume": ([_P, _P, _P, _P, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, _P], ctypes.c_int),
    "ebag_a2a_backward": ([_P, _P, _P, ctypes.c_uint32, _P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P], ctypes.c_int),
    "ebag_a2a_deliver": ([_P, _P, _P, _P, ctypes.c_int64, ctypes.c_int32, _P], ctypes.c_int),
    "ebag_a2a_status": ([_P, _P, _P], ctypes.c_int),
    "ebag_a2a_status_ex": ([_P, _P], ctypes.c_int),
    "ebag_a2a_reset": ([_P], ctypes.c_int),
    "ebag_a2a_trace": ([_P, _P, _P, ctypes.c_int64, _P], ctypes.c_int),
    "ebag_a2a_occupancy": ([_P, ctypes.c_int32, _P], ctypes.c_int),
    "ebag_a2a_queue_stream_create": ([_P], ctypes.c_int),
    "ebag_a2a_queue_stream_destroy": ([_P], ctypes.c_int),
    "ebag_a2a_destroy": ([_P], None),
    "ebag_a2a_last_error": ([], ctypes.c_char_p),
    "gemv_ar_default_opts": ([_P], ctypes.c_int),
    "gemv_ar_create": ([_P, ctypes.c_int32, ctypes.c_int64, _P, ctypes.c_int32, _P], ctypes.c_int),
    "gemv_ar_forward": ([_P, _P, _P, _P, _P, _P], ctypes.c_int),
    "gemv_ar_unfused_forward": ([_P, _P, _P, _P, _P, _P], ctypes.c_int),
    "gemv_ar_status": ([_P, _P], ctypes.c_int),
    "gemv_ar_reset": ([_P], ctypes.c_int),
    "gemv_ar_launch_info": ([_P, _P], ctypes.c_int),
    "gemv_ar_destroy": ([_P], None),
}


def symbols():
    """Names of the C ABI entry points this binding expects."""
    return list(_SIGS)


def load(path: str = LIB_PATH):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library {path} not found: build it with `python __graft_entry__.py` "
                           "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    for name, (args, res) in _SIGS.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def last_error() -> str:
    return load().ebag_a2a_last_error().decode()


def _check(rc: int):
    if rc != EBAG_OK:
        raise EbagError(rc, last_error())


def _addr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _need(buf, nbytes: int, what: str):
    """A torch tensor passed as a buffer must hold at least nbytes (raw
    integer addresses are the caller's responsibility)."""
    if buf is not None and hasattr(buf, "numel") and buf.numel() * buf.element_size() < nbytes:
        raise ValueError(f"{what} holds {buf.numel() * buf.element_size()} bytes, needs {nbytes}")


F32 = ("float32",)
I32 = ("int32",)
I64 = ("int64",)
FLAG_TYPES = ("int32", "uint32")


def _is_tensor(x) -> bool:
    return x is not None and not isinstance(x, int) and hasattr(x, "is_contiguous")


def _validate(*specs):
    """Every torch tensor handed to a kernel must be contiguous, of the
    element type the C ABI reads and on the GPU.  specs: (tensor, name,
    allowed dtype names or None, element bytes or None); None and raw integer
    addresses are skipped (those are the caller's responsibility).  Layout and
    type are checked for every tensor before the device of any."""
    ts = [sp for sp in specs if _is_tensor(sp[0])]
    for x, what, kinds, elt in ts:
        if not x.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        name = str(x.dtype).replace("torch.", "")
        if kinds is not None and name not in kinds:
            raise ValueError(f"{what} must be {' or '.join(kinds)}, not {name}")
        if elt is not None and x.element_size() != elt:
            raise ValueError(f"{what} must have {elt}-byte elements, not {x.element_size()}-byte {name}")
    for x, what, _, _ in ts:
        if x.device.type != "cuda":
            raise ValueError(f"{what} must be a GPU tensor, not one on {x.device}")


def _elt(dtype) -> int:
    return 4 if int(dtype) == EBAG_F32 else 2


def queue_stream():
    """A torch stream on a hardware queue of its own (ebag_a2a_queue_stream_create)."""
    import torch
    s = ctypes.c_void_p()
    _check(load().ebag_a2a_queue_stream_create(ctypes.byref(s)))
    return torch.cuda.ExternalStream(s.value)


def queue_stream_destroy(stream):
    """Drain and destroy a stream from queue_stream() (ebag_a2a_queue_stream_destroy)."""
    _check(load().ebag_a2a_queue_stream_destroy(_stream(stream)))


def default_opts() -> Opts:
    o = Opts()
    _check(load().ebag_a2a_default_opts(ctypes.byref(o)))
    return o


NOALLOC_MAX_TABLES, NOALLOC_MAX_FLAGS = 1024, 65536


def forward_noalloc(rows, dims, dtype, chunk_samples, tables, indices, offsets, weights, B, R, send, flags,
                    stream=None, **opts):
    """Plan-free fused forward (``ebag_a2a_forward_noalloc``): the same result
    as ``Plan(rows, dims, dtype, chunk_samples, ..., **opts).forward(...)``,
    with the plan's device memory in the library's static per-GPU array."""
    lib = load()
    o = default_opts()
    for k, v in opts.items():
        if not hasattr(o, k):
            raise TypeError(f"unknown option {k}")
        setattr(o, k, int(v))
    T = len(rows)
    if len(dims) != T or len(tables) != T:
        raise ValueError("rows, dims and tables must have one entry per table")
    n_flags = (int(B) // int(chunk_samples)) * (T if o.slice_granule == 1 else 1)
    _need(send, 4 * int(B) * sum(int(d) for d in dims), "send buffer")
    _need(flags, 4 * n_flags, "flags")
    _need(offsets, 8 * (T * int(B) + 1), "offsets")
    _validate(*[(t, f"table {i}", None, _elt(dtype)) for i, t in enumerate(tables)],
              (indices, "indices", I32, None), (offsets, "offsets", I64, None), (weights, "weights", F32, None),
              (send, "send buffer", F32, None), (flags, "flags", FLAG_TYPES, None))
    if hasattr(indices, "numel") and indices.numel() == 0:
        raise ValueError("indices must have a device address: pass a one-element buffer when every bag is empty")
    rows_a = (ctypes.c_int64 * T)(*[int(r) for r in rows])
    dims_a = (ctypes.c_int32 * T)(*[int(d) for d in dims])
    tabs = (ctypes.c_void_p * T)(*[_addr(t) for t in tables])
    _check(lib.ebag_a2a_forward_noalloc(T, rows_a, dims_a, int(dtype), int(chunk_samples), ctypes.byref(o), tabs,
                                        _addr(indices), _addr(offsets), _addr(weights), int(B), int(R), _addr(send),
                                        _addr(flags), _stream(stream)))


class Plan:
    """A plan for T tables (``ebag_a2a_create``); methods mirror the C ABI."""

    def __init__(self, rows: Sequence[int], dims: Sequence[int], dtype: int, chunk_samples: int, max_batch: int,
                 max_ranks: int, **opts):
        lib = load()
        o = default_opts()
        for k, v in opts.items():
            if not hasattr(o, k):
                raise TypeError(f"unknown option {k}")
            setattr(o, k, int(v))
        self.T = len(rows)
        self.dims = [int(d) for d in dims]
        self.C = int(chunk_samples)
        self.elt = _elt(dtype)
        self.opts = o
        rows_a = (ctypes.c_int64 * self.T)(*[int(r) for r in rows])
        dims_a = (ctypes.c_int32 * self.T)(*self.dims)
        h = ctypes.c_void_p()
        _check(lib.ebag_a2a_create(ctypes.byref(h), self.T, rows_a, dims_a, int(dtype), self.C, int(max_batch),
                                   int(max_ranks), ctypes.byref(o)))
        self._h = h
        self._lib = lib
        self._tab_cache = None
        self._empty_idx = None

    def _indices(self, indices):
        """An empty index tensor (every bag empty) has no device address; the
        C ABI takes a valid pointer that is never read, so pass a one-element
        device buffer instead."""
        if hasattr(indices, "numel") and indices.numel() == 0:
            if self._empty_idx is None or self._empty_idx.device != indices.device:
                import torch
                self._empty_idx = torch.zeros(1, dtype=torch.int32, device=indices.device)
            return self._empty_idx.data_ptr()
        return _addr(indices)

    def _tables(self, tables):
        ptrs = [_addr(t) for t in tables]
        if len(ptrs) != self.T:
            raise ValueError(f"expected {self.T} tables, got {len(ptrs)}")
        if self._tab_cache is None or self._tab_cache[0] != ptrs:
            self._tab_cache = (ptrs, (ctypes.c_void_p * self.T)(*ptrs))
        return self._tab_cache[1]

    def _fwd_sizes(self, B, send, flags):
        _need(send, 4 * int(B) * sum(self.dims), "send buffer")
        _need(flags, 4 * self.n_flags(int(B)), "flags")

    def _offsets(self, B, offsets):
        _need(offsets, 8 * (self.T * int(B) + 1), "offsets")
        return _addr(offsets)

    def _fwd_types(self, tables, indices, offsets, weights, send, flags):
        _validate(*[(t, f"table {i}", None, self.elt) for i, t in enumerate(tables)],
                  (indices, "indices", I32, None), (offsets, "offsets", I64, None), (weights, "weights", F32, None),
                  (send, "send buffer", F32, None), (flags, "flags", FLAG_TYPES, None))

    def forward(self, tables, indices, offsets, weights, B, R, send, flags, stream=None):
        self._fwd_sizes(B, send, flags)
        _need(offsets, 8 * (self.T * int(B) + 1), "offsets")
        self._fwd_types(tables, indices, offsets, weights, send, flags)
        _check(self._lib.ebag_a2a_forward(self._h, self._tables(tables), self._indices(indices),
                                          self._offsets(B, offsets), _addr(weights), int(B), int(R), _addr(send),
                                          _addr(flags), _stream(stream)))

    def unfused_forward(self, tables, indices, offsets, weights, B, R, send, flags, stream=None):
        self._fwd_sizes(B, send, flags)
        _need(offsets, 8 * (self.T * int(B) + 1), "offsets")
        self._fwd_types(tables, indices, offsets, weights, send, flags)
        _check(self._lib.ebag_a2a_unfused_forward(self._h, self._tables(tables), self._indices(indices),
                                                  self._offsets(B, offsets), _addr(weights), int(B), int(R),
                                                  _addr(send), _addr(flags), _stream(stream)))

    def consume(self, send, flags, recv, B, R, expected_epoch, stream=None):
        self._fwd_sizes(B, send, flags)
        _need(recv, 4 * int(B) * sum(self.dims), "recv buffer")
        _validate((send, "send buffer", F32, None), (flags, "flags", FLAG_TYPES, None), (recv, "recv buffer", F32, None))
        _check(self._lib.ebag_a2a_consume(self._h, _addr(send), _addr(flags), _addr(recv), int(B), int(R),
                                          int(expected_epoch) & 0xFFFFFFFF, _stream(stream)))

    def backward(self, grad, offsets, weights, B, R, values, grad_flags=None, expected_epoch=0, stream=None):
        self._fwd_sizes(B, grad, grad_flags)
        _need(offsets, 8 * (self.T * int(B) + 1), "offsets")
        _validate((grad, "gradient", F32, None), (grad_flags, "gradient flags", FLAG_TYPES, None),
                  (offsets, "offsets", I64, None), (weights, "weights", F32, None), (values, "values", F32, None))
        _check(self._lib.ebag_a2a_backward(self._h, _addr(grad), _addr(grad_flags), int(expected_epoch) & 0xFFFFFFFF,
                                           self._offsets(B, offsets), _addr(weights), int(B), int(R), _addr(values),
                                           _stream(stream)))

    def deliver(self, src, dst, flags, B, R, stream=None):
        self._fwd_sizes(B, src, flags)
        _need(dst, 4 * int(B) * sum(self.dims), "destination buffer")
        _validate((src, "source buffer", F32, None), (dst, "destination buffer", F32, None),
                  (flags, "flags", FLAG_TYPES, None))
        _check(self._lib.ebag_a2a_deliver(self._h, _addr(src), _addr(dst), _addr(flags), int(B), int(R),
                                          _stream(stream)))

    def status(self):
        """(timed_out, first_missing_flag); synchronises the device."""
        s = (ctypes.c_int32 * 4)()
        _check(self._lib.ebag_a2a_status_ex(self._h, s))
        return s[0], s[1]

    def status_ex(self):
        s = (ctypes.c_int32 * 4)()
        _check(self._lib.ebag_a2a_status_ex(self._h, s))
        return tuple(s)

    def reset(self):
        _check(self._lib.ebag_a2a_reset(self._h))

    def n_flags(self, B):
        """Flag count of a forward over B samples (B / C, times T per-table)."""
        return (B // self.C) * (self.T if self.opts.slice_granule == 1 else 1)

    def trace(self, n):
        import numpy as np
        rel = np.zeros(n, dtype=np.uint64)
        drn = np.zeros(n, dtype=np.uint64)
        tpu = ctypes.c_double()
        _check(self._lib.ebag_a2a_trace(self._h, rel.ctypes.data, drn.ctypes.data, n, ctypes.byref(tpu)))
        return rel, drn, tpu.value

    def occupancy(self, weighted=False):
        """(max resident WGs per CU, CUs, threads per WG, bags per run) of the fused kernel."""
        s = (ctypes.c_int32 * 4)()
        _check(self._lib.ebag_a2a_occupancy(self._h, int(bool(weighted)), s))
        return tuple(s)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.ebag_a2a_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gemv_default_opts() -> GemvOpts:
    o = GemvOpts()
    _check(load().gemv_ar_default_opts(ctypes.byref(o)))
    return o


class GemvAR:
    """A fused GEMV + AllReduce plan (``gemv_ar_create``) for R ranks; methods
    mirror the C ABI.  A, x, y are sequences of R device buffers."""

    def __init__(self, R: int, M: int, K: Sequence[int], dtype: int, **opts):
        lib = load()
        o = gemv_default_opts()
        for k, v in opts.items():
            if not hasattr(o, k):
                raise TypeError(f"unknown option {k}")
            setattr(o, k, int(v))
        self.R, self.M, self.K = int(R), int(M), [int(k) for k in K]
        self.elt = _elt(dtype)
        self.opts = o
        ks = (ctypes.c_int64 * len(self.K))(*self.K)
        h = ctypes.c_void_p()
        _check(lib.gemv_ar_create(ctypes.byref(h), self.R, self.M, ks, int(dtype), ctypes.byref(o)))
        self._h = h
        self._lib = lib

    def _arrays(self, A, x, y):
        if not (len(A) == len(x) == len(y) == self.R):
            raise ValueError(f"expected {self.R} buffers each for A, x and y")
        for r in range(self.R):
            _need(A[r], self.M * self.K[r] * self.elt, f"A[{r}]")
            _need(x[r], self.K[r] * self.elt, f"x[{r}]")
        _validate(*[(A[r], f"A[{r}]", None, self.elt) for r in range(self.R)],
                  *[(x[r], f"x[{r}]", None, self.elt) for r in range(self.R)],
                  *[(y[r], f"y[{r}]", F32, None) for r in range(self.R)])
        arr = ctypes.c_void_p * self.R
        return arr(*[_addr(a) for a in A]), arr(*[_addr(v) for v in x]), arr(*[_addr(v) for v in y])

    def _out_sizes(self, y, out_flags):
        for v in y:
            _need(v, 4 * self.M, "output vector")
        _need(out_flags, 4 * self.R * self.launch_info()[0], "out_flags")
        _validate((out_flags, "out_flags", FLAG_TYPES, None))

    def forward(self, A, x, y, out_flags=None, stream=None):
        self._out_sizes(y, out_flags)
        a, xv, yv = self._arrays(A, x, y)
        _check(self._lib.gemv_ar_forward(self._h, a, xv, yv, _addr(out_flags), _stream(stream)))

    def unfused_forward(self, A, x, y, out_flags=None, stream=None):
        self._out_sizes(y, out_flags)
        a, xv, yv = self._arrays(A, x, y)
        _check(self._lib.gemv_ar_unfused_forward(self._h, a, xv, yv, _addr(out_flags), _stream(stream)))

    def status(self):
        """(timed_out, first missing peer flag); synchronises the device."""
        s = (ctypes.c_int32 * 2)()
        rc = self._lib.gemv_ar_status(self._h, s)
        if rc not in (EBAG_OK, EBAG_ETIMEOUT):
            _check(rc)
        return s[0], s[1]

    def reset(self):
        _check(self._lib.gemv_ar_reset(self._h))

    def launch_info(self):
        """(workgroups per rank P, threads per workgroup, tiles, resident workgroups, rows per tile)."""
        s = (ctypes.c_int32 * 5)()
        _check(self._lib.gemv_ar_launch_info(self._h, s))
        return tuple(s)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.gemv_ar_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
