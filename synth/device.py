"""Device copies of seeded inputs (torch tensors in HBM).

Counter-valued tables are filled in place by ``libebag_synth.so`` (same value
function as :func:`synth.gen.counter_values`); host-valued tables, indices,
offsets and weights are copied from the host arrays.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional

import numpy as np

from .configs import BF16, F16, F32
from .gen import VALUE_KIND, Inputs, table_seed

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libebag_synth.so")
_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} not built: run `python __graft_entry__.py`")
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        lib.synth_fill.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32, P]
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_copy.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, P]
        lib.synth_copy.restype = ctypes.c_int
        lib.synth_gather_probe.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, P, P]
        lib.synth_gather_probe.restype = ctypes.c_int
        lib.synth_stream_read.argtypes = [P, ctypes.c_int64, ctypes.c_int32, P, P]
        lib.synth_stream_read.restype = ctypes.c_int
        _lib = lib
    return _lib


def torch_dtype(dtype: int):
    import torch
    return {F32: torch.float32, F16: torch.float16, BF16: torch.bfloat16}[dtype]


@dataclasses.dataclass
class DeviceInputs:
    tables: List  # torch tensors (rows_t, D_t) in storage dtype
    indices: object
    offsets: object
    weights: Optional[object]


def fill_table(tensor, seed: int, kind: int, dtype: int, stream=None):
    import torch
    rows, dim = tensor.shape
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    rc = load().synth_fill(tensor.data_ptr(), rows, dim, dtype, seed, kind, s)
    if rc != 0:
        raise RuntimeError(f"synth_fill failed: {rc}")


def host_to_tensor(arr: np.ndarray, dtype: int, device):
    import torch
    if dtype == BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def tables_to_device(inp: Inputs, device) -> List:
    import torch
    w = inp.w
    out = []
    for t in range(w.T):
        if inp.host_tables is not None:
            out.append(host_to_tensor(inp.host_tables[t], w.dtype, device))
        else:
            x = torch.empty((w.rows[t], w.dims[t]), dtype=torch_dtype(w.dtype), device=device)
            fill_table(x, table_seed(w.cfg_id, t), VALUE_KIND[w.values], w.dtype)
            out.append(x)
    return out


def to_device(inp: Inputs, device="cuda") -> DeviceInputs:
    import torch
    tables = tables_to_device(inp, device)
    idx = torch.from_numpy(inp.indices).to(device)
    off = torch.from_numpy(inp.offsets).to(device)
    wts = None if inp.weights is None else torch.from_numpy(inp.weights).to(device)
    return DeviceInputs(tables, idx, off, wts)


def copy(dst, src, nbytes: int, grid: int = 0, stream=None):
    """16-byte vector copy kernel (HBM probe / byte-counter calibration)."""
    import torch
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    rc = load().synth_copy(dst.data_ptr(), src.data_ptr(), nbytes, grid, s)
    if rc != 0:
        raise RuntimeError(f"synth_copy failed: {rc}")


def gather_probe(buf, row_bytes: int, steps: int, grid: int, out, nt: bool = True, stream=None) -> int:
    """Random-row read probe over the bytes of ``buf`` (see synth/fill.hip);
    returns the bytes it reads."""
    import torch
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    nbytes = buf.numel() * buf.element_size()
    if out.numel() * out.element_size() < grid * 256 * 4:
        raise ValueError("probe output too small")
    rc = load().synth_gather_probe(buf.data_ptr(), nbytes, row_bytes, steps, grid, int(nt), out.data_ptr(), s)
    if rc != 0:
        raise RuntimeError(f"synth_gather_probe failed: {rc}")
    return grid * 4 * steps * 1024


def stream_read(buf, grid: int, out, stream=None) -> int:
    """Streaming read of every byte of ``buf`` (see synth/fill.hip); returns
    the bytes it reads."""
    import torch
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    nbytes = buf.numel() * buf.element_size()
    if out.numel() * out.element_size() < grid * 256 * 4:
        raise ValueError("probe output too small")
    rc = load().synth_stream_read(buf.data_ptr(), nbytes, grid, out.data_ptr(), s)
    if rc != 0:
        raise RuntimeError(f"synth_stream_read failed: {rc}")
    return nbytes
