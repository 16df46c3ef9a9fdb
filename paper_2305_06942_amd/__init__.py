"""Fused embedding-bag pooling + All-to-All send layout, and fused GEMV +
AllReduce, for MI355X (gfx950).

Python binding of the C ABI in ``include/ebag_a2a.h`` (argument marshalling
only: every step of the operation runs in the HIP library
``libebag_a2a.so`` built next to this file).  There is no fallback: if the
library is missing, :func:`load` raises.
"""
from .abi import (EBAG_BF16, EBAG_F16, EBAG_F32, EbagError, GemvAR, Plan, default_opts,  # noqa: F401
                  forward_noalloc, gemv_default_opts, last_error, load, queue_stream, queue_stream_destroy, symbols)
