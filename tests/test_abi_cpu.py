"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments before touching the GPU (no GPU needed)."""
import ctypes
import os
import re
import shutil

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("ebag_a2a.h", "gemv_ar.h")]


def _declared():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b((?:ebag_a2a|gemv_ar)_\w+)\s*\(", src))
    return sorted(names)


def test_every_header_is_checked():
    assert sorted(os.listdir(os.path.join(ROOT, "include"))) == sorted(os.path.basename(h) for h in HEADERS)


@pytest.fixture(scope="module")
def lib():
    import paper_2305_06942_amd as ebag
    return ebag.load()


def test_exports_every_declared_symbol(lib):
    import paper_2305_06942_amd as ebag
    names = _declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), f"{n} declared in the header but not exported"
    assert set(names) == set(ebag.symbols()), "binding and header disagree"


def test_default_opts(lib):
    import paper_2305_06942_amd as ebag
    o = ebag.default_opts()
    assert (o.waves_per_wg, o.rows_in_flight, o.debug_suppress_flag) == (4, 8, -1)
    assert (o.backward_bags_per_run, o.backward_waves_per_wg) == (4, 16)
    assert (o.consumer_wgs, o.deliver_wgs, o.deliver_waves_per_wg) == (512, 32, 8)


def _create(lib, T=2, rows=(10, 10), dims=(64, 64), dtype=0, C=32, max_batch=256, max_ranks=2, opts=None):
    import paper_2305_06942_amd.abi as abi
    h = ctypes.c_void_p()
    r = (ctypes.c_int64 * len(rows))(*rows)
    d = (ctypes.c_int32 * len(dims))(*dims)
    rc = lib.ebag_a2a_create(ctypes.byref(h), T, r, d, dtype, C, max_batch, max_ranks,
                             None if opts is None else ctypes.byref(opts))
    return rc, h


@pytest.mark.parametrize("kw,msg", [
    (dict(T=0), "num_tables"),
    (dict(dims=(64, 6)), "multiple of 16"),
    (dict(dtype=1, dims=(64, 4)), "multiple of 16"),
    (dict(dtype=7), "dtype"),
    (dict(C=0), "chunk_samples"),
    (dict(max_batch=0), "max_batch"),
    (dict(rows=(10, -1)), "rows"),
    (dict(dims=(1 << 20, 1 << 20), C=1024, max_batch=2048), "below 2 GiB"),
])
def test_create_rejects(lib, kw, msg):
    import paper_2305_06942_amd as ebag
    rc, h = _create(lib, **kw)
    assert rc == ebag.abi.EBAG_EINVAL
    assert msg in ebag.last_error()
    assert not h.value


@pytest.mark.parametrize("field,value,msg", [
    ("waves_per_wg", 0, "waves_per_wg"), ("waves_per_wg", 17, "waves_per_wg"),
    ("rows_in_flight", 5, "rows_in_flight"), ("bags_per_run", 0, "bags_per_run"),
    ("chunk_order", 2, "chunk_order"), ("consumer_wgs", 0, "consumer_wgs"),
    ("backward_bags_per_run", 0, "backward_bags_per_run"), ("backward_waves_per_wg", 17, "backward_waves_per_wg"),
    ("table_major", 3, "table_major"), ("table_major", -1, "table_major"), ("consume_nontemporal", 3, "consume_nontemporal"),
    ("deliver_wgs", 0, "deliver_wgs"), ("deliver_waves_per_wg", 0, "deliver_waves_per_wg"),
    ("deliver_waves_per_wg", 17, "deliver_waves_per_wg"),
])
def test_create_rejects_opts(lib, field, value, msg):
    import paper_2305_06942_amd as ebag
    o = ebag.default_opts()
    setattr(o, field, value)
    rc, _ = _create(lib, opts=o)
    assert rc == ebag.abi.EBAG_EINVAL and msg in ebag.last_error()


def test_null_plan_rejected(lib):
    import paper_2305_06942_amd as ebag
    assert lib.ebag_a2a_forward(None, None, None, None, None, 4, 2, None, None, None) == ebag.abi.EBAG_EINVAL
    assert lib.ebag_a2a_consume(None, None, None, None, 4, 2, 1, None) == ebag.abi.EBAG_EINVAL
    assert lib.ebag_a2a_reset(None) == ebag.abi.EBAG_EINVAL
    lib.ebag_a2a_destroy(None)


def test_package_has_no_fallback():
    """The product package never imports the oracle or a CPU path."""
    pkg = os.path.join(ROOT, "paper_2305_06942_amd")
    for dp, _, fs in os.walk(pkg):
        for f in fs:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                src = open(os.path.join(dp, f)).read()
                assert "oracle" not in src.replace("Oracle", ""), f


@pytest.mark.parametrize("kw,msg", [
    (dict(R=0), "R="), (dict(R=17), "R="), (dict(M=0), "M="), (dict(K=(8, 0)), "K[1]"),
    (dict(K=(8, 6)), "multiple of 16"), (dict(dtype=5), "dtype"), (dict(K=(8, 1 << 20)), "LDS"),
])
def test_gemv_create_rejects(lib, kw, msg):
    import paper_2305_06942_amd as ebag
    args = dict(R=2, M=100, K=(8, 8), dtype=0)
    args.update(kw)
    K = args["K"] if len(args["K"]) >= max(args["R"], 1) else tuple(args["K"]) * args["R"]
    h = ctypes.c_void_p()
    ks = (ctypes.c_int64 * len(K))(*K)
    rc = lib.gemv_ar_create(ctypes.byref(h), args["R"], args["M"], ks, args["dtype"], None)
    assert rc in (ebag.abi.EBAG_EINVAL, ebag.abi.EBAG_EUNSUPPORTED) and msg in ebag.last_error(), ebag.last_error()
    assert not h.value


def test_gemv_null_plan_rejected(lib):
    import paper_2305_06942_amd as ebag
    assert lib.gemv_ar_forward(None, None, None, None, None, None) == ebag.abi.EBAG_EINVAL
    assert lib.gemv_ar_unfused_forward(None, None, None, None, None, None) == ebag.abi.EBAG_EINVAL
    assert lib.gemv_ar_reset(None) == ebag.abi.EBAG_EINVAL
    o = ebag.gemv_default_opts()
    assert (o.tile_rows, o.waves_per_wg, o.comm_aware, o.debug_suppress_flag, o.reduce_mode) == (0, 2, 1, -1, 0)
    lib.gemv_ar_destroy(None)


class _NoCalls:
    """Stands in for the loaded library: any entry point called fails the test."""

    def __getattr__(self, name):
        def call(*a):
            raise AssertionError(f"{name} reached the C ABI with an undersized buffer")
        return call


def _sizing_plan(T=2, dims=(64, 32), C=8):
    import paper_2305_06942_amd as ebag
    p = object.__new__(ebag.Plan)
    p.T, p.dims, p.C, p.elt = T, list(dims), C, 4
    p.opts = ebag.default_opts()
    p._h, p._lib, p._tab_cache, p._empty_idx = None, _NoCalls(), None, None
    return p


@pytest.mark.parametrize("short", ["send", "flags", "offsets"])
def test_binding_rejects_undersized_buffers(lib, short):
    """The binding checks tensor sizes before any call: send [B][sum D] fp32,
    flags one uint32 per slice, offsets T*B+1 int64."""
    import torch
    p = _sizing_plan()
    B, R = 32, 2
    send = torch.zeros(B * sum(p.dims) - (4 if short == "send" else 0))
    flags = torch.zeros(B // p.C - (1 if short == "flags" else 0), dtype=torch.int32)
    offsets = torch.zeros(p.T * B + 1 - (1 if short == "offsets" else 0), dtype=torch.int64)
    tables = [torch.zeros(16, d) for d in p.dims]
    idx = torch.zeros(4, dtype=torch.int32)
    for call in (p.forward, p.unfused_forward):
        with pytest.raises(ValueError, match=short):
            call(tables, idx, offsets, None, B, R, send, flags, stream=0)
    if short != "send":
        with pytest.raises(ValueError, match=short):
            p.backward(send, offsets, None, B, R, torch.zeros(8), grad_flags=flags, stream=0)


def _typed_args(p, B=32, bad=None):
    """Forward arguments of the right sizes as CPU tensors, one of them made
    wrong in layout or element type by `bad`."""
    import torch
    send = torch.zeros(B, sum(p.dims))
    flags = torch.zeros(B // p.C, dtype=torch.int32)
    offsets = torch.zeros(p.T * B + 1, dtype=torch.int64)
    tables = [torch.zeros(16, d) for d in p.dims]
    idx = torch.zeros(4, dtype=torch.int32)
    wts = None
    if bad == "send_strided":
        send = torch.zeros(sum(p.dims), B).t()
    elif bad == "send_f64":
        send = send.double()
    elif bad == "indices_i64":
        idx = idx.long()
    elif bad == "offsets_i32":
        offsets = torch.zeros(2 * (p.T * B + 1), dtype=torch.int32)
    elif bad == "weights_f16":
        wts = torch.zeros(4, dtype=torch.float16)
    elif bad == "flags_f32":
        flags = torch.zeros(B // p.C)
    elif bad == "table_f16":
        tables[1] = torch.zeros(16, 2 * p.dims[1], dtype=torch.float16)
    return tables, idx, offsets, wts, send, flags


@pytest.mark.parametrize("bad,msg", [
    ("send_strided", "send buffer must be contiguous"), ("send_f64", "send buffer must be float32"),
    ("indices_i64", "indices must be int32"), ("offsets_i32", "offsets must be int64"),
    ("weights_f16", "weights must be float32"), ("flags_f32", "flags must be int32 or uint32"),
    ("table_f16", "table 1 must have 4-byte elements"), (None, "table 0 must be a GPU tensor")])
def test_binding_rejects_wrong_layout_type_or_device(lib, bad, msg):
    """Tensors reach a kernel only when contiguous, of the element type the
    C ABI reads, and on the GPU: each wrong case is refused on the host
    before any call (these CPU tensors of the right sizes fail on layout or
    type first, and on the device last)."""
    p = _sizing_plan()
    tables, idx, offsets, wts, send, flags = _typed_args(p, bad=bad)
    for call in (p.forward, p.unfused_forward):
        with pytest.raises(ValueError, match=msg):
            call(tables, idx, offsets, wts, 32, 2, send, flags, stream=0)


def test_binding_rejects_wrong_backward_and_consumer_buffers(lib):
    import torch
    p = _sizing_plan()
    B = 32
    grad = torch.zeros(B, sum(p.dims))
    offsets = torch.zeros(p.T * B + 1, dtype=torch.int64)
    with pytest.raises(ValueError, match="values must be float32"):
        p.backward(grad, offsets, None, B, 2, torch.zeros(8, dtype=torch.float64), stream=0)
    with pytest.raises(ValueError, match="gradient must be contiguous"):
        p.backward(torch.zeros(sum(p.dims), B).t(), offsets, None, B, 2, torch.zeros(8), stream=0)
    flags = torch.zeros(B // p.C, dtype=torch.int32)
    with pytest.raises(ValueError, match="recv buffer must be contiguous"):
        p.consume(grad, flags, torch.zeros(sum(p.dims), B).t(), B, 2, 1, stream=0)
    with pytest.raises(ValueError, match="destination buffer must be float32"):
        p.deliver(grad, torch.zeros(B, sum(p.dims), dtype=torch.float64), flags, B, 2, stream=0)


def _noalloc(lib, T=2, rows=(10, 10), dims=(64, 64), dtype=0, C=32, B=256, R=2, opts=None, null_send=False):
    r = (ctypes.c_int64 * max(T, 1))(*(list(rows) + [10] * max(T - len(rows), 0))[:max(T, 1)])
    d = (ctypes.c_int32 * max(T, 1))(*(list(dims) + [64] * max(T - len(dims), 0))[:max(T, 1)])
    fake = 1 << 20  # a 16-byte aligned address that is never dereferenced: every case fails on the host
    tabs = (ctypes.c_void_p * max(T, 1))(*([fake] * max(T, 1)))
    return lib.ebag_a2a_forward_noalloc(T, r, d, dtype, C, None if opts is None else ctypes.byref(opts), tabs,
                                        fake, fake, None, B, R, None if null_send else fake, fake, None)


@pytest.mark.parametrize("kw,code,msg", [
    (dict(T=0), "EBAG_EINVAL", "num_tables"),
    (dict(T=1025), "EBAG_EINVAL", "num_tables"),
    (dict(dims=(64, 6)), "EBAG_EINVAL", "multiple of 16"),
    (dict(dtype=9), "EBAG_EINVAL", "dtype"),
    (dict(B=255), "EBAG_EINVAL", "multiple of R"),
    (dict(B=2 * 65537 * 32, R=2), "EBAG_EINVAL", "slice counters"),
    (dict(null_send=True), "EBAG_EINVAL", "null"),
    (dict(opts="trace"), "EBAG_EUNSUPPORTED", "plan"),
    (dict(opts="check_indices"), "EBAG_EUNSUPPORTED", "plan"),
    (dict(opts="waves"), "EBAG_EINVAL", "waves_per_wg"),
])
def test_noalloc_rejects_before_touching_the_device(lib, kw, code, msg):
    """Sizes beyond the static array and bad arguments fail with a clear
    error before anything is enqueued (no GPU here)."""
    import paper_2305_06942_amd as ebag
    if isinstance(kw.get("opts"), str):
        o = ebag.default_opts()
        if kw["opts"] == "waves":
            o.waves_per_wg = 0
        else:
            setattr(o, kw["opts"], 1)
        kw = dict(kw, opts=o)
    rc = _noalloc(lib, **kw)
    assert rc == getattr(ebag.abi, code), (rc, ebag.last_error())
    assert msg in ebag.last_error(), ebag.last_error()


@pytest.mark.skipif(shutil.which("gcc") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs gcc and the HIP headers")
def test_headers_are_c_and_the_readme_example_compiles(tmp_path):
    """Both headers are plain C11 (no C++ constructs), and the README's call
    sequence compiles against them with the declared signatures."""
    import re
    import subprocess
    readme = open(os.path.join(ROOT, "README.md")).read()
    code = re.search(r"```c\n(.*?)```", readme, re.S).group(1)
    prog = ('#include "ebag_a2a.h"\n#include "gemv_ar.h"\n#include <hip/hip_runtime_api.h>\nint main(void) {\n'
            "  int32_t T = 2; int64_t rows[2] = {10, 10}; int32_t dims[2] = {64, 64};\n"
            "  int32_t C = 8; int64_t B = 64; int32_t R = 2;\n"
            "  const void* tables[2] = {0, 0}; const int32_t* indices = 0; const int64_t* offsets = 0;\n"
            "  float* send = 0; float* recv = 0; uint32_t* flags = 0;\n" + code + "  return 0;\n}\n")
    src = tmp_path / "readme_example.c"
    src.write_text(prog)
    r = subprocess.run(["gcc", "-std=c11", "-fsyntax-only", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
