"""Benchmark of the fused embedding-bag pooling + All-to-All send layout.

One step = one fused forward over one batch of the workload: pool every bag
(gather L rows, sum or weighted-sum in fp32), store each pooled vector at its
destination slot of the [R][B/R][sum D] send buffer and release the
per-(destination, slice) ready flags.  Inputs are resident in HBM before the
timed region.  Prints one JSON line (the headline workload, or one per
workload with --all).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--all] [--no-cpu-baseline] [--profile]
       (no --workload: the large workload's line, with the other four
       workloads' fused / unfused / consumer times and rooflines in it)
       python bench.py --summarize DIR     (rocprofv3 csv output -> text summary)
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, public specification
# Sources whose text fixes each profiled kernel: committed counter records
# are used only while the hash of these files is unchanged.
KERNEL_SOURCES = {
    "fused_pool_kernel": ["paper_2305_06942_amd/csrc/pool.hip", "paper_2305_06942_amd/csrc/common.h"],
    "backward_kernel": ["paper_2305_06942_amd/csrc/backward.hip", "paper_2305_06942_amd/csrc/backward.h",
                        "paper_2305_06942_amd/csrc/common.h"],
    "gemv_ar_last_arriver_kernel": ["paper_2305_06942_amd/csrc/gemv_ar.hip"],
}
# GEMV + AllReduce records are keyed by the output size: workload "m<M>".
TRAFFIC_FILE = {"fused_pool_kernel": "traffic_{}.json", "backward_kernel": "traffic_backward_{}.json",
                "gemv_ar_last_arriver_kernel": "traffic_gemv_{}.json"}
# Launch options per workload (every other option at its default):
#  * where rows are reused -- Zipf indices (skewed, large), or tables small
#    enough for the Infinity Cache (mixed's 64-256 MB tables) -- rows are
#    read through the caches (stream_rows = 0) and pooled table by table with
#    the paper's per-table slices (slice_granule = 1), so a table's rows stay
#    cached while it is pooled: skewed with one table per XCD at a time
#    (table_major = 1, its hot rows fit an XCD's L2), large and mixed with
#    one table at a time for the whole device (table_major = 2, the table's
#    working set shares the device-wide cache);
#  * launch shapes from a sweep in each workload's order: skewed pools with 2
#    wavefronts x 8 bags per workgroup, large with 8 bags per run;
#  * the delivery stand-in that feeds the overlapped backward runs on a few
#    multi-wave workgroups (library default 32 x 8 waves; large, whose
#    backward runs longest, 16 x 16), so it holds few CUs;
#  * there the consumer copies non-temporally (consume_nontemporal = 1), so
#    its stream does not displace the producer's cached rows, with 1024-2048
#    single-wave workgroups for the many short per-table items; dlrm streams
#    its rows and keeps the defaults.
PLAN_OPTS = {"skewed": {"stream_rows": 0, "table_major": 1, "slice_granule": 1, "consume_nontemporal": 1,
                        "waves_per_wg": 2, "bags_per_run": 8, "backward_bags_per_run": 3},
             "large": {"stream_rows": 0, "table_major": 2, "slice_granule": 1, "consume_nontemporal": 1,
                       "bags_per_run": 8, "deliver_wgs": 16, "deliver_waves_per_wg": 16},
             "mixed": {"stream_rows": 0, "table_major": 2, "slice_granule": 1, "consume_nontemporal": 1,
                       "backward_bags_per_run": 8}}
# Options that only steer the consumer (and, for the forward, the backward):
# they do not change what a profiled kernel does.
_NOT_FORWARD = {"consumer_wgs", "consume_nontemporal", "consume_timeout_us", "backward_bags_per_run",
                "backward_waves_per_wg", "deliver_wgs", "deliver_waves_per_wg"}
_NOT_BACKWARD = {"consumer_wgs", "consume_nontemporal", "deliver_wgs", "deliver_waves_per_wg", "stream_rows",
                 "persistent_wgs_per_cu", "rows_in_flight",
                 "waves_per_wg", "bags_per_run", "check_indices", "release_mode"}


def _kernel_options(kernel, opts):
    drop = _NOT_FORWARD if kernel == "fused_pool_kernel" else _NOT_BACKWARD
    return {k: v for k, v in (opts or {}).items() if k not in drop}
PAPER_CONTEXT = ("the paper's fused embedding + All-to-All reduced execution time by 20% intra-node "
                 "(4x MI210 over Infinity Fabric, 80 GB/s) and 31% inter-node (2x MI210 over InfiniBand, "
                 "20 GB/s); context only, those numbers include real inter-GPU transport")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash(kernel="fused_pool_kernel"):
    """Hash of the kernel's sources with comments and blank space removed:
    it changes when the code does, not when a comment does."""
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(w, lengths, weighted, n_flags=None):
    """Bytes the method itself must move for one forward: every gathered row,
    every index (+ weight), the CSR offsets, the fp32 output and one flag per
    slice."""
    import numpy as np
    L = lengths.reshape(w.T, w.B).sum(axis=1)  # indices per table
    rows = int(sum(int(L[t]) * w.dims[t] * w.elt for t in range(w.T)))
    nnz = int(L.sum())
    n_flags = w.n_chunks if n_flags is None else n_flags
    return rows + 4 * nnz + (4 * nnz if weighted else 0) + 8 * (w.T * w.B + 1) + 4 * w.B * w.sum_dim + 4 * n_flags


def traffic_record(workload, kernel="fused_pool_kernel"):
    """HBM bytes per launch from committed rocprofv3 counter runs, only if the
    kernel sources have not changed since they were taken."""
    path = os.path.join(ROOT, "profiles", TRAFFIC_FILE[kernel].format(workload))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if (rec.get("kernel_hash") != kernel_hash(kernel)
            or _kernel_options(kernel, rec.get("plan_options")) != _kernel_options(kernel, PLAN_OPTS.get(workload))):
        return None
    return rec


def time_launches(fn, steps, stream):
    import torch
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(steps):
        fn()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps  # ms per launch sequence


def time_each(fn, steps, stream):
    """Per-launch times (ms): an event pair on `stream` around every launch."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def gather_probe_gbs(row_bytes, nt=True, reps=5, buf_bytes=16 << 30, _cache={}):
    """Read rate (GB/s) of the random-row probe: uniformly random rows of
    row_bytes over a buf_bytes buffer, 16-byte loads, 8 in flight per lane --
    the practical ceiling of a uniform gather of rows that wide."""
    import torch
    from synth import device as sdev
    key = (row_bytes, nt)
    if key in _cache:
        return _cache[key]
    buf = torch.empty(buf_bytes, dtype=torch.uint8, device="cuda")
    grid = 8192
    out = torch.empty(grid * 256, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()
    nbytes = sdev.gather_probe(buf, row_bytes, 64, grid, out, nt=nt)
    ms = time_launches(lambda: sdev.gather_probe(buf, row_bytes, 64, grid, out, nt=nt), reps, s)
    del buf, out
    _cache[key] = nbytes / (ms * 1e-3) / 1e9
    return _cache[key]


def probe_ceiling(w, lengths, weighted, nt):
    """Time the fused kernel would take if every table's rows were gathered at
    the probe's rate for their width and the other bytes moved at the probe's
    widest-row rate; returns (ceiling GB/s of algorithmic bytes, us)."""
    L = lengths.reshape(w.T, w.B).sum(axis=1)
    us = 0.0
    row_total = 0
    for t in range(w.T):
        rb = w.dims[t] * w.elt
        nb = int(L[t]) * rb
        row_total += nb
        us += nb / gather_probe_gbs(rb, nt) / 1e3
    alg = algorithmic_bytes(w, lengths, weighted)
    us += (alg - row_total) / gather_probe_gbs(512, nt) / 1e3
    return alg / (us * 1e-6) / 1e9, us


def run_torch_baseline(name, steps, warmup):
    """PyTorch's own path for the same operation, as a framework user would
    write it: one torch.nn.functional.embedding_bag per table, then a
    concatenation into the [B][sum D] send layout (every pooled vector
    written into its destination row).  For comparison only: it is PyTorch's
    kernel, not this library's."""
    import torch
    import torch.nn.functional as F
    w, inp, dev, send, _ = _setup(name)
    s = torch.cuda.current_stream()
    offs = [(dev.offsets[t * w.B:(t + 1) * w.B] - dev.offsets[t * w.B]).contiguous() for t in range(w.T)]
    idx = [dev.indices[int(inp.offsets[t * w.B]):int(inp.offsets[(t + 1) * w.B])].long() for t in range(w.T)]
    wts = None if dev.weights is None else [dev.weights[int(inp.offsets[t * w.B]):int(inp.offsets[(t + 1) * w.B])]
                                            for t in range(w.T)]

    def step():
        outs = [F.embedding_bag(idx[t], dev.tables[t], offs[t], mode="sum",
                                per_sample_weights=None if wts is None else wts[t].to(dev.tables[t].dtype))
                for t in range(w.T)]
        torch.cat([o.float() for o in outs], dim=1, out=send)

    for _ in range(warmup):
        step()
    ms = time_launches(step, steps, s)
    alg = algorithmic_bytes(w, inp.lengths, inp.weights is not None)
    row = {"operator": "torch_embedding_bag_then_concat", "workload": name, "us": round(ms * 1e3, 1),
           "algorithmic_gbs": round(alg / ms / 1e6, 1), "pct_hbm_peak": round(100 * alg / ms / 1e6 / HBM_PEAK_GBS, 2),
           "torch": torch.__version__,
           "note": "per-table F.embedding_bag (storage dtype) + cat into [B][sum D] fp32; indices widened to int64 "
                   "beforehand (not timed)"}
    print(json.dumps(row), flush=True)
    # The backward the same way: autograd of the per-table embedding_bag
    # with sparse=True, whose table gradients hold one row per lookup (the
    # values ebag_a2a_backward writes); only the backward call is timed.
    for t in range(w.T):
        dev.tables[t].requires_grad_(True)
    grad = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(2305), device="cuda")
    col = 0
    grads = []
    for t in range(w.T):
        grads.append(grad[:, col:col + w.dims[t]].to(dev.tables[t].dtype).contiguous())
        col += w.dims[t]
    times = []
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for it in range(warmup + steps):
        for t in range(w.T):
            dev.tables[t].grad = None
        outs = [F.embedding_bag(idx[t], dev.tables[t], offs[t], mode="sum", sparse=True,
                                per_sample_weights=None if wts is None else wts[t].to(dev.tables[t].dtype))
                for t in range(w.T)]
        torch.cuda.synchronize()
        ev0.record(s)
        torch.autograd.backward(outs, grads)
        ev1.record(s)
        torch.cuda.synchronize()
        if it >= warmup:
            times.append(ev0.elapsed_time(ev1))
    ms = sum(times) / len(times)
    bb = backward_bytes(w, inp.lengths, inp.weights is not None)
    brow = {"operator": "torch_embedding_bag_sparse_backward", "workload": name, "us": round(ms * 1e3, 1),
            "algorithmic_gbs": round(bb / ms / 1e6, 1), "torch": torch.__version__,
            "note": "autograd of per-table F.embedding_bag(sparse=True): sparse table gradients with one row per "
                    "lookup; the backward call alone is timed"}
    print(json.dumps(brow), flush=True)
    for t in range(w.T):
        dev.tables[t].requires_grad_(False)
        dev.tables[t].grad = None
    return row


def run_torch_gemv_baseline(steps, warmup, R=4):
    """PyTorch's path for GEMV + AllReduce on one GPU: torch.mv of every
    rank's fp16 block (the vendor BLAS), then a sum of the R partial vectors
    in fp32 -- for comparison with the fused operator's shapes."""
    import torch
    s = torch.cuda.current_stream()
    out = []
    for M, K in GEMV_SHAPES:
        Ks = [K // R] * R
        g = torch.Generator(device="cuda").manual_seed(2305 + M)
        A = [torch.randn((M, k), generator=g, device="cuda").half() for k in Ks]
        x = [torch.randn((k,), generator=g, device="cuda").half() for k in Ks]

        def step():
            torch.stack([torch.mv(A[r], x[r]).float() for r in range(R)]).sum(0)

        for _ in range(warmup):
            step()
        ms = time_launches(step, steps, s)
        nbytes = gemv_ar_bytes(R, M, K, 2)
        row = {"operator": "torch_mv_then_sum", "ranks": R, "M": M, "K": K, "us": round(ms * 1e3, 1),
               "algorithmic_gbs": round(nbytes / ms / 1e6, 1), "torch": torch.__version__}
        print(json.dumps(row), flush=True)
        out.append(row)
        del A, x
    return out


def run_stream_probe(reps=20):
    """Streaming ceilings: reads (synth_stream_read, 16-byte non-temporal
    loads, 8 in flight per lane; best of several grid sizes) and writes
    (torch fill_) of 256 MiB, 1 GiB and 4 GiB."""
    import torch
    from synth import device as sdev
    s = torch.cuda.current_stream()
    rows = []
    for nbytes in (256 << 20, 1 << 30, 4 << 30):
        buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        best = None
        for grid in (1024, 2048, 4096, 8192, 16384):
            out = torch.empty(grid * 256, dtype=torch.int32, device="cuda")
            sdev.stream_read(buf, grid, out)
            ms = time_launches(lambda: sdev.stream_read(buf, grid, out), reps, s)
            if best is None or ms < best[1]:
                best = (grid, ms)
        fill_ms = time_launches(lambda: buf.fill_(2.0), reps, s)
        row = {"bytes": nbytes, "read_gbs": round(nbytes / best[1] / 1e6, 1), "read_grid": best[0],
               "write_gbs": round(nbytes / fill_ms / 1e6, 1)}
        rows.append(row)
        print(json.dumps(row), flush=True)
        del buf
    return rows


def run_row_probe():
    rows = []
    for rb in (64, 128, 256, 512, 1024):
        for nt in (True, False):
            g = gather_probe_gbs(rb, nt)
            row = {"row_bytes": rb, "nontemporal": nt, "gbs": round(g, 1), "rows_per_us": round(g * 1e3 / rb, 1)}
            rows.append(row)
            print(json.dumps(row), flush=True)
    return rows


def cpu_baseline(w, inp, bytes_fn, max_tables=None, min_seconds=10.0, mean=False):
    """The CPU oracle timed on this host's cores over the first tables of the
    same workload (all B samples of each)."""
    import numpy as np
    import oracle
    cores = len(os.sched_getaffinity(0))
    T = w.T if max_tables is None else min(w.T, max_tables)
    try:
        avail = int([l for l in open("/proc/meminfo") if l.startswith("MemAvailable")][0].split()[1]) * 1024
    except Exception:
        avail = 0
    per_table = w.table_bytes() / w.T
    while T > 1 and T * per_table * 2.5 > avail:
        T //= 2
    t0 = time.time()
    tables = [inp.table(t) for t in range(T)]
    gen_s = time.time() - t0
    off = inp.offsets[:T * w.B + 1]
    idx = inp.indices[:int(off[-1])]
    wts = None if inp.weights is None else inp.weights[:int(off[-1])]
    sub = w.with_(T=T, rows=w.rows[:T], dims=w.dims[:T])
    nbytes = bytes_fn(sub, inp.lengths[:T * w.B], inp.weights is not None)
    # Repeat the pass until about min_seconds of CPU time have been measured
    # (at least 3 passes) and report the median pass.
    times = []
    while len(times) < 3 or sum(times) < min_seconds:
        t0 = time.time()
        oracle.pool(tables, w.dtype, sub.dims, idx, off, wts, w.B, w.R, w.C, nthreads=cores,
                    want_abs=False, want_sum=True, want_send=True, mean=mean)
        times.append(time.time() - t0)
    med = sorted(times)[len(times) // 2]
    cpu_model = ""
    try:
        cpu_model = [l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name")][0]
    except Exception:
        pass
    return {"value": round(nbytes / med / 1e9, 3), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"C oracle (fp64) over tables 0..{T - 1} of {w.T}, all {w.B} samples "
                      f"({nbytes / 1e9:.2f} GB algorithmic), median of {len(times)} passes ({sum(times):.1f} s in all), "
                      f"{med:.3f} s per pass; "
                      f"host tables generated in {gen_s:.1f} s (not timed); CPU {cpu_model}"}


def e2e_us(plan, w, dev, send, recv, flags, epoch, fused_path, consumer_first, prod, cons, stream, steps, warmup):
    """Median microseconds from the start of the first enqueued kernel to the
    end of both the forward (on prod) and the consumer (on cons).  epoch is a
    one-element list holding the flags' current epoch."""
    import torch
    fwd = plan.forward if fused_path else plan.unfused_forward
    ev0 = torch.cuda.Event(enable_timing=True)
    ev_p, ev_c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    first, second = (cons, prod) if consumer_first else (prod, cons)
    times = []
    for it in range(warmup + steps):
        first.wait_stream(stream)
        ev0.record(first)
        second.wait_event(ev0)
        epoch[0] += 1
        for s in (first, second):
            with torch.cuda.stream(s):
                if s is prod:
                    fwd(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags)
                else:
                    plan.consume(send, flags, recv, w.B, w.R, epoch[0])
        ev_p.record(prod)
        ev_c.record(cons)
        torch.cuda.synchronize()
        if it >= warmup:
            times.append(max(ev0.elapsed_time(ev_p), ev0.elapsed_time(ev_c)))
    st = plan.status_ex()
    assert st == (0, -1, 0, -1), f"consumer status {st}"
    assert torch.equal(send.view(torch.int32), recv.view(torch.int32)), "consumer copy differs"
    return round(1e3 * sorted(times)[len(times) // 2], 2) if times else None


ZIPF = ("skewed", "large")  # workloads whose rows repeat: HBM bytes are argued on counters and unique rows


def roofline(name, alg, unique_bytes, fused_ms, traffic_bytes):
    """Roofline of the fused pooling kernel for one workload.  frac: the
    method's algorithmic bytes (every gathered row) over the kernel time, the
    contract figure; under Zipf indices many rows hit L2 or the Infinity
    Cache, so it can exceed the HBM peak.  frac_unique_rows: distinct rows
    plus every other byte over the same time, the least HBM traffic the
    launch can have.  frac_counter: the L2 fill and write bytes measured by
    counters (FETCH_SIZE + WRITE_SIZE, an upper bound on HBM traffic, since
    fills served by the Infinity Cache count too), null when the committed
    counter record does not match the kernel sources.  claim names the
    figure the workload's HBM efficiency is stated on."""
    t = fused_ms * 1e-3
    r = {"bound": "hbm", "achieved": round(alg / t / 1e9, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": round(alg / t / 1e9 / HBM_PEAK_GBS, 4), "traffic": traffic_bytes,
         "kernel": "fused_pool_kernel",
         "frac_unique_rows": round(unique_bytes / t / 1e9 / HBM_PEAK_GBS, 4),
         "frac_counter": None if traffic_bytes is None else round(traffic_bytes / t / 1e9 / HBM_PEAK_GBS, 4)}
    if name in ZIPF:
        r["claim"] = "frac_unique_rows"
        r["basis"] = ("Zipf indices: rows repeat, so algorithmic bytes overstate HBM traffic; the claim is distinct "
                      "rows + other bytes over the kernel time (a lower bound on HBM bytes), next to the counter "
                      "bytes (an upper bound)")
    else:
        r["claim"] = "frac"
        r["basis"] = ("uniform indices: a row's repeats are far apart in time, so every lookup is fetched past L2 "
                      "(counter bytes match algorithmic bytes); distinct-row bytes are a looser lower bound")
    return r


def run_workload(name, steps, warmup, with_cpu, profile, mean=False, per_table=False, light=False, cpu_tables=None,
                 queues=None):
    """One workload's figures.  light: fused and unfused times, the
    concurrent-consumer times and the roofline only (no per-launch timing,
    trace, probes, CPU oracle or environment).  queues: a (producer,
    consumer) pair of hardware-queue streams to reuse."""
    import dataclasses

    import numpy as np
    import torch

    import paper_2305_06942_amd as ebag
    import synth
    from synth import device as sdev

    w = synth.FULL[name]
    t0 = time.time()
    inp = synth.make_inputs(w)
    if mean:
        # mean pooling takes no weights: the same bags, unweighted
        w = w.with_(weighted=False)
        inp = dataclasses.replace(inp, w=w, weights=None)
    log(f"[{name}] inputs generated in {time.time() - t0:.1f} s (nnz={inp.nnz})")
    dev = sdev.to_device(inp)
    torch.cuda.synchronize()
    opts = dict(PLAN_OPTS.get(name, {}))
    if mean:
        opts["pooling_mode"] = 1
    if per_table:
        opts["slice_granule"] = 1
    per_table_slices = opts.get("slice_granule", 0) == 1
    n_flags = w.n_chunks * (w.T if per_table_slices else 1)
    alg = algorithmic_bytes(w, inp.lengths, inp.weights is not None, n_flags)
    plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, **opts)
    send = torch.empty((w.B, w.sum_dim), dtype=torch.float32, device="cuda")
    recv = torch.empty_like(send)
    flags = torch.zeros(n_flags, dtype=torch.int32, device="cuda")
    epoch = [0]
    stream = torch.cuda.current_stream()

    def fused():
        plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags)
        epoch[0] += 1

    def unfused():
        plan.unfused_forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags)
        epoch[0] += 1

    for _ in range(warmup):
        fused()
    fused_ms = time_launches(fused, steps, stream)
    for _ in range(warmup):
        unfused()
    unfused_ms = time_launches(unfused, steps, stream)
    # the same launches one at a time, for the median and the fastest
    each = {} if (profile or light) else {"fused": time_each(fused, steps, stream),
                                          "unfused": time_each(unfused, steps, stream)}
    log(f"[{name}] fused {fused_ms * 1e3:.1f} us  unfused {unfused_ms * 1e3:.1f} us")
    assert np.all(flags.cpu().numpy().view(np.uint32) == epoch[0]), "flags do not match the number of forwards"

    out = {
        "metric": "fused pooled-gather GB/s (% HBM peak) + fused vs unfused us per batch",
        "value": round(alg / (fused_ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(fused_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {0: "f32", 1: "f16->f32", 2: "bf16->f32"}[w.dtype],
        "data": "synthetic (seeded generator; shapes of the workload below)",
        "config": {"workload": name, "tables": w.T, "rows": w.rows[0], "dims": sorted(set(w.dims)),
                   "storage": {0: "f32", 1: "f16", 2: "bf16"}[w.dtype], "global_batch": w.B,
                   "bag_lengths": w.lengths, "indices": w.indices, "weighted": w.weighted,
                   "pooling": "mean" if mean else "sum",
                   "slices": "per table" if per_table_slices else "all tables",
                   "run_order": {0: "slice-major", 1: "table-major, one table per XCD at a time",
                                 2: "table-major, one table at a time"}[opts.get("table_major", 0)],
                   "destinations": w.R, "slice_samples": w.C, "parallelism": "1 GPU, R logical destinations"},
        "fused_us": round(fused_ms * 1e3, 2),
        "unfused_us": round(unfused_ms * 1e3, 2),
        "fused_speedup_vs_unfused": round(unfused_ms / fused_ms, 4),
        **{f"{k}_us_{stat}": round(f(v) * 1e3, 2) for k, v in each.items()
           for stat, f in (("median", lambda x: float(np.median(x))), ("min", min))},
        "pct_hbm_peak": round(100 * alg / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "algorithmic_bytes": alg,
        "plan_options": opts,
    }
    if profile:
        # a plain copy of known size: calibrates the byte counters per dispatch
        import torch as _t
        from synth import device as _sd
        nb = 1 << 30
        src = _t.ones(nb // 4, device="cuda")
        dst = _t.empty_like(src)
        for _ in range(2):
            _sd.copy(dst, src, nb)
        _t.cuda.synchronize()
        out["calibration_copy_bytes"] = nb
        return out
    # End to end with the concurrent consumer: producer enqueued first, each
    # on a stream with a hardware queue of its own, so the two always run
    # concurrently.
    own_queues = queues is None
    prod, cons = (ebag.queue_stream(), ebag.queue_stream()) if own_queues else queues
    # Below 0.1 ms the launch and cross-queue latencies dominate each sample:
    # take the median over more of them.
    e2e_steps = steps if fused_ms >= 0.1 else max(steps, 200)
    for fused_path in (True, False):
        key = ("fused" if fused_path else "unfused") + "_plus_consumer_us"
        out[key] = e2e_us(plan, w, dev, send, recv, flags, epoch, fused_path, False, prod, cons, stream, e2e_steps,
                          warmup)
    if not light:
        # overlap evidence from device timestamps
        tplan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, trace=1, **opts)
        e2e_us(tplan, w, dev, send, recv, flags, epoch, True, False, prod, cons, stream, 1, 0)
        rel, drn, tpu = tplan.trace(n_flags)
        tplan.close()
        out["first_drain_before_last_release_us"] = round(float(int(rel.max()) - int(drn.min())) / tpu, 2)
        out["slices_drained_before_last_release"] = int((drn < rel.max()).sum())
        out["median_drain_lag_us"] = round(float(np.median(drn.astype(np.int64) - rel.astype(np.int64))) / tpu, 2)
        out["n_slices"] = n_flags
    if own_queues:
        for q in (prod, cons):
            ebag.queue_stream_destroy(q)
    rows_alg = int(sum(int(inp.lengths.reshape(w.T, w.B)[t].sum()) * w.dims[t] * w.elt for t in range(w.T)))
    unique_bytes = alg - rows_alg + inp.unique_row_bytes()
    out["unique_row_bytes"] = unique_bytes
    out["unique_row_gbs"] = round(unique_bytes / (fused_ms * 1e-3) / 1e9, 2)
    if not light and name not in ZIPF:
        ceil_gbs, ceil_us = probe_ceiling(w, inp.lengths, inp.weights is not None, bool(opts.get("stream_rows", 1)))
        out["random_row_probe_ceiling"] = {
            "gbs": round(ceil_gbs, 1), "us": round(ceil_us, 1), "frac": round(out["value"] / ceil_gbs, 4),
            "note": "uniform random rows of each table's width at the probe's measured rate"}
    tr = None if (mean or per_table) else traffic_record(name)
    out["roofline"] = roofline(name, alg, unique_bytes, fused_ms, tr["hbm_bytes_per_launch"] if tr else None)
    if light:
        del dev, send, recv
        return out
    out["paper_context"] = PAPER_CONTEXT
    del dev, send, recv
    torch.cuda.empty_cache()
    if with_cpu:
        log(f"[{name}] timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(w, inp, algorithmic_bytes, max_tables=cpu_tables, mean=mean)
    out["env"] = env_info(inp)
    return out


# The headline line: the largest workload that fits one GPU (131 GB of tables
# resident), many tables and long Zipf-distributed bags, the closest of the
# five to the paper's many-table, long-pooling setting.
HEADLINE = "large"
# Tables the CPU oracle is timed on (all B samples of each), where the whole
# workload would take too long or too much host memory.
CPU_TABLES = {"large": 4}
SECONDARY = ("tiny", "dlrm", "skewed", "mixed")
_LIGHT_KEYS = ("fused_us", "unfused_us", "fused_speedup_vs_unfused", "fused_plus_consumer_us",
               "unfused_plus_consumer_us", "pct_hbm_peak", "algorithmic_bytes", "unique_row_bytes", "plan_options")


def run_headline(steps, warmup, with_cpu=True):
    """The default line: the headline workload in full, and for each of the
    other four its fused and unfused times, concurrent-consumer times and
    roofline under "workloads" (no probes or CPU legs for those)."""
    import paper_2305_06942_amd as ebag
    import torch
    queues = (ebag.queue_stream(), ebag.queue_stream())
    try:
        out = run_workload(HEADLINE, steps, warmup, with_cpu=with_cpu, profile=False,
                           cpu_tables=CPU_TABLES.get(HEADLINE), queues=queues)
        torch.cuda.empty_cache()
        others = {}
        for n in SECONDARY:
            try:
                r = run_workload(n, steps, warmup, with_cpu=False, profile=False, light=True, queues=queues)
                others[n] = {k: r[k] for k in _LIGHT_KEYS if k in r}
                others[n]["roofline"] = {k: r["roofline"][k] for k in
                                         ("frac", "frac_unique_rows", "frac_counter", "traffic", "claim")}
            except Exception as e:  # one failing workload must not lose the headline
                others[n] = {"error": f"{type(e).__name__}: {e}"}
            torch.cuda.empty_cache()
        out["workloads"] = others
    finally:
        for q in queues:
            ebag.queue_stream_destroy(q)
    return out


def git_head():
    """The checked-out commit, read from .git without running git (None when
    the tree has no .git)."""
    try:
        with open(os.path.join(ROOT, ".git", "HEAD")) as f:
            head = f.read().strip()
        if head.startswith("ref: "):
            ref = head[5:]
            path = os.path.join(ROOT, ".git", ref)
            if os.path.exists(path):
                with open(path) as f:
                    return f.read().strip()[:12]
            with open(os.path.join(ROOT, ".git", "packed-refs")) as f:
                for line in f:
                    if line.strip().endswith(" " + ref):
                        return line.split()[0][:12]
            return None
        return head[:12]
    except OSError:
        return None


def env_info(inp=None):
    """Where and on what the numbers were taken: device, architecture, HIP
    and torch versions, the hash of the pooling kernels' sources, the git
    commit when the tree has one, and a digest of the workload's inputs."""
    import torch
    props = torch.cuda.get_device_properties(0)
    env = {"device": torch.cuda.get_device_name(0), "arch": getattr(props, "gcnArchName", None),
           "cus": props.multi_processor_count, "hip": torch.version.hip, "torch": torch.__version__,
           "kernel_sources": kernel_hash()}
    env["git"] = git_head()
    if inp is not None:
        h = hashlib.sha256()
        for a in (inp.offsets, inp.indices, inp.weights):
            if a is not None:
                h.update(a.tobytes())
        env["inputs_sha256"] = h.hexdigest()[:16]
    return env


def _setup(name):
    import torch
    import synth
    from synth import device as sdev
    w = synth.FULL[name]
    inp = synth.make_inputs(w)
    dev = sdev.to_device(inp)
    send = torch.empty((w.B, w.sum_dim), dtype=torch.float32, device="cuda")
    flags = torch.zeros(w.n_chunks * w.T, dtype=torch.int32, device="cuda")  # room for per-table slices
    return w, inp, dev, send, flags


def run_placement(name, steps, warmup, reps=3):
    """Fused and unfused kernel time with the send buffer allocated before the
    tables and with it allocated after them (the benchmark's own order), on
    the same inputs in one process, alternating.  The kernels write the send
    layout's row pieces at a stride of sum(D) floats; where the buffer's pages
    land decides how those pieces fall on the memory channels."""
    import torch
    import synth
    import paper_2305_06942_amd as ebag
    from synth import device as sdev
    w = synth.FULL[name]
    inp = synth.make_inputs(w)
    before = torch.empty((w.B, w.sum_dim), dtype=torch.float32, device="cuda")
    dev = sdev.to_device(inp)
    after = torch.empty((w.B, w.sum_dim), dtype=torch.float32, device="cuda")
    flags = torch.zeros(w.n_chunks * w.T, dtype=torch.int32, device="cuda")
    plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, **dict(PLAN_OPTS.get(name, {})))
    s = torch.cuda.current_stream()
    out = {"study": "send-buffer placement", "workload": name, "steps": steps, "warmup": warmup,
           "plan_options": PLAN_OPTS.get(name, {}),
           "send_before_tables": hex(before.data_ptr()), "send_after_tables": hex(after.data_ptr()),
           "first_table": hex(dev.tables[0].data_ptr()),
           "fused_us": {"before_tables": [], "after_tables": []},
           "unfused_us": {"before_tables": [], "after_tables": []}}
    for _ in range(reps):
        for key, buf in (("before_tables", before), ("after_tables", after)):
            for kind, call in (("fused_us", plan.forward), ("unfused_us", plan.unfused_forward)):
                f = lambda: call(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, buf, flags)
                for _ in range(warmup):
                    f()
                out[kind][key].append(round(time_launches(f, steps, s) * 1e3, 1))
    plan.close()
    return out


def run_occupancy(name, steps, warmup):
    """Fused-kernel time versus the fraction of resident workgroup slots a
    persistent grid occupies (Sec. IV-C, Fig. 13), for 2, 4 and 8 waves per
    workgroup, next to the default one-workgroup-per-run grid."""
    import torch
    import paper_2305_06942_amd as ebag
    w, inp, dev, send, flags = _setup(name)
    alg = algorithmic_bytes(w, inp.lengths, w.weighted)
    base = dict(PLAN_OPTS.get(name, {}))
    base.pop("persistent_wgs_per_cu", None)  # the swept parameter
    s = torch.cuda.current_stream()
    rows = []
    for waves in (2, 4, 8):
        probe = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, waves_per_wg=waves, **base)
        max_wgs, cus, block, K = probe.occupancy(w.weighted)
        probe.close()
        for per_cu in [0] + list(range(1, max_wgs + 1)):
            plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, waves_per_wg=waves,
                             persistent_wgs_per_cu=per_cu, **base)
            f = lambda: plan.forward(dev.tables, dev.indices, dev.offsets, dev.weights, w.B, w.R, send, flags)
            for _ in range(warmup):
                f()
            ms = time_launches(f, steps, s)
            plan.close()
            row = {"workload": name, "waves_per_wg": waves, "persistent_wgs_per_cu": per_cu,
                   "max_wgs_per_cu": max_wgs, "occupancy": round(per_cu / max_wgs, 4) if per_cu else None,
                   "grid": "one workgroup per run" if per_cu == 0 else f"{per_cu * cus} persistent",
                   "fused_us": round(ms * 1e3, 2), "gbs": round(alg / (ms * 1e-3) / 1e9, 1)}
            rows.append(row)
            print(json.dumps(row), flush=True)
    return rows


def run_timeline(name, warmup):
    """Per-slice release and drain times of one traced forward + concurrent
    consumer (enqueued after it, on its own hardware queue), in natural slice order and in communication-aware order
    (destination self_rank = 0 kept local and produced last; Sec. III-A,
    Sec. IV-C, Fig. 14).  Times in us from the first release."""
    import numpy as np
    import torch
    import paper_2305_06942_amd as ebag
    w, inp, dev, send, flags = _setup(name)
    recv = torch.empty_like(send)
    # whole slices in slice-major order: the study is the order of slices
    base = {k: v for k, v in PLAN_OPTS.get(name, {}).items() if k not in ("slice_granule", "table_major")}
    prod, cons = ebag.queue_stream(), ebag.queue_stream()
    stream = torch.cuda.current_stream()
    epoch = [0]
    per = w.n_chunks // w.R
    out = []
    for order in (0, 1):
        plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, trace=1, chunk_order=order, self_rank=0, **base)
        e2e_us(plan, w, dev, send, recv, flags, epoch, True, False, prod, cons, stream, 1, warmup)
        assert plan.status_ex() == (0, -1, 0, -1)
        rel, drn, tpu = plan.trace(w.n_chunks)
        t0 = int(rel.min())
        r_us = (rel.astype(np.int64) - t0) / tpu
        d_us = (drn.astype(np.int64) - t0) / tpu
        remote = np.ones(w.n_chunks, dtype=bool)
        remote[0:per] = False  # destination 0 is the local one
        row = {"workload": name, "chunk_order": order, "self_rank": 0, "n_slices": w.n_chunks,
               "last_release_us": round(float(r_us.max()), 2),
               "last_remote_release_us": round(float(r_us[remote].max()), 2),
               "last_local_release_us": round(float(r_us[~remote].max()), 2),
               "last_remote_drain_us": round(float(d_us[remote].max()), 2),
               "last_drain_us": round(float(d_us.max()), 2),
               "median_drain_lag_us": round(float(np.median(d_us - r_us)), 2),
               "release_us_by_slice": [round(float(x), 1) for x in r_us],
               "drain_us_by_slice": [round(float(x), 1) for x in d_us]}
        plan.close()
        out.append(row)
        print(json.dumps(row), flush=True)
    for q in (prod, cons):
        ebag.queue_stream_destroy(q)
    return out


def backward_bytes(w, lengths, weighted):
    """Bytes the embedding backward must move: every per-lookup row written,
    the pooled gradient read once, the CSR offsets, and the weights."""
    L = lengths.reshape(w.T, w.B).sum(axis=1)
    rows = int(sum(int(L[t]) * w.dims[t] * 4 for t in range(w.T)))
    nnz = int(L.sum())
    return rows + 4 * w.B * w.sum_dim + 8 * (w.T * w.B + 1) + (4 * nnz if weighted else 0)


def backward_cpu_baseline(w, inp, grad, mean=False, max_bytes=2 << 30, min_seconds=10.0):
    """The C oracle's embedding backward (one thread) timed on this host over
    the first tables of the workload whose per-lookup rows fit in max_bytes
    (all B samples of each), repeated until about min_seconds."""
    import numpy as np
    import oracle
    L = inp.lengths.reshape(w.T, w.B).sum(axis=1)
    T, acc = 0, 0
    while T < w.T and acc + int(L[T]) * w.dims[T] * 4 <= max_bytes:
        acc += int(L[T]) * w.dims[T] * 4
        T += 1
    T = max(T, 1)
    sub = w.with_(T=T, rows=w.rows[:T], dims=w.dims[:T])
    off = inp.offsets[:T * w.B + 1]
    nnz = int(off[-1])
    wts = None if inp.weights is None else inp.weights[:nnz]
    g = np.ascontiguousarray(grad[:, :sub.sum_dim])
    nbytes = backward_bytes(sub, inp.lengths[:T * w.B], wts is not None)
    times = []
    while len(times) < 3 or sum(times) < min_seconds:
        t0 = time.time()
        oracle.backward(sub.dims, off, wts, g, w.B, w.R, mean=mean)
        times.append(time.time() - t0)
    med = sorted(times)[len(times) // 2]
    return {"value": round(nbytes / med / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"C oracle (one thread) over tables 0..{T - 1} of {w.T}, all {w.B} samples "
                      f"({nbytes / 1e9:.2f} GB algorithmic), median of {len(times)} passes ({sum(times):.1f} s in all)"}


def run_backward(name, steps, warmup, profile=False, with_cpu=True):
    """Embedding backward: the kernel alone (gradient complete), the
    bulk-synchronous sequence (delivery of the gradient, then the backward)
    and the fused one (backward expanding slices as the delivery lands).
    profile: the kernel alone and the delivery, on one ordinary stream (for
    rocprofv3 kernel traces)."""
    import torch
    import paper_2305_06942_amd as ebag
    w, inp, dev, _, _ = _setup(name)
    opts = dict(PLAN_OPTS.get(name, {}))
    opts.pop("stream_rows", None)
    opts.pop("persistent_wgs_per_cu", None)
    plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, **opts)
    n_vals = int(sum((inp.offsets[(t + 1) * w.B] - inp.offsets[t * w.B]) * w.dims[t] for t in range(w.T)))
    values = torch.empty((n_vals,), device="cuda")
    g = torch.Generator(device="cuda").manual_seed(2305)
    grad_dp = torch.randn((w.B, w.sum_dim), generator=g, device="cuda")
    grad_recv = torch.empty_like(grad_dp)
    flags = torch.zeros(plan.n_flags(w.B), dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()
    nbytes = backward_bytes(w, inp.lengths, inp.weights is not None)
    bwd = lambda: plan.backward(grad_recv, dev.offsets, dev.weights, w.B, w.R, values)
    for _ in range(warmup):
        bwd()
    k_ms = time_launches(bwd, steps, s)
    if profile:
        d_ms = time_launches(lambda: plan.deliver(grad_dp, grad_recv, flags, w.B, w.R), steps, s)
        from synth import device as _sd
        src = torch.ones((1 << 30) // 4, device="cuda")  # counter calibration: two 1 GiB copies
        dst = torch.empty_like(src)
        for _ in range(2):
            _sd.copy(dst, src, 1 << 30)
        torch.cuda.synchronize()
        print(json.dumps({"operator": "embedding_backward", "workload": name, "kernel_us": round(k_ms * 1e3, 2),
                          "deliver_us": round(d_ms * 1e3, 2), "algorithmic_bytes": nbytes,
                          "calibration_copy_bytes": 1 << 30}), flush=True)
        plan.close()
        return None
    epoch = [0]
    send_q, bwd_q = ebag.queue_stream(), ebag.queue_stream()
    # The bulk-synchronous sequence waits for the whole delivery, so it gets
    # the fastest one: a bandwidth-sized copy of 2048 single-wave workgroups.
    # The overlapped sequence uses the plan's delivery, which holds few CUs
    # while the backward runs beside it.
    bulk = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, **dict(opts, deliver_wgs=2048, deliver_waves_per_wg=1))

    def sequence(fused):
        ev0, ev1, ev2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        times = []
        for it in range(warmup + steps):
            send_q.wait_stream(s)
            ev0.record(send_q)
            bwd_q.wait_event(ev0)
            epoch[0] += 1
            with torch.cuda.stream(send_q):
                (plan if fused else bulk).deliver(grad_dp, grad_recv, flags, w.B, w.R)
            if not fused:
                bwd_q.wait_stream(send_q)
            with torch.cuda.stream(bwd_q):
                plan.backward(grad_recv, dev.offsets, dev.weights, w.B, w.R, values,
                              grad_flags=flags if fused else None, expected_epoch=epoch[0])
            ev1.record(send_q)
            ev2.record(bwd_q)
            torch.cuda.synchronize()
            if it >= warmup:
                times.append(max(ev0.elapsed_time(ev1), ev0.elapsed_time(ev2)))
        assert plan.status_ex() == (0, -1, 0, -1)
        return sorted(times)[len(times) // 2]
    f_ms = sequence(True)
    u_ms = sequence(False)
    tr = traffic_record(name, "backward_kernel")
    row = {"operator": "embedding_backward", "workload": name, "values_bytes": 4 * n_vals,
           "algorithmic_bytes": nbytes, "kernel_us": round(k_ms * 1e3, 2),
           "fused_with_delivery_us": round(f_ms * 1e3, 2), "delivery_then_backward_us": round(u_ms * 1e3, 2),
           "fused_speedup": round(u_ms / f_ms, 4),
           "roofline": {"bound": "hbm", "achieved": round(nbytes / (k_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(nbytes / (k_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "traffic": tr["hbm_bytes_per_launch"] if tr else None},
           "data": "synthetic: the workload's bags, a seeded torch.randn pooled gradient"}
    if with_cpu:
        row["cpu_baseline"] = backward_cpu_baseline(w, inp, grad_dp.cpu().numpy())
    row["env"] = env_info(inp)
    print(json.dumps(row), flush=True)
    plan.close()
    bulk.close()
    for q in (send_q, bwd_q):
        ebag.queue_stream_destroy(q)
    return row


def run_backward_sweep(name, steps, warmup):
    """Backward kernel time over its launch shape: bags and waves per
    workgroup (the gradient complete; one JSON line per shape), in the
    workload's own run order and slices (its PLAN_OPTS)."""
    import torch
    import paper_2305_06942_amd as ebag
    w, inp, dev, _, _ = _setup(name)
    opts = {k: v for k, v in PLAN_OPTS.get(name, {}).items() if not k.startswith("backward_")}
    n_vals = int(sum((inp.offsets[(t + 1) * w.B] - inp.offsets[t * w.B]) * w.dims[t] for t in range(w.T)))
    values = torch.empty((n_vals,), device="cuda")
    grad = torch.randn((w.B, w.sum_dim), generator=torch.Generator(device="cuda").manual_seed(2305), device="cuda")
    nbytes = backward_bytes(w, inp.lengths, inp.weights is not None)
    s = torch.cuda.current_stream()
    for waves in (4, 8, 16):
        for bags in (1, 2, 3, 4, 6, 8, 16):
            plan = ebag.Plan(w.rows, w.dims, w.dtype, w.C, w.B, w.R, backward_waves_per_wg=waves,
                             backward_bags_per_run=bags, **opts)
            f = lambda: plan.backward(grad, dev.offsets, dev.weights, w.B, w.R, values)
            for _ in range(warmup):
                f()
            ms = time_launches(f, steps, s)
            print(json.dumps({"operator": "embedding_backward", "workload": name, "waves_per_wg": waves,
                              "bags_per_wg": bags, "kernel_us": round(ms * 1e3, 1),
                              "GB/s": round(nbytes / ms / 1e6, 1)}), flush=True)
            plan.close()


GEMV_SHAPES = [(16384, 8192), (32768, 8192), (65536, 8192)]  # (M outputs, K total), R = 4 ranks, fp16


def gemv_ar_bytes(R, M, K, elt):
    """Bytes the fused GEMV + AllReduce must move: every matrix element and
    vector element once, each rank's partial vector written and read once
    (the reduce-scatter) and the reduced vector written to every rank (the
    all-gather)."""
    return M * K * elt + K * elt + 2 * R * M * 4 + R * M * 4


def run_gemv_ar(steps, warmup, R=4, dtype=1, shapes=GEMV_SHAPES, with_cpu=True, profile=False):
    """GEMV + AllReduce (Sec. III-B) on R logical ranks: fused (one launch;
    the last arriver reduces) against bulk-synchronous (GEMV kernel, then
    AllReduce kernel, then flags), one JSON line per shape.  profile: also
    two 1 GiB copies that calibrate the byte counters."""
    import numpy as np
    import torch
    import paper_2305_06942_amd as ebag
    s = torch.cuda.current_stream()
    elt = 4 if dtype == 0 else 2
    tdt = {0: torch.float32, 1: torch.float16, 2: torch.bfloat16}[dtype]
    out = []
    for M, K in shapes:
        Ks = [K // R] * R
        g = torch.Generator(device="cuda").manual_seed(2305 + M)
        A = [torch.randn((M, k), generator=g, device="cuda").to(tdt) for k in Ks]
        x = [torch.randn((k,), generator=g, device="cuda").to(tdt) for k in Ks]
        y = [torch.empty((M,), device="cuda") for _ in range(R)]
        plan = ebag.GemvAR(R, M, Ks, dtype)
        P, block, n_tiles, resident, tile_rows = plan.launch_info()
        flags = torch.zeros(R * P, dtype=torch.int32, device="cuda")
        fused = lambda: plan.forward(A, x, y, flags)
        unfused = lambda: plan.unfused_forward(A, x, y, flags)
        for _ in range(warmup):
            fused()
            unfused()
        f_ms = time_launches(fused, steps, s)
        u_ms = time_launches(unfused, steps, s)
        assert plan.status() == (0, -1)
        nbytes = gemv_ar_bytes(R, M, K, elt)
        row = {"operator": "gemv_allreduce", "ranks": R, "M": M, "K": K, "dtype": {0: "f32", 1: "f16", 2: "bf16"}[dtype],
               "tile_rows": tile_rows, "wgs_per_rank": P, "threads_per_wg": block,
               "fused_us": round(f_ms * 1e3, 2), "unfused_us": round(u_ms * 1e3, 2),
               "fused_speedup_vs_unfused": round(u_ms / f_ms, 4), "algorithmic_bytes": nbytes,
               "roofline": {"bound": "hbm", "achieved": round(nbytes / (f_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                            "unit": "GB/s", "frac": round(nbytes / (f_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                            "traffic": None, "kernel": "gemv_ar_last_arriver_kernel"},
               "data": "synthetic: torch.randn on the device, seeded"}
        tr = traffic_record(f"m{M}", "gemv_ar_last_arriver_kernel")
        if tr:
            row["roofline"]["traffic"] = tr["hbm_bytes_per_launch"]
        if profile:
            # a plain copy of known size: calibrates the byte counters per dispatch
            from synth import device as _sd
            src = torch.ones((1 << 30) // 4, device="cuda")
            dst = torch.empty_like(src)
            for _ in range(2):
                _sd.copy(dst, src, 1 << 30)
            torch.cuda.synchronize()
            row["calibration_copy_bytes"] = 1 << 30
            del src, dst
        if with_cpu and M == shapes[0][0]:
            import oracle
            hA = [a.cpu().numpy() if dtype != 2 else a.view(torch.int16).cpu().numpy().view(np.uint16) for a in A]
            hx = [v.cpu().numpy() if dtype != 2 else v.view(torch.int16).cpu().numpy().view(np.uint16) for v in x]
            times = []
            while len(times) < 3 or sum(times) < 10.0:
                t0 = time.time()
                oracle.gemv_ar(hA, hx, dtype)
                times.append(time.time() - t0)
            med = sorted(times)[len(times) // 2]
            row["cpu_baseline"] = {"value": round(nbytes / med / 1e9, 3), "unit": "GB/s",
                                   "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
                                   "sample": f"C oracle (fp64) over the whole {M} x {K} problem, median of "
                                             f"{len(times)} passes, {med:.3f} s per pass"}
        row["env"] = env_info()
        out.append(row)
        print(json.dumps(row), flush=True)
        plan.close()
        del A, x, y, flags
        torch.cuda.empty_cache()
    return out


def summarize(d, dispatches=None):
    """Summarise rocprofv3 csv output under d: per-kernel dispatch count and
    mean / median duration, and per-kernel mean counter values.  dispatches
    "A:B" keeps each kernel's dispatches A..B (1-based, in start order) --
    e.g. the timed region of a bench run after its warm-up launches."""
    import csv
    import statistics
    lines = []
    lo, hi = (int(x) for x in dispatches.split(":")) if dispatches else (1, None)
    for path in sorted(glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)):
        per = {}
        with open(path) as f:
            recs = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
        for r in recs:
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            per.setdefault(r["Kernel_Name"], []).append(dur)
        per = {k: v[lo - 1:hi] for k, v in per.items() if v[lo - 1:hi]}
        lines.append(f"# kernel trace: {os.path.relpath(path, d)}" + (f" (dispatches {dispatches} of each kernel)" if dispatches else ""))
        lines.append(f"{'kernel':60s} {'calls':>6s} {'mean_us':>10s} {'median_us':>10s} {'min_us':>10s}")
        for k, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
            lines.append(f"{k[:60]:60s} {len(v):6d} {statistics.mean(v):10.2f} {statistics.median(v):10.2f} "
                         f"{min(v):10.2f}")
    for path in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
        per = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                key = (r["Kernel_Name"], r["Counter_Name"])
                per.setdefault(key, []).append(float(r["Counter_Value"]))
        lines.append(f"# counters: {os.path.relpath(path, d)}")
        lines.append(f"{'kernel':60s} {'counter':>12s} {'calls':>6s} {'mean':>14s} {'median':>14s}")
        for (k, c), v in sorted(per.items()):
            lines.append(f"{k[:60]:60s} {c:>12s} {len(v):6d} {statistics.mean(v):14.1f} {statistics.median(v):14.1f}")
    return "\n".join(lines)


def traffic(fetch_dir, write_dir, workload, kernel="fused_pool_kernel", calib="copy_kernel"):
    """HBM bytes per launch of `kernel` from two rocprofv3 counter runs of
    `bench.py --profile` (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch),
    each scaled by what the same counter reads for the plain copy of
    calibration_copy_bytes (1 GiB read + 1 GiB written) in the same run."""
    import csv
    import statistics

    def per_kernel(d, counter):
        vals = {}
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for r in csv.DictReader(f):
                    if r["Counter_Name"] == counter:
                        vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return {k: statistics.median(v) for k, v in vals.items()}

    nb = 1 << 30
    fe, wr = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    kf = next(k for k in fe if k.startswith(kernel))
    cf = next(k for k in fe if k.startswith(calib))
    kw = next(k for k in wr if k.startswith(kernel))
    cw = next(k for k in wr if k.startswith(calib))
    f_scale = (nb / 1024.0) / fe[cf]
    w_scale = (nb / 1024.0) / wr[cw]
    fetch_b = fe[kf] * f_scale * 1024
    write_b = wr[kw] * w_scale * 1024
    return {"workload": workload, "kernel": kernel, "kernel_hash": kernel_hash(kernel),
            "plan_options": PLAN_OPTS.get(workload, {}),
            "fetch_kib_raw": fe[kf], "write_kib_raw": wr[kw], "fetch_scale": round(f_scale, 4),
            "write_scale": round(w_scale, 4), "fetch_bytes": int(fetch_b), "write_bytes": int(write_b),
            "hbm_bytes_per_launch": int(fetch_b + write_b)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="one workload (default: the large workload's line, with the other four in it)")
    ap.add_argument("--all", action="store_true", help="every workload, one JSON line each")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile", action="store_true", help="timing loops only (for rocprofv3 runs)")
    ap.add_argument("--summarize", metavar="DIR")
    ap.add_argument("--dispatches", metavar="A:B", help="with --summarize: each kernel's dispatches A..B only")
    ap.add_argument("--traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--occupancy", action="store_true", help="persistent-grid occupancy sweep of the fused kernel")
    ap.add_argument("--timeline", action="store_true", help="per-slice release / drain times, both slice orders")
    ap.add_argument("--mean", action="store_true", help="mean pooling (the same bags without weights)")
    ap.add_argument("--row-probe", action="store_true", help="random-row read rate by row width")
    ap.add_argument("--per-table-slices", action="store_true", help="a ready flag per (slice, table)")
    ap.add_argument("--gemv-ar", action="store_true", help="fused GEMV + AllReduce (Sec. III-B), several shapes")
    ap.add_argument("--gemv-m", type=int, default=0, help="with --gemv-ar: only the shape with this M")
    ap.add_argument("--backward", action="store_true", help="embedding backward fused with the gradient's arrival")
    ap.add_argument("--backward-sweep", action="store_true", help="backward kernel time per launch shape")
    ap.add_argument("--stream-probe", action="store_true", help="streaming read and write ceilings")
    ap.add_argument("--torch-baseline", action="store_true", help="PyTorch's embedding_bag path, for comparison")
    ap.add_argument("--placement", action="store_true",
                    help="fused and unfused time with the send buffer allocated before vs after the tables")
    a = ap.parse_args()
    if a.summarize:
        print(summarize(a.summarize, a.dispatches))
        return 0
    if a.traffic:
        if a.gemv_ar:
            kernel, workload = "gemv_ar_last_arriver_kernel", f"m{a.gemv_m}"
        else:
            kernel, workload = ("backward_kernel" if a.backward else "fused_pool_kernel"), a.workload
        print(json.dumps(traffic(a.traffic[0], a.traffic[1], workload, kernel=kernel), indent=1))
        return 0
    headline = a.workload is None
    a.workload = a.workload or HEADLINE
    if a.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU; --gpus {a.gpus} is not supported (the R destinations "
              "are logical slices of one GPU's send buffer)", file=sys.stderr)
        return 2
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if a.occupancy:
        run_occupancy(a.workload, a.steps, a.warmup)
        return 0
    if a.placement:
        print(json.dumps(run_placement(a.workload, a.steps, a.warmup)), flush=True)
        return 0
    if a.timeline:
        run_timeline(a.workload, a.warmup)
        return 0
    if a.stream_probe:
        run_stream_probe()
        return 0
    if a.torch_baseline:
        for n in (["tiny", "dlrm", "skewed", "large", "mixed"] if a.all else [a.workload]):
            run_torch_baseline(n, a.steps, a.warmup)
        if a.all:
            run_torch_gemv_baseline(a.steps, a.warmup)
        return 0
    if a.row_probe:
        run_row_probe()
        return 0
    if a.backward_sweep:
        for n in (["dlrm", "skewed", "large", "mixed"] if a.all else [a.workload]):
            run_backward_sweep(n, a.steps, a.warmup)
        return 0
    if a.backward:
        for n in (["tiny", "dlrm", "skewed", "large", "mixed"] if a.all else [a.workload]):
            run_backward(n, a.steps, a.warmup, profile=a.profile, with_cpu=not a.no_cpu_baseline)
        return 0
    if a.gemv_ar:
        shapes = [sh for sh in GEMV_SHAPES if a.gemv_m in (0, sh[0])]
        if not shapes:
            print(f"bench.py: no GEMV shape with M={a.gemv_m}", file=sys.stderr)
            return 2
        run_gemv_ar(a.steps, a.warmup, shapes=shapes, with_cpu=not (a.no_cpu_baseline or a.profile), profile=a.profile)
        return 0
    if headline and not (a.all or a.profile or a.mean or a.per_table_slices):
        print(json.dumps(run_headline(a.steps, a.warmup, with_cpu=not a.no_cpu_baseline)), flush=True)
        return 0
    names = ["tiny", "dlrm", "skewed", "large", "mixed"] if a.all else [a.workload]
    for n in names:
        out = run_workload(n, a.steps, a.warmup, with_cpu=(not a.no_cpu_baseline and not a.profile), profile=a.profile,
                           mean=a.mean, per_table=a.per_table_slices,
                           cpu_tables=CPU_TABLES.get(n))
        print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
