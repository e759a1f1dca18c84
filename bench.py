"""Benchmark of the tensor-group hot path on one MI355X.

One step is one pass of the whole path over a ResNet-50 v1 parameter group
(161 tensors, 25,557,032 binary32 elements) with K = 8 worker copies:

  1. pack     the K workers' per-layer gradient tensors -> the K copies'
              group buffer(s)
  2. reduce   AVG over the K gradient copies (the synchronous tensor average)
  3. easgd    fused center reduction + elastic + SGD update of the K worker
              copies and the center (eta = 0.05, rho = 0.9/(K eta))
  4. unpack   the K worker copies -> per-layer parameter tensors

The K copies are held either in the tensor layout (one buffer, copies
interleaved in slots of four elements: tc_pack_tensor, tc_reduce_tensor,
easgd_step_tensor, tc_unpack_tensor), the headline, or as K separate flat
buffers (tc_pack, tc_reduce, easgd_step, tc_unpack), measured in the same
run and reported beside it.  The bytes moved are the same.  The same run
also times the whole step as one launch (easgd_pipeline_tensor: the four
operations with the intermediates kept on chip, 172 instead of 268 bytes
per element at K = 8) and reports it under fused_pipeline.

Inputs are seeded synthetic values resident in HBM before timing starts.
The reported value is the step's algorithmic HBM traffic (every input read
once, every output written once) divided by the measured step time.  Kernel
durations come from HIP events recorded on the stream the kernels run on.
The CPU baseline times the oracle (single thread) on a bounded sample of the
same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--layout tensor|separate] [--no-compare]
"""

from __future__ import annotations

import argparse
import itertools
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s

WORKLOADS = {
    # name -> (workload key in paper_1801_03855_amd.workloads, ops per step, default layout)
    "resnet50_k8_pipeline": ("resnet50_k8_easgd", ("pack", "reduce", "easgd", "unpack"), "tensor"),
    "vgg16_k4_pipeline": ("vgg16_k4_easgd", ("pack", "reduce", "easgd", "unpack"), "tensor"),
    # 10,000 mostly misaligned tensors and K = 16 bfloat16 copies: pack and
    # unpack are faster on separate buffers, the fused step much faster on the
    # tensor layout, and the whole step slightly faster there
    "many_small_k16_bf16_pipeline": ("many_small_k16_bf16", ("pack", "reduce", "easgd", "unpack"), "tensor"),
    # the 8-tensor group at K = 2 (7,392 elements): bound by launch and host
    # overhead, selectable so that a kernel trace can split the two
    "tiny_k2_pipeline": ("tiny_k2", ("pack", "reduce", "easgd", "unpack"), "tensor"),
    # the same steps with the reduction and the step as one call
    # (reduce_easgd_step): three calls per step
    "resnet50_k8_fused": ("resnet50_k8_easgd", ("pack", "reduce_easgd", "unpack"), "tensor"),
    "vgg16_k4_fused": ("vgg16_k4_easgd", ("pack", "reduce_easgd", "unpack"), "tensor"),
    "many_small_k16_bf16_fused": ("many_small_k16_bf16", ("pack", "reduce_easgd", "unpack"), "tensor"),
}
LAYOUTS = ("tensor", "separate")


def op_bytes(op: str, K: int, N: int, s_g: int) -> int:
    """Algorithmic bytes of one op over N elements and K copies."""
    if op == "pack":      # read K gradient copies, write K flat copies
        return 2 * K * N * s_g
    if op == "reduce":    # read K gradient copies, write one binary32 average
        return (K * s_g + 4) * N
    if op == "easgd":     # read+write K workers and the center, read K gradients
        return ((8 + s_g) * K + 8) * N
    if op == "reduce_easgd":  # the step's bytes and the binary32 average written
        return ((8 + s_g) * K + 12) * N
    if op == "unpack":    # read K flat workers, write K per-layer copies
        return 2 * K * N * 4
    raise ValueError(op)



def layer_lists(tc, g, flats, sizes):
    """A model's per-layer tensors for each flat copy: one allocation per
    layer and copy (torch.empty, no kernel), filled from the flat copies by
    one tc_unpack launch for all copies.  (A clone per tensor would issue
    K x n copy kernels: 160,000 for the 10,000-tensor group at K = 16.)"""
    import torch

    lists = [[torch.empty(s, dtype=f.dtype, device=f.device) for s in sizes] for f in flats]
    tc.unpack(tc.TensorList(g, lists), flats)
    return lists

# What defines the kernels measured by the hardware counters: every HIP source
# and header of the library, and the compiler flags it is built with (the
# public header only declares the ABI).
def kernel_sources():
    import glob

    csrc = os.path.join(ROOT, "paper_1801_03855_amd", "csrc")
    files = sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h")))
    return [os.path.relpath(f, ROOT) for f in files]


# C/C++ comments, and string or character literals kept as they are
_COMMENT = re.compile(r'("(?:\\.|[^"\\\n])*"|\'(?:\\.|[^\'\\\n])*\')|//[^\n]*|/\*.*?\*/', re.S)


def strip_comments(text: str) -> str:
    return _COMMENT.sub(lambda m: m.group(1) or "", text)


def kernel_source_sha() -> str:
    """Hash of what the kernels are compiled from: every source with its
    comments removed, and the compiler flags.  Editing a comment leaves it
    unchanged; any change to code or flags changes it."""
    import hashlib

    from paper_1801_03855_amd import build as b

    h = hashlib.sha256()
    for rel in kernel_sources():
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(strip_comments(f.read()).encode())
    h.update(" ".join(b.FLAGS).encode())
    return h.hexdigest()


def recorded_traffic(workload: str, layout: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary of this workload and layout, or {} when there is none
    or the kernels have changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_{layout}_hbm_traffic.md")
    if not os.path.exists(path) and workload.endswith("_fused"):
        # the same group and kernels as the four-call workload, whose counter
        # passes include the fused call
        path = os.path.join(ROOT, "profiles", f"{workload[:-len('_fused')]}_pipeline_{layout}_hbm_traffic.md")
    if not os.path.exists(path):
        return {}
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and (line.startswith("source_sha256") or line.startswith("traffic_bytes_")):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != kernel_source_sha():
        return {}
    return {k[len("traffic_bytes_"):]: int(v) for k, v in vals.items() if k.startswith("traffic_bytes_")}


def host_cpu() -> dict:
    """The host the oracle runs on: CPU model, sockets, logical CPUs, and the
    CPUs this process may use."""
    model, sockets = "unknown", set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key, val = key.strip(), val.strip()
                if key == "model name" and model == "unknown":
                    model = val
                elif key == "physical id":
                    sockets.add(val)
    except OSError:
        pass
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "sockets": len(sockets) or None, "logical_cpus": os.cpu_count(),
            "usable_cpus": usable}


def cpu_baseline(wkey: str, ops, sample_elems: int = 30_000_000, min_seconds: float = 10.0,
                 max_reps: int = 20):
    """The oracle, as it is, on the first tensors of the group (at least
    sample_elems elements or the whole group), single-threaded, repeated
    until min_seconds of CPU work (at most max_reps passes); GB/s of
    algorithmic bytes over all passes."""
    import numpy as np
    import torch

    import oracle
    from paper_1801_03855_amd import workloads as wl

    w = wl.WORKLOADS[wkey]
    sizes = w.sizes()
    sub = []
    for s in sizes:
        sub.append(s)
        if sum(sub) >= sample_elems:
            break
    n = sum(sub)
    orc = oracle.load()
    gflat = wl.make_gradients(w, n, "cpu")
    host_g = [(g.view(torch.int16).numpy().view(np.uint16) if g.dtype == torch.bfloat16 else g.numpy())
              for g in gflat]
    s_g = host_g[0].dtype.itemsize
    g_parts = [orc.unpack(h, sub) for h in host_g]
    xs, xc = wl.make_state(w, n, "cpu")
    x64 = [x.numpy().astype(np.float64) for x in xs]
    c64 = xc.numpy().astype(np.float64)
    t = {o: 0.0 for o in ("pack", "reduce", "easgd", "unpack")}
    reps = 0
    while reps < max_reps and (reps == 0 or sum(t.values()) < min_seconds):
        t0 = time.perf_counter()
        packed = [orc.pack(p) for p in g_parts]
        t["pack"] += time.perf_counter() - t0
        t0 = time.perf_counter()
        orc.reduce(packed, oracle.AVG)
        t["reduce"] += time.perf_counter() - t0
        t0 = time.perf_counter()
        orc.easgd_step(x64, packed, c64, w.eta, w.rho)
        t["easgd"] += time.perf_counter() - t0
        xf = [x.astype(np.float32) for x in x64]
        t0 = time.perf_counter()
        for x in xf:
            orc.unpack(x, sub)
        t["unpack"] += time.perf_counter() - t0
        reps += 1
    t["reduce_easgd"] = t["reduce"] + t["easgd"]  # the oracle defines it as the two
    secs = sum(t[o] for o in ops)
    nbytes = reps * sum(op_bytes(o, w.K, n, s_g) for o in ops)
    out = {"value": round(nbytes / secs / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
           "sample": f"{reps} passes of {'+'.join(ops)} over the first {len(sub)} tensors of the group "
                     f"({n} elements, K={w.K}); binary64 C oracle, 1 thread",
           "seconds": round(secs, 3),
           "steps_per_s": round(reps * n / (secs * sum(sizes)), 4),
           "host": host_cpu()}

    # the same oracle functions on every usable host CPU: the flat range is
    # cut into one contiguous block per thread, inside tensors where a cut
    # falls there, and each thread takes its block's pieces through the four
    # operations (the operations are elementwise, so no two threads share an
    # element and every element is computed as in the single-thread pass)
    from concurrent.futures import ThreadPoolExecutor

    threads = max(1, out["host"]["usable_cpus"] or 1)
    offs = np.cumsum([0] + sub)
    cuts = [n * j // threads for j in range(threads + 1)]

    def pieces(lo, hi):
        """(tensor, start, stop) of every tensor piece inside [lo, hi)."""
        t0, t1 = int(np.searchsorted(offs, lo, "right")) - 1, int(np.searchsorted(offs, hi, "left"))
        return [(t, max(lo, int(offs[t])) - int(offs[t]), min(hi, int(offs[t + 1])) - int(offs[t]))
                for t in range(t0, t1) if min(hi, int(offs[t + 1])) > max(lo, int(offs[t]))]

    blocks = [(lo, hi, pieces(lo, hi)) for lo, hi in zip(cuts[:-1], cuts[1:]) if hi > lo]

    def block_pass(lo, hi, pcs):
        packed = [orc.pack([p[t][a:b] for t, a, b in pcs]) for p in g_parts]
        orc.reduce(packed, oracle.AVG)
        xb = [x[lo:hi] for x in x64]
        orc.easgd_step(xb, packed, c64[lo:hi], w.eta, w.rho)
        for x in xb:
            orc.unpack(x.astype(np.float32), [b - a for _, a, b in pcs])

    with ThreadPoolExecutor(max_workers=len(blocks)) as pool:
        preps, t0 = 0, time.perf_counter()
        while preps < max_reps and (preps == 0 or time.perf_counter() - t0 < min_seconds / 2):
            list(pool.map(lambda blk: block_pass(*blk), blocks))
            preps += 1
        psecs = time.perf_counter() - t0
    out["parallel"] = {"value": round(preps * sum(op_bytes(o, w.K, n, s_g) for o in ops) / psecs / 1e9, 3),
                       "unit": "GB/s", "cores": len(blocks), "kind": "oracle",
                       "sample": f"{preps} passes of the same sample, {len(blocks)} threads (every usable CPU), "
                                 f"each taking one contiguous block of the flat range (cut inside tensors where "
                                 f"a cut falls there) through {'+'.join(ops)}",
                       "seconds": round(psecs, 3)}
    return out


def run_pipeline(tc, wl, w, sizes, g, ops, layout, steps, warmup, name):
    """Set up one layout's buffers, warm up, time `steps` steps; returns the
    average step and per-op times (ms) from HIP events on the stream."""
    import torch

    N, K = g.numel, w.K
    dev = "cuda"
    gdt = torch.bfloat16 if w.g_dtype == "bf16" else torch.float32
    print(f"# setup {name} ({layout} layout): n={len(sizes)} N={N} K={K}", file=sys.stderr, flush=True)
    g_tensors = layer_lists(tc, g, wl.make_gradients(w, N, dev), sizes)
    g_tl = tc.TensorList(g, g_tensors)
    xs, xc = wl.make_state(w, N, dev)
    gbar = torch.empty(N, dtype=torch.float32, device=dev)
    x_tensors = [[torch.empty(s, dtype=torch.float32, device=dev) for s in sizes] for _ in range(K)]
    x_tl = tc.TensorList(g, x_tensors)
    stream = torch.cuda.current_stream()
    if layout == "tensor":
        G = torch.empty(tc.tensor_numel(g, K), dtype=gdt, device=dev)
        X = torch.empty(tc.tensor_numel(g, K), dtype=torch.float32, device=dev)
        tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X, stream)
        del xs

        def run_op(op):
            if op == "pack":
                tc.pack_tensor(g_tl, G, stream)
            elif op == "reduce":
                tc.reduce_tensor(g, K, G, gbar, "avg", stream)
            elif op == "easgd":
                tc.easgd_step_tensor(g, K, X, G, xc, w.eta, w.rho, stream)
            elif op == "reduce_easgd":
                tc.reduce_easgd_step_tensor(g, K, X, G, xc, gbar, w.eta, w.rho, "avg", stream)
            elif op == "unpack":
                tc.unpack_tensor(x_tl, X, stream)
    else:
        gflat = [torch.empty(N, dtype=gdt, device=dev) for _ in range(K)]

        def run_op(op):
            if op == "pack":
                tc.pack(g_tl, gflat, stream)
            elif op == "reduce":
                tc.reduce(g, gflat, gbar, "avg", stream)
            elif op == "easgd":
                tc.easgd_step(g, xs, gflat, xc, w.eta, w.rho, stream)
            elif op == "reduce_easgd":
                tc.reduce_easgd_step(g, xs, gflat, xc, gbar, w.eta, w.rho, "avg", stream)
            elif op == "unpack":
                tc.unpack(x_tl, xs, stream)

    for _ in range(warmup):
        for op in ops:
            run_op(op)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        ev[s][0].record(stream)
        for i, op in enumerate(ops):
            run_op(op)
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    print(f"# {layout}: timed {steps} steps in {time.perf_counter() - t0:.3f} s", file=sys.stderr, flush=True)
    per_op_ms = {op: sum(ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(steps)) / steps
                 for i, op in enumerate(ops)}
    step_list = sorted(ev[s][0].elapsed_time(ev[s][len(ops)]) for s in range(steps))
    step_ms = sum(step_list) / steps
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return {"step_ms": step_ms, "per_op_ms": per_op_ms, "step_ms_median": step_list[steps // 2],
            "step_ms_min": step_list[0]}


def copy_ceiling(tc, reps: int = 20) -> dict:
    """Plain device-to-device copies of 1 GiB (read + write bytes over the
    time): torch's copy_ and the library's 16-byte vector copy (tc_broadcast
    into one copy); the faster is what this machine's HBM gives the simplest
    stream."""
    import torch

    src = torch.ones(256 << 20, device="cuda")
    dst = torch.empty_like(src)
    one = tc.Group([src.numel()])
    out = {}
    for name, fn in (("torch copy_", lambda: dst.copy_(src)), ("tc_broadcast, K = 1", lambda: tc.broadcast(one, src, [dst]))):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name] = round(2 * (1 << 30) / (a.elapsed_time(b) / reps * 1e-3) / 1e9, 1)
    del src, dst
    torch.cuda.empty_cache()
    best = max(out, key=out.get)
    return {"GB/s": out[best], "by": best, "all": out, "what": "1 GiB device-to-device copy, read + write bytes"}


def fused_bytes(K: int, N: int, s_g: int, write_g: bool = True) -> int:
    """Algorithmic bytes of the one-pass pipeline: read the K gradient
    lists, the K workers and the center; write the packed gradients (when
    asked), the AVG, the K workers, the center and the K parameter lists."""
    return ((2 * s_g if write_g else s_g) + 12) * K * N + 12 * N


def run_fused(tc, wl, w, sizes, g, steps, warmup):
    """The whole step as one easgd_pipeline_tensor launch, with and without
    writing the packed gradients; average step times (ms) from HIP events on
    the stream."""
    import torch

    N, K = g.numel, w.K
    dev = "cuda"
    gdt = torch.bfloat16 if w.g_dtype == "bf16" else torch.float32
    print(f"# setup one-pass pipeline: n={len(sizes)} N={N} K={K}", file=sys.stderr, flush=True)
    grads = tc.TensorList(g, layer_lists(tc, g, wl.make_gradients(w, N, dev), sizes))
    xs, xc = wl.make_state(w, N, dev)
    X = torch.empty(tc.tensor_numel(g, K), dtype=torch.float32, device=dev)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    del xs
    G = torch.empty(tc.tensor_numel(g, K), dtype=gdt, device=dev)
    gbar = torch.empty(N, dtype=torch.float32, device=dev)
    params = tc.TensorList(g, [[torch.empty(s, dtype=torch.float32, device=dev) for s in sizes] for _ in range(K)])
    stream = torch.cuda.current_stream()
    out = {}
    for write_g in (True, False):
        gt = G if write_g else None
        for _ in range(warmup):
            tc.easgd_pipeline_tensor(grads, params, gt, gbar, X, xc, w.eta, w.rho, stream)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(steps):
            tc.easgd_pipeline_tensor(grads, params, gt, gbar, X, xc, w.eta, w.rho, stream)
        b.record(stream)
        torch.cuda.synchronize()
        out[write_g] = a.elapsed_time(b) / steps
    del grads, X, G, gbar, params, xc
    torch.cuda.empty_cache()
    return out


def run_reduce_easgd(tc, wl, w, sizes, g, steps, warmup):
    """The AVG reduction and the step on both layouts, as two calls
    (tc_reduce + easgd_step) and as one (reduce_easgd_step); average times
    (ms) from HIP events on the stream, over `steps` back-to-back pairs or
    calls."""
    import torch

    N, K = g.numel, w.K
    dev = "cuda"
    print(f"# setup reduction fused with the step: N={N} K={K}", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    gs = wl.make_gradients(w, N, dev)
    xs, xc = wl.make_state(w, N, dev)
    gbar = torch.empty(N, dtype=torch.float32, device=dev)
    X = torch.empty(tc.tensor_numel(g, K), dtype=torch.float32, device=dev)
    G = torch.empty(tc.tensor_numel(g, K), dtype=gs[0].dtype, device=dev)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in gs]), G)
    calls = {
        "separate": (lambda: (tc.reduce(g, gs, gbar, "avg", stream),
                              tc.easgd_step(g, xs, gs, xc, w.eta, w.rho, stream)),
                     lambda: tc.reduce_easgd_step(g, xs, gs, xc, gbar, w.eta, w.rho, "avg", stream)),
        "tensor": (lambda: (tc.reduce_tensor(g, K, G, gbar, "avg", stream),
                            tc.easgd_step_tensor(g, K, X, G, xc, w.eta, w.rho, stream)),
                   lambda: tc.reduce_easgd_step_tensor(g, K, X, G, xc, gbar, w.eta, w.rho, "avg", stream)),
    }
    out = {}
    for lay, fns in calls.items():
        out[lay] = []
        for fn in fns:
            for _ in range(warmup):
                fn()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            for _ in range(steps):
                fn()
            b.record(stream)
            torch.cuda.synchronize()
            out[lay].append(a.elapsed_time(b) / steps)
    del gs, xs, xc, gbar, X, G
    torch.cuda.empty_cache()
    return out


def _time_launches(fns, reps, flush=None):
    """Median and minimum time (ms) of single launches, cycling through the
    callables in fns (one per input set), from HIP events on the stream;
    flush, when given, runs before each launch, outside the timed interval."""
    import torch

    stream = torch.cuda.current_stream()
    for f in fns:
        f()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda.synchronize()
    for r in range(reps):
        if flush is not None:
            flush()
        ev[r][0].record(stream)
        fns[r % len(fns)]()
        ev[r][1].record(stream)
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) for a, b in ev)
    return t[reps // 2], t[0]


def tensorlist_rows(tc, wl, reps=5):
    """Host cost of describing K per-layer tensor lists to the library
    (tc_tensorlist_create: argument checks, a hipMalloc of the K*n-pointer
    table and a synchronous upload), which a caller whose per-layer tensors
    move between steps would pay once per step: the raw C call on a
    prepared pointer array, median of reps, and the matching destroy."""
    import ctypes

    import torch

    out = {}
    L = tc.lib()
    for wkey in ("resnet50_k8_easgd", "many_small_k16_bf16"):
        w = wl.WORKLOADS[wkey]
        sizes = w.sizes()
        g = tc.Group(sizes)
        dt = torch.bfloat16 if w.g_dtype == "bf16" else torch.float32
        flats = [torch.empty(g.numel, dtype=dt, device="cuda") for _ in range(w.K)]
        lists = [wl.split_views(f, sizes) for f in flats]
        ptrs = tc._ptr_array([t.data_ptr() if t.numel() else 0 for c in lists for t in c])
        code = tc.TC_BF16 if dt == torch.bfloat16 else tc.TC_F32
        times = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            h = L.tc_tensorlist_create(g.handle, w.K, ptrs, code)
            t1 = time.perf_counter()
            if not h:
                raise RuntimeError(tc.last_error())
            L.tc_tensorlist_destroy(h)
            times.append(t1 - t0)
        times.sort()
        out[wkey] = {"pointers": w.K * len(sizes), "create_ms_median": round(times[reps // 2] * 1e3, 4),
                     "create_ms_min": round(times[0] * 1e3, 4)}
        del flats, lists
    torch.cuda.empty_cache()
    return out


def graph_step_rows(tc, wl, reps=200):
    """The tiny group's whole step (pack, AVG, fused step, unpack on the
    tensor layout; and the same as one easgd_pipeline_tensor launch), timed
    over reps back-to-back steps: issued eagerly, and replayed from a HIP
    graph captured once.  A group this small is bound by launch and
    host-call overhead, which the graph removes."""
    import torch

    w = wl.WORKLOADS["tiny_k2"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K, dev = g.numel, w.K, "cuda"
    gs = wl.make_gradients(w, N, dev)
    xs, xc = wl.make_state(w, N, dev)
    grads = tc.TensorList(g, layer_lists(tc, g, gs, sizes))
    params = tc.TensorList(g, [[torch.empty(n, device=dev) for n in sizes] for _ in range(K)])
    X = torch.zeros(tc.tensor_numel(g, K), device=dev)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    G = torch.zeros(tc.tensor_numel(g, K), device=dev)
    gbar = torch.empty(N, device=dev)

    def four(s):
        tc.pack_tensor(grads, G, s)
        tc.reduce_tensor(g, K, G, gbar, "avg", s)
        tc.easgd_step_tensor(g, K, X, G, xc, w.eta, w.rho, s)
        tc.unpack_tensor(params, X, s)

    def one(s):
        tc.easgd_pipeline_tensor(grads, params, G, gbar, X, xc, w.eta, w.rho, s)

    def per_step(fn):
        stream = torch.cuda.current_stream()
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out = {"workload": "tiny group, K = 2, tensor layout", "N": N, "K": K}
    for name, step in (("four calls", four), ("one launch", one)):
        eager = per_step(lambda: step(torch.cuda.current_stream()))
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            step(side)
        torch.cuda.synchronize()
        replay = per_step(graph.replay)
        out[name] = {"eager_ms": round(eager, 5), "graph_ms": round(replay, 5),
                     "eager_steps_per_s": round(1e3 / eager, 1), "graph_steps_per_s": round(1e3 / replay, 1)}
        del graph
    torch.cuda.synchronize()
    return out


def config_table(tc, wl, reps=20):
    """Every configured workload's operations on both layouts: median and
    minimum time of single launches, algorithmic GB/s at the median and its
    fraction of peak.  The ResNet-50 K = 4 reduction (511 MB per call, about
    twice the 256 MB last-level cache) is also timed cold: two sets of inputs
    and output in turn, and before each call a 1 GiB copy with cacheable
    loads and stores (outside the timed interval), so that no call finds its
    inputs or its output left in that cache (non-temporal reads alone do not
    evict an output written with cache-retaining stores); the tiny group is
    launch-bound, so only its times mean anything there."""
    import torch

    dev = "cuda"
    out = {}

    def row(nbytes, fns, flush=None):
        med, mn = _time_launches(fns, reps, flush)
        gbs = nbytes / (med * 1e-3) / 1e9
        return {"ms_median": round(med, 5), "ms_min": round(mn, 5), "per_s": round(1e3 / med, 1),
                "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}

    for wkey in ("tiny_k2", "resnet50_k4_reduce", "resnet50_k8_easgd", "vgg16_k4_easgd", "many_small_k16_bf16"):
        w = wl.WORKLOADS[wkey]
        sizes = w.sizes()
        g = tc.Group(sizes)
        N, K = g.numel, w.K
        s_g = 2 if w.g_dtype == "bf16" else 4
        print(f"# config {wkey}", file=sys.stderr, flush=True)
        sets = 2 if wkey == "resnet50_k4_reduce" else 1
        gsep = [wl.make_gradients(w, N, dev, seed_offset=k) for k in range(sets)]
        gten = []
        for gs in gsep:
            G = torch.empty(tc.tensor_numel(g, K), dtype=gs[0].dtype, device=dev)
            tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in gs]), G)
            gten.append(G)
        avg = torch.empty(N, device=dev)
        avgs = [avg] + [torch.empty(N, device=dev) for _ in range(sets - 1)]
        if sets > 1:
            fl = (torch.empty(1 << 28, device=dev), torch.empty(1 << 28, device=dev))

            def flush(fl=fl):
                fl[1].copy_(fl[0])
        r = {"N": N, "K": K}
        for op in [o for o in ("reduce_sum", "reduce_avg") if o in w.ops]:
            kind = op.split("_")[1]
            nb = op_bytes("reduce", K, N, s_g)
            r[f"{op} separate"] = row(nb, [lambda gs=gs: tc.reduce(g, gs, avg, kind) for gs in gsep[:1]])
            r[f"{op} tensor"] = row(nb, [lambda G=G: tc.reduce_tensor(g, K, G, avg, kind) for G in gten[:1]])
            if sets > 1:
                r[f"{op} separate, cold"] = row(nb, [lambda gs=gs, o=o: tc.reduce(g, gs, o, kind)
                                                     for gs, o in zip(gsep, avgs)], flush)
                r[f"{op} tensor, cold"] = row(nb, [lambda G=G, o=o: tc.reduce_tensor(g, K, G, o, kind)
                                                   for G, o in zip(gten, avgs)], flush)
        if "easgd" in w.ops:
            xs, xc = wl.make_state(w, N, dev)
            X = torch.empty(tc.tensor_numel(g, K), device=dev)
            tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
            xc2 = xc.clone()
            nb = op_bytes("easgd", K, N, s_g)
            r["easgd separate"] = row(nb, [lambda: tc.easgd_step(g, xs, gsep[0], xc, w.eta, w.rho)])
            r["easgd tensor"] = row(nb, [lambda: tc.easgd_step_tensor(g, K, X, gten[0], xc2, w.eta, w.rho)])
            nb = op_bytes("reduce_easgd", K, N, s_g)
            r["reduce_avg + easgd, one call, separate"] = row(
                nb, [lambda: tc.reduce_easgd_step(g, xs, gsep[0], xc, avg, w.eta, w.rho, "avg")])
            r["reduce_avg + easgd, one call, tensor"] = row(
                nb, [lambda: tc.reduce_easgd_step_tensor(g, K, X, gten[0], xc2, avg, w.eta, w.rho, "avg")])
            if "pack" in w.ops:
                grads = tc.TensorList(g, layer_lists(tc, g, gsep[0], sizes))
                params = tc.TensorList(g, [[torch.empty(n, device=dev) for n in sizes] for _ in range(K)])
                r["pipeline (easgd_pipeline_tensor)"] = row(
                    fused_bytes(K, N, s_g), [lambda: tc.easgd_pipeline_tensor(grads, params, gten[0], avg, X, xc2,
                                                                              w.eta, w.rho)])
                del grads, params
            del xs, xc, X, xc2
        out[wkey] = r
        del gsep, gten, avg, avgs
        fl = flush = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def next_rows(tc, wl, steps=20):
    """Per-op bandwidth of the schedule and synchronous-SGD operations on the
    ResNet-50 group, K = 8, binary32, both layouts (HIP events on the
    stream; algorithmic bytes as in op_bytes)."""
    import torch

    w = wl.WORKLOADS["resnet50_k8_easgd"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K, dev = g.numel, w.K, "cuda"
    stream = torch.cuda.current_stream()
    order = list(range(K))
    xs, xc = wl.make_state(w, N, dev)
    gs = wl.make_gradients(w, N, dev)
    # The broadcast rotates over sources totalling more than three times the
    # 256 MB last-level cache: its kernel reads the source with cacheable
    # loads, so a source reused call after call would be served from that
    # cache and not from HBM.
    n_src = -(-3 * (256 << 20) // (4 * N)) + 1
    srcs = [torch.randn(N, device=dev) for _ in range(n_src)]
    rot = {"separate": itertools.cycle(srcs), "tensor": itertools.cycle(srcs)}
    dsts = [torch.empty(N, device=dev) for _ in range(K)]
    X = torch.empty(tc.tensor_numel(g, K), device=dev)
    G = torch.empty(tc.tensor_numel(g, K), device=dev)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X, stream)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in gs]), G, stream)
    bytes_ = {"sgd": 12 * K * N, "elastic_async": (8 * K + 8) * N, "sync_sgd_broadcast": 16 * K * N,
              "broadcast": (4 + 4 * K) * N}
    ops = {
        "separate": {
            "sgd": lambda: tc.sgd_step(g, xs, gs, 1e-6, stream),
            "elastic_async": lambda: tc.elastic_async(g, xs, xc, order, 0.1125, stream),
            "sync_sgd_broadcast": lambda: tc.sync_sgd_step(g, xs, gs, 1e-6, 1.0, True, stream),
            "broadcast": lambda: tc.broadcast(g, next(rot["separate"]), dsts, stream),
        },
        "tensor": {
            "sgd": lambda: tc.sgd_step_tensor(g, K, X, G, 1e-6, stream),
            "elastic_async": lambda: tc.elastic_async_tensor(g, K, X, xc, order, 0.1125, stream),
            "sync_sgd_broadcast": lambda: tc.sync_sgd_step_tensor(g, K, X, G, 1e-6, 1.0, True, stream),
            "broadcast": lambda: tc.broadcast_tensor(g, K, next(rot["tensor"]), X, stream),
        },
    }
    out = {}
    for lay, table in ops.items():
        out[lay] = {}
        for name, fn in table.items():
            for _ in range(3):
                fn()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            for _ in range(steps):
                fn()
            b.record(stream)
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / steps
            gbs = bytes_[name] / (ms * 1e-3) / 1e9
            out[lay][name] = {"ms": round(ms, 5), "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
    # the periodic schedule (tau = 64): 63 SGD steps and one elastic step
    for lay in out:
        out[lay]["easgd_period_tau64_bytes_per_iter"] = round((63 * bytes_["sgd"] + 104 * N) / 64)
    del xs, gs, X, G, dsts, srcs
    torch.cuda.empty_cache()
    return {"workload": "ResNet-50 group, K=8, binary32", "ops": out,
            "broadcast_sources": f"{n_src} sources of {4 * N} bytes, used in turn (no source cached between calls)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="resnet50_k8_pipeline", choices=sorted(WORKLOADS))
    ap.add_argument("--layout", default=None, choices=LAYOUTS,
                    help="how the K copies are held: one interleaved buffer (tensor) or K buffers "
                         "(default: the workload's faster one)")
    ap.add_argument("--no-compare", action="store_true", help="skip the other layout")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fused", action="store_true",
                    help="skip timing the one-pass pipeline (easgd_pipeline_tensor) and the reduction "
                         "fused with the step (reduce_easgd_step)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip timing every configured workload's operations")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip timing the schedule and synchronous-SGD operations")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="only run one plain device copy of 1 GiB (read 1 GiB, write 1 GiB), the known "
                         "reference for scaling hardware byte counters, and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library models the K workers as K resident copies "
              f"in one GPU's memory and has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibration_copy:
        src = torch.ones(256 << 20, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.add(src, 0.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes_read": src.numel() * 4,
                          "calibration_copy_bytes_written": dst.numel() * 4}))
        return

    import paper_1801_03855_amd as tc
    from paper_1801_03855_amd import workloads as wl

    wkey, ops, default_layout = WORKLOADS[args.workload]
    w = wl.WORKLOADS[wkey]
    torch.cuda.set_device(0)
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    s_g = 2 if w.g_dtype == "bf16" else 4

    first = args.layout or default_layout
    results = {first: run_pipeline(tc, wl, w, sizes, g, ops, first, args.steps, args.warmup, args.workload)}
    if not args.no_compare:
        other = [l for l in LAYOUTS if l != first][0]
        results[other] = run_pipeline(tc, wl, w, sizes, g, ops, other, args.steps, args.warmup, args.workload)
    step_ms = results[first]["step_ms"]
    per_op_ms = results[first]["per_op_ms"]
    step_bytes = sum(op_bytes(op, K, N, s_g) for op in ops)
    value = step_bytes / (step_ms * 1e-3) / 1e9

    def kernel_table(pm):
        out = {}
        for op in ops:
            b = op_bytes(op, K, N, s_g)
            gbs = b / (pm[op] * 1e-3) / 1e9
            out[op] = {"ms": round(pm[op], 5), "bytes": b, "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
        return out

    kernels = kernel_table(per_op_ms)
    dom = next((o for o in ("easgd", "reduce_easgd") if o in ops), None)
    dom = dom or max(ops, key=lambda o: per_op_ms[o])
    traffic = recorded_traffic(args.workload, first).get(dom)
    roof = {"bound": "hbm", "kernel": f"{dom} ({first} layout)", "achieved": kernels[dom]["GB/s"],
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": kernels[dom]["frac"], "traffic": traffic,
            "algorithmic_bytes": kernels[dom]["bytes"], "avg_ms": kernels[dom]["ms"]}
    copy = copy_ceiling(tc)
    roof["copy_ceiling"] = copy
    roof["frac_of_copy_ceiling"] = round(kernels[dom]["GB/s"] / copy["GB/s"], 4)
    layouts = {}
    for lay, r in results.items():
        layouts[lay] = {"value": round(step_bytes / (r["step_ms"] * 1e-3) / 1e9, 2), "ms_per_step": round(r["step_ms"], 5),
                        "kernels": kernel_table(r["per_op_ms"])}

    fused = None
    if not args.no_fused and set(ops) == {"pack", "reduce", "easgd", "unpack"}:
        ft = run_fused(tc, wl, w, sizes, g, args.steps, args.warmup)
        # against the faster of the measured layouts' four calls
        four_lay = min(results, key=lambda l: results[l]["step_ms"])
        four_ms = results[four_lay]["step_ms"]
        fused = {"entry_point": "easgd_pipeline_tensor", "layout": "tensor", "four_calls_compared": four_lay}
        for write_g, key in ((True, "with_packed_gradients"), (False, "without_packed_gradients")):
            b = fused_bytes(K, N, s_g, write_g)
            gbs = b / (ft[write_g] * 1e-3) / 1e9
            fused[key] = {"ms_per_step": round(ft[write_g], 5), "steps_per_s": round(1e3 / ft[write_g], 2),
                          "algorithmic_bytes": b, "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                          "speedup_vs_four_calls": round(four_ms / ft[write_g], 3),
                          "traffic": recorded_traffic(args.workload, "tensor").get(
                              "pipeline" if write_g else "pipeline_no_g")}

    fused_re = None
    if not args.no_fused and {"reduce", "easgd"} <= set(ops):
        rt = run_reduce_easgd(tc, wl, w, sizes, g, args.steps, args.warmup)
        b = op_bytes("reduce_easgd", K, N, s_g)
        fused_re = {"entry_points": {"separate": "reduce_easgd_step", "tensor": "reduce_easgd_step_tensor"},
                    "op": "avg", "algorithmic_bytes": b}
        for lay, (two_ms, one_ms) in rt.items():
            gbs = b / (one_ms * 1e-3) / 1e9
            fused_re[lay] = {"ms": round(one_ms, 5), "per_s": round(1e3 / one_ms, 1), "GB/s": round(gbs, 1),
                             "frac": round(gbs / HBM_PEAK_GBS, 4), "two_calls_ms": round(two_ms, 5),
                             "speedup_vs_two_calls": round(two_ms / one_ms, 3),
                             "traffic": recorded_traffic(args.workload, lay).get("reduce_easgd")}

    configs = None
    if not args.no_configs:
        configs = config_table(tc, wl)
        configs["tiny_k2"]["whole step, eager and HIP graph"] = graph_step_rows(tc, wl)
        configs["tensor_list_create"] = tensorlist_rows(tc, wl)

    extra = None
    if not args.no_next_rows and args.workload == "resnet50_k8_pipeline":
        print("# schedule and synchronous-SGD operations", file=sys.stderr, flush=True)
        extra = next_rows(tc, wl)

    cpu = None
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle, 1 thread)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wkey, ops)

    out = {
        "metric": "effective HBM GB/s and reduce+EASGD steps/sec vs HBM roofline, 1 GPU",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 5),
        "ms_per_step_median": round(results[first]["step_ms_median"], 5),
        "ms_per_step_min": round(results[first]["step_ms_min"], 5),
        "steps_per_s": round(1e3 / step_ms, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if s_g == 4 else "f32 (bf16 gradients)",
        "data": "synthetic (seeded; group shapes only, no weights or datasets)",
        "config": {"workload": args.workload, "group": w.group, "n_tensors": len(sizes), "N": N, "K": K,
                   "layout": first, "ops": list(ops), "eta": w.eta, "rho": w.rho, "step_bytes": step_bytes},
        "kernels": kernels,
        "layouts": layouts,
        "roofline": roof,
        "fused_pipeline": fused,
        "fused_reduce_easgd": fused_re,
        "configs": configs,
        "next_rows": extra,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
