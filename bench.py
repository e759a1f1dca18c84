"""Benchmark of the tensor-group hot path on one MI355X.

One step is one pass of the whole path over a ResNet-50 v1 parameter group
(161 tensors, 25,557,032 binary32 elements) with K = 8 worker copies:

  1. tc_pack     the K workers' per-layer gradient tensors -> K flat buffers
  2. tc_reduce   AVG of the K flat gradients (the synchronous tensor average)
  3. easgd_step  fused center reduction + elastic + SGD update of the K flat
                 worker copies and the center (eta = 0.05, rho = 0.9/(K eta))
  4. tc_unpack   the K flat worker copies -> per-layer parameter tensors

Inputs are seeded synthetic values resident in HBM before timing starts.
The reported value is the step's algorithmic HBM traffic (every input read
once, every output written once) divided by the measured step time.  Kernel
durations come from HIP events recorded on the stream the kernels run on.
The CPU baseline times the oracle (single thread) on a bounded sample of the
same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s

WORKLOADS = {
    # name -> (workload key in paper_1801_03855_amd.workloads, ops per step)
    "resnet50_k8_pipeline": ("resnet50_k8_easgd", ("pack", "reduce", "easgd", "unpack")),
    "vgg16_k4_pipeline": ("vgg16_k4_easgd", ("pack", "reduce", "easgd", "unpack")),
    "many_small_k16_bf16_pipeline": ("many_small_k16_bf16", ("pack", "reduce", "easgd", "unpack")),
}


def op_bytes(op: str, K: int, N: int, s_g: int) -> int:
    """Algorithmic bytes of one op over N elements and K copies."""
    if op == "pack":      # read K gradient copies, write K flat copies
        return 2 * K * N * s_g
    if op == "reduce":    # read K gradient copies, write one binary32 average
        return (K * s_g + 4) * N
    if op == "easgd":     # read+write K workers and the center, read K gradients
        return ((8 + s_g) * K + 8) * N
    if op == "unpack":    # read K flat workers, write K per-layer copies
        return 2 * K * N * 4
    raise ValueError(op)


# Files whose contents define the kernels measured by the hardware counters.
KERNEL_SOURCES = ("paper_1801_03855_amd/csrc/tc_elementwise.hip", "paper_1801_03855_amd/csrc/tc_pack.hip",
                  "paper_1801_03855_amd/csrc/tc_internal.h", "paper_1801_03855_amd/build.py")


def kernel_source_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary of this workload, or {} when there is none or the
    kernels have changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.md")
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
    secs = sum(t[o] for o in ops)
    nbytes = reps * sum(op_bytes(o, w.K, n, s_g) for o in ops)
    return {"value": round(nbytes / secs / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} passes of {'+'.join(ops)} over the first {len(sub)} tensors of the group "
                      f"({n} elements, K={w.K}); binary64 C oracle, 1 thread",
            "seconds": round(secs, 3),
            "steps_per_s": round(reps * n / (secs * sum(sizes)), 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="resnet50_k8_pipeline", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="only run one plain device copy of 1 GiB (read 1 GiB, write 1 GiB), the known "
                         "reference for scaling hardware byte counters, and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build models the K workers as K resident copies "
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

    wkey, ops = WORKLOADS[args.workload]
    w = wl.WORKLOADS[wkey]
    dev = "cuda"
    torch.cuda.set_device(0)
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    gdt = torch.bfloat16 if w.g_dtype == "bf16" else torch.float32
    s_g = 2 if w.g_dtype == "bf16" else 4

    print(f"# setup {args.workload}: n={len(sizes)} N={N} K={K}", file=sys.stderr, flush=True)
    g_tensors = [wl.separate_tensors(f, sizes) for f in wl.make_gradients(w, N, dev)]
    g_tl = tc.TensorList(g, g_tensors)
    gflat = [torch.empty(N, dtype=gdt, device=dev) for _ in range(K)]
    xs, xc = wl.make_state(w, N, dev)
    gbar = torch.empty(N, dtype=torch.float32, device=dev)
    x_tensors = [[torch.empty(s, dtype=torch.float32, device=dev) for s in sizes] for _ in range(K)]
    x_tl = tc.TensorList(g, x_tensors)
    stream = torch.cuda.current_stream()

    def run_op(op):
        if op == "pack":
            tc.pack(g_tl, gflat, stream)
        elif op == "reduce":
            tc.reduce(g, gflat, gbar, "avg", stream)
        elif op == "easgd":
            tc.easgd_step(g, xs, gflat, xc, w.eta, w.rho, stream)
        elif op == "unpack":
            tc.unpack(x_tl, xs, stream)

    for _ in range(args.warmup):
        for op in ops:
            run_op(op)
    torch.cuda.synchronize()
    print(f"# warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        ev[s][0].record(stream)
        for i, op in enumerate(ops):
            run_op(op)
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print(f"# timed {args.steps} steps in {wall:.3f} s", file=sys.stderr, flush=True)

    per_op_ms = {op: 0.0 for op in ops}
    step_ms = 0.0
    for s in range(args.steps):
        for i, op in enumerate(ops):
            per_op_ms[op] += ev[s][i].elapsed_time(ev[s][i + 1])
        step_ms += ev[s][0].elapsed_time(ev[s][len(ops)])
    per_op_ms = {op: v / args.steps for op, v in per_op_ms.items()}
    step_ms /= args.steps
    step_bytes = sum(op_bytes(op, K, N, s_g) for op in ops)
    value = step_bytes / (step_ms * 1e-3) / 1e9

    kernels = {}
    for op in ops:
        b = op_bytes(op, K, N, s_g)
        gbs = b / (per_op_ms[op] * 1e-3) / 1e9
        kernels[op] = {"ms": round(per_op_ms[op], 5), "bytes": b, "GB/s": round(gbs, 1),
                       "frac": round(gbs / HBM_PEAK_GBS, 4)}
    dom = "easgd" if "easgd" in ops else max(ops, key=lambda o: per_op_ms[o])
    traffic = recorded_traffic(args.workload).get(dom)
    roof = {"bound": "hbm", "kernel": dom, "achieved": kernels[dom]["GB/s"], "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": kernels[dom]["frac"], "traffic": traffic,
            "algorithmic_bytes": kernels[dom]["bytes"], "avg_ms": kernels[dom]["ms"]}

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
        "steps_per_s": round(1e3 / step_ms, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if s_g == 4 else "f32 (bf16 gradients)",
        "data": "synthetic (seeded; group shapes only, no weights or datasets)",
        "config": {"workload": args.workload, "group": w.group, "n_tensors": len(sizes), "N": N, "K": K,
                   "ops": list(ops), "eta": w.eta, "rho": w.rho, "step_bytes": step_bytes},
        "kernels": kernels,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
