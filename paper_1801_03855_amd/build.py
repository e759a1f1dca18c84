"""Compiles the HIP library (``libtc_amd.so``) for gfx950 with hipcc.

``python -m paper_1801_03855_amd.build`` or ``build()`` from Python.  Extra
``-D`` definitions (kernel tunables) and a different output path may be
given, which is how variant builds for tuning are made without touching the
sources.
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys
from typing import Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libtc_amd.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-fvisibility=hidden",
    # binary32 arithmetic exactly as written: fused multiply-adds only where
    # the source calls fma
    "-ffp-contract=off",
    # no packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def sources() -> list:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(output: str = LIBRARY, defines: Sequence[str] = (), verbose: bool = False) -> str:
    """Compiles every source to an object in parallel (the translation units
    share no device code), then links the shared library."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor

    compile_flags = [f for f in FLAGS if f != "-shared"]
    with tempfile.TemporaryDirectory(prefix="tc_build_") as tmp:
        jobs = []
        for src in sources():
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            jobs.append((obj, [HIPCC, *compile_flags, *[f"-D{d}" for d in defines], "-I", INCLUDE, "-I", CSRC,
                               "-c", src, "-o", obj]))

        def run(cmd):
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.run(cmd, check=True)

        with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1, 8)) as pool:
            for f in [pool.submit(run, cmd) for _, cmd in jobs]:
                f.result()
        run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", output + ".tmp", *[o for o, _ in jobs]])
    os.replace(output + ".tmp", output)
    return output


if __name__ == "__main__":
    out = LIBRARY
    defs = []
    args = sys.argv[1:]
    while args:
        arg = args.pop(0)
        if arg.startswith("-D"):
            defs.append(arg[2:] or args.pop(0))
        elif arg.startswith("-o"):
            out = arg[2:] or args.pop(0)
        else:
            sys.exit(f"usage: python -m paper_1801_03855_amd.build [-D NAME=VALUE ...] [-o OUTPUT.so] (got {arg!r})")
    if not out:
        sys.exit("empty output path")
    print(build(os.path.abspath(out), defs, verbose=True))
