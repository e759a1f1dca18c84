"""Seeded synthetic workloads: tensor-group shapes and input values.

A *tensor group* is the list of a model's per-layer parameter (or gradient)
tensors, in layer order, treated as one flat object; a workload adds the
number K of per-worker copies, the value distributions and the step
hyper-parameters.  ResNet-50 v1 and VGG-16 contribute only the sizes of their
parameter tensors (built from the published architecture rules); no weights,
images or datasets are involved.

This module draws inputs and nothing else.  It holds none of the reduction's
or the update's arithmetic, and it is the one piece of code shared by the GPU
path's tests and benchmark and by the CPU oracle's tests.  (The center
variable of a workload is *initialised* from the workers' mean, as the
workload definitions ask; that is input construction, done here in float64
with plain torch ops, not a step of the method.)
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np
import torch

# --------------------------------------------------------------------------
# Group shapes
# --------------------------------------------------------------------------


def tiny_sizes() -> List[int]:
    """Eight small tensors: a 3x3x16x16 and a 3x3x16x32 convolution, their
    biases / norm vectors and a 32x10 classifier (7,392 elements)."""
    return [64, 3 * 3 * 16 * 16, 16, 16, 3 * 3 * 16 * 32, 32, 32, 32 * 10]


def resnet50_sizes() -> List[int]:
    """ResNet-50 v1 parameter tensors in layer order (161 tensors,
    25,557,032 elements).

    Stem: 7x7 conv 3->64 and its batch-norm scale and shift.  Four stages of
    bottleneck blocks (widths 64, 128, 256, 512; 3, 4, 6, 3 blocks).  A block
    is 1x1 conv (in->w), BN(w), 3x3 conv (w->w), BN(w), 1x1 conv (w->4w),
    BN(4w); the first block of each stage adds a 1x1 projection (in->4w) and
    its BN(4w).  Head: 2048->1000 fully connected weight and bias.
    """
    sizes = [64 * 3 * 7 * 7, 64, 64]
    cin = 64
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(blocks):
            sizes += [width * cin, width, width,
                      width * width * 9, width, width,
                      4 * width * width, 4 * width, 4 * width]
            if b == 0:
                sizes += [4 * width * cin, 4 * width, 4 * width]
            cin = 4 * width
    sizes += [1000 * 2048, 1000]
    return sizes


def vgg16_sizes() -> List[int]:
    """VGG-16 (configuration D) parameter tensors in layer order (32 tensors,
    138,357,544 elements): 13 3x3 convolutions with their biases, then the
    25088->4096, 4096->4096 and 4096->1000 fully connected layers."""
    chans = [64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512]
    sizes: List[int] = []
    cin = 3
    for c in chans:
        sizes += [c * cin * 9, c]
        cin = c
    for fin, fout in ((25088, 4096), (4096, 4096), (4096, 1000)):
        sizes += [fout * fin, fout]
    return sizes


def many_small_sizes(n: int = 10_000, seed: int = 5, max_size: int = 65536) -> List[int]:
    """n sizes drawn log-uniformly from [1, max_size]:
    floor(exp(U * ln(max_size + 1))) clamped to [1, max_size], U ~ U[0, 1)
    from numpy's default_rng(seed)."""
    u = np.random.default_rng(seed).random(n)
    s = np.floor(np.exp(u * math.log(max_size + 1.0)))
    return [int(v) for v in np.clip(s, 1, max_size)]


GROUPS = {
    "tiny": tiny_sizes,
    "resnet50": resnet50_sizes,
    "vgg16": vgg16_sizes,
    "many_small": many_small_sizes,
}


def group_sizes(name: str) -> List[int]:
    return list(GROUPS[name]())


# --------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic configuration.

    x_init: "uniform" -> x ~ U(-x_scale, x_scale); "normal" -> N(0, x_scale).
    center: "mean"  -> x_c = mean_i x_i;  "mean+drift" -> that plus
            N(0, drift) per element.
    eta, rho are given as the binary32 values both implementations receive.
    """

    name: str
    group: str
    K: int
    g_dtype: str              # "f32" or "bf16"
    g_scale: float            # g ~ N(0, g_scale)
    seed: int
    x_init: str = "normal"
    x_scale: float = 0.05
    center: str = "mean+drift"
    drift: float = 1e-3
    eta: Optional[float] = None
    rho: Optional[float] = None
    iterations: int = 1
    ops: tuple = ()

    def sizes(self) -> List[int]:
        return group_sizes(self.group)


def f32(v: float) -> float:
    """Round a Python float to the nearest binary32 value."""
    return float(np.float32(v))


def _rho_for(K: int, eta: float) -> float:
    # rho = 0.9 / (K * eta), formed in double and rounded once to binary32
    return f32(0.9 / (K * eta))


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("tiny_k2", "tiny", K=2, g_dtype="f32", g_scale=0.01, seed=0,
                 x_init="uniform", x_scale=0.1, center="mean",
                 eta=f32(0.1), rho=f32(0.5), ops=("reduce_avg", "easgd")),
        Workload("resnet50_k4_reduce", "resnet50", K=4, g_dtype="f32",
                 g_scale=1e-2, seed=2, ops=("reduce_sum", "reduce_avg")),
        Workload("resnet50_k8_easgd", "resnet50", K=8, g_dtype="f32",
                 g_scale=1e-2, seed=3, eta=f32(0.05), rho=_rho_for(8, 0.05),
                 iterations=100, ops=("easgd",)),
        Workload("vgg16_k4_easgd", "vgg16", K=4, g_dtype="f32", g_scale=1e-2,
                 seed=4, eta=f32(0.05), rho=_rho_for(4, 0.05),
                 ops=("easgd",)),
        Workload("many_small_k16_bf16", "many_small", K=16, g_dtype="bf16",
                 g_scale=1e-2, seed=5, eta=f32(0.05), rho=_rho_for(16, 0.05),
                 ops=("reduce_avg", "easgd", "pack", "unpack")),
    ]
}


# --------------------------------------------------------------------------
# Value generation
# --------------------------------------------------------------------------


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_gradients(w: Workload, n: int, device="cpu", seed_offset: int = 0) -> List[torch.Tensor]:
    """K flat gradient copies of n elements, g ~ N(0, g_scale), stored as
    binary32 or as bfloat16 (each binary32 draw rounded to nearest-even)."""
    gen = _gen(device, 1000 * w.seed + 1 + seed_offset)
    out = []
    for _ in range(w.K):
        g = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
        g.mul_(w.g_scale)
        out.append(g.to(torch.bfloat16) if w.g_dtype == "bf16" else g)
    return out


def make_state(w: Workload, n: int, device="cpu", seed_offset: int = 0):
    """K flat worker copies x_i and the center x_c, all binary32."""
    gen = _gen(device, 1000 * w.seed + 2 + seed_offset)
    xs = []
    for _ in range(w.K):
        if w.x_init == "uniform":
            x = torch.rand(n, generator=gen, device=device, dtype=torch.float32)
            x.mul_(2.0 * w.x_scale).sub_(w.x_scale)
        else:
            x = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
            x.mul_(w.x_scale)
        xs.append(x)
    acc = torch.zeros(n, dtype=torch.float64, device=device)
    for x in xs:
        acc.add_(x.to(torch.float64))
    acc.div_(w.K)
    if w.center == "mean+drift":
        d = torch.randn(n, generator=gen, device=device, dtype=torch.float64)
        acc.add_(d.mul_(w.drift))
    xc = acc.to(torch.float32)
    return xs, xc


def integer_values(n: int, K: int, lim: int, seed: int, device="cpu") -> List[torch.Tensor]:
    """K binary32 copies holding integers drawn uniformly from [-lim, lim]."""
    gen = _gen(device, seed)
    return [torch.randint(-lim, lim + 1, (n,), generator=gen, device=device).to(torch.float32)
            for _ in range(K)]


def split_views(flat: torch.Tensor, sizes: List[int]) -> List[torch.Tensor]:
    """Views of a flat buffer, one per tensor of the group (no copy)."""
    out, at = [], 0
    for s in sizes:
        out.append(flat[at:at + s])
        at += s
    return out


def separate_tensors(flat: torch.Tensor, sizes: List[int]) -> List[torch.Tensor]:
    """Separately allocated tensors holding the group's pieces of a flat
    buffer (each its own allocation, as a model's layer tensors are)."""
    return [v.clone() for v in split_views(flat, sizes)]
