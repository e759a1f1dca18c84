"""The seeded input generators: shapes, determinism and distributions."""

import numpy as np
import torch

from paper_1801_03855_amd import workloads as wl


def test_group_shapes():
    r = wl.group_sizes("resnet50")
    v = wl.group_sizes("vgg16")
    assert (len(r), sum(r), max(r)) == (161, 25_557_032, 2_359_296)
    assert (len(v), sum(v), v[26]) == (32, 138_357_544, 25088 * 4096)
    assert all(s % 4 == 0 for s in r + v)
    m = wl.group_sizes("many_small")
    assert len(m) == 10_000 and min(m) >= 1 and max(m) <= 65536
    assert sum(m) == 59_303_476
    assert sum(s % 4 != 0 for s in m) > 7000  # most flat offsets are not 16-byte aligned


def test_generators_are_seeded():
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    a = wl.make_gradients(w, 1000)
    b = wl.make_gradients(w, 1000)
    assert all(torch.equal(x, y) for x, y in zip(a, b))
    xs, xc = wl.make_state(w, 1000)
    xs2, xc2 = wl.make_state(w, 1000)
    assert torch.equal(xc, xc2) and all(torch.equal(x, y) for x, y in zip(xs, xs2))


def test_distributions():
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    n = 200_000
    gs = wl.make_gradients(w, n)
    assert abs(float(gs[0].std()) - 1e-2) < 2e-4
    xs, xc = wl.make_state(w, n)
    assert abs(float(xs[0].std()) - 0.05) < 1e-3
    mean = sum(x.double() for x in xs) / w.K
    assert abs(float((xc.double() - mean).std()) - 1e-3) < 3e-5
    t = wl.WORKLOADS["tiny_k2"]
    xs, xc = wl.make_state(t, 5000)
    assert float(xs[0].abs().max()) <= 0.1
    assert torch.equal(xc, ((xs[0].double() + xs[1].double()) / 2).float())


def test_bf16_gradients_round_to_nearest_even():
    w = wl.WORKLOADS["many_small_k16_bf16"]
    g = wl.make_gradients(w, 1000)[0]
    assert g.dtype == torch.bfloat16
    codes = g.view(torch.int16).numpy().view(np.uint16)
    back = (codes.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(back, g.float().numpy())


def test_step_hyperparameters():
    assert wl.WORKLOADS["resnet50_k8_easgd"].rho == np.float32(2.25)
    assert wl.WORKLOADS["vgg16_k4_easgd"].rho == np.float32(4.5)
    assert wl.WORKLOADS["many_small_k16_bf16"].rho == np.float32(1.125)
    assert wl.WORKLOADS["tiny_k2"].eta == np.float32(0.1)
