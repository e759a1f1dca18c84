"""Buffers of 4 GiB and more: every kernel switches from 32-bit byte offsets to
64-bit indices there.  Separate buffers of 2^30 + 1000 binary32 elements, and
a tensor layout of K = 4 copies of 2^28 + 10 elements (a ragged last slot),
through reduce, the fused step, the reduction fused with the step,
pack/unpack and the one-launch pipeline.  Sampled positions (random, around
element 2^30 and byte 2^32 of each buffer, and the last ones) are checked
against the oracle; pack/unpack, the fused reduction and step, and the
pipeline bit for bit against their definitions and the separate calls.
About 40 GB of device memory in total.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_1801_03855_amd as tc
from paper_1801_03855_amd import workloads as wl
from tests.helpers import assert_close, easgd_mags, host_f32, reduce_mag

pytestmark = pytest.mark.gpu

DEV = "cuda"
ETA, RHO = 0.05, 2.25


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _samples(n, seed, marks):
    rng = np.random.default_rng(seed)
    near = [np.arange(max(0, m - 8), min(n, m + 8)) for m in marks]
    return np.unique(np.concatenate([rng.integers(0, n, 200_000), np.arange(n - 64, n), *near]))


def _randn(n, gen, scale):
    return torch.randn(n, generator=gen, device=DEV).mul_(scale)


def test_separate_buffers_beyond_4gib(orc):
    K, N = 2, (1 << 30) + 1000
    sizes = [(1 << 29) + 4, N - (1 << 29) - 4]
    g = tc.Group(sizes)
    gen = torch.Generator(device=DEV).manual_seed(11)
    gs = [_randn(N, gen, 0.01) for _ in range(K)]
    xs = [_randn(N, gen, 0.05) for _ in range(K)]
    xc = _randn(N, gen, 0.05)
    idx = _samples(N, 12, [1 << 30, (1 << 29) + 4])
    ti = torch.from_numpy(idx).to(DEV)
    h_g = [host_f32(t[ti]) for t in gs]
    h_x = [host_f32(t[ti]) for t in xs]
    h_c = host_f32(xc[ti])
    xs2, xc2 = [t.clone() for t in xs], xc.clone()
    avg = torch.empty(N, device=DEV)
    tc.reduce(g, gs, avg, "avg")
    tc.easgd_step(g, xs, gs, xc, ETA, RHO)
    # the same as one call, bit for bit
    avg2 = torch.empty(N, device=DEV)
    tc.reduce_easgd_step(g, xs2, gs, xc2, avg2, ETA, RHO, "avg")
    torch.cuda.synchronize()
    assert torch.equal(avg2.view(torch.int32), avg.view(torch.int32))
    assert torch.equal(xc2.view(torch.int32), xc.view(torch.int32))
    for i in range(K):
        assert torch.equal(xs2[i].view(torch.int32), xs[i].view(torch.int32)), i
    del xs2, xc2, avg2
    assert_close(host_f32(avg[ti]), orc.reduce(h_g, oracle.AVG), reduce_mag(h_g, True), "avg beyond 4 GiB")
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, ETA, RHO)
    orc.easgd_step(rx, h_g, rc, ETA, RHO)
    for i in range(K):
        assert_close(host_f32(xs[i][ti]), rx[i], mx[i], f"x[{i}] beyond 4 GiB")
    assert_close(host_f32(xc[ti]), rc, mc, "x_c beyond 4 GiB")
    del avg, xc, xs
    # pack / unpack: per-layer views of one copy into a 4 GiB flat buffer and back
    flat = torch.empty(N, device=DEV)
    tc.pack(tc.TensorList(g, [wl.split_views(gs[0], sizes)]), [flat])
    torch.cuda.synchronize()
    assert torch.equal(flat, gs[0])
    back = torch.empty(N, device=DEV)
    tc.unpack(tc.TensorList(g, [wl.split_views(back, sizes)]), [flat])
    torch.cuda.synchronize()
    assert torch.equal(back, gs[0])


def test_tensor_layout_beyond_4gib(orc):
    K, N = 4, (1 << 28) + 10
    sizes = [1 << 27, (1 << 27) + 10]
    g = tc.Group(sizes)
    assert tc.tensor_numel(g, K) * 4 >= (1 << 32)
    gen = torch.Generator(device=DEV).manual_seed(21)
    gs = [_randn(N, gen, 0.01) for _ in range(K)]
    xs = [_randn(N, gen, 0.05) for _ in range(K)]
    xc = _randn(N, gen, 0.05)
    idx = _samples(N, 22, [1 << 27, (1 << 28) // 4 * 4])
    ti = torch.from_numpy(idx).to(DEV)
    h_g = [host_f32(t[ti]) for t in gs]
    h_x = [host_f32(t[ti]) for t in xs]
    h_c = host_f32(xc[ti])
    X = torch.empty(tc.tensor_numel(g, K), device=DEV)
    G = torch.empty(tc.tensor_numel(g, K), device=DEV)
    grads = tc.TensorList(g, [wl.split_views(t, sizes) for t in gs])
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    del xs
    Xp, xcp = X.clone(), xc.clone()
    Xf, xcf = X.clone(), xc.clone()
    # the four calls
    tc.pack_tensor(grads, G)
    gbar = torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, G, gbar, "avg")
    tc.easgd_step_tensor(g, K, X, G, xc, ETA, RHO)
    outs = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in outs]), X)
    # the reduction and the step as one call, bit for bit
    gbarf = torch.empty(N, device=DEV)
    tc.reduce_easgd_step_tensor(g, K, Xf, G, xcf, gbarf, ETA, RHO, "avg")
    torch.cuda.synchronize()
    assert torch.equal(gbarf.view(torch.int32), gbar.view(torch.int32))
    assert torch.equal(xcf.view(torch.int32), xc.view(torch.int32))
    assert torch.equal(Xf.view(torch.int32), X.view(torch.int32))
    del G, Xf, xcf, gbarf
    # the same step as one launch (packed gradients not written)
    gbarp = torch.empty(N, device=DEV)
    params = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.easgd_pipeline_tensor(grads, tc.TensorList(g, [wl.split_views(t, sizes) for t in params]), None, gbarp,
                             Xp, xcp, ETA, RHO)
    torch.cuda.synchronize()
    assert torch.equal(gbarp, gbar) and torch.equal(xcp, xc) and torch.equal(Xp, X)
    for k in range(K):
        assert torch.equal(params[k], outs[k]), k
    assert_close(host_f32(gbar[ti]), orc.reduce(h_g, oracle.AVG), reduce_mag(h_g, True), "tensor avg beyond 4 GiB")
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, ETA, RHO)
    orc.easgd_step(rx, h_g, rc, ETA, RHO)
    for k in range(K):
        assert_close(host_f32(outs[k][ti]), rx[k], mx[k], f"tensor x[{k}] beyond 4 GiB")
    assert_close(host_f32(xc[ti]), rc, mc, "tensor x_c beyond 4 GiB")
