"""Full-size VGG-16 group (32 tensors, 138,357,544 binary32 elements), K = 4,
on the tensor layout, in the launch configuration the benchmark times:
tc_pack_tensor of the per-layer gradient lists, tc_reduce_tensor (AVG),
easgd_step_tensor, tc_unpack_tensor into per-layer parameter lists, and the
same step as one easgd_pipeline_tensor launch.

Each tensor-layout buffer holds 4 x 138,357,544 binary32 values (2.2 GB), so
its byte offsets run through [2^31, 2^32): the kernels' 32-bit unsigned
offsets are exercised above the signed range.  Checks:
- every element bit for bit equal to the separate-buffer path (tc_pack,
  tc_reduce, easgd_step, tc_unpack; K = 4 is a power of two, so both sum
  by the same pairwise tree), and the pipeline equal to the four calls;
- the packed tensors against the oracle's index map on windows of slots,
  among them the windows around byte 2^31 of the buffers;
- the AVG, the workers and the center against the oracle on ~4M sampled
  positions, every tensor boundary and the elements around byte 2^31,
  within the guarded tolerance of tests/helpers.py.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_1801_03855_amd as tc
from paper_1801_03855_amd import workloads as wl
from tests.helpers import assert_bits_equal, assert_close, easgd_mags, host_f32, host_stored, reduce_mag

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _as_copies(T, K, N):
    """The K copies held in a tensor-layout buffer, as a (K, N) view-derived
    tensor (slot j of copy i at slot index j*K + i; N is a multiple of 4)."""
    return T.view(N // 4, K, 4).transpose(0, 1).reshape(K, N)


def _windows(N, K, sizes, seed):
    """Flat windows [a, b) with a, b multiples of 4: the start, the end, the
    elements whose tensor-layout bytes lie around 2^31, each tensor boundary,
    and random ones."""
    e31 = (1 << 31) // (4 * K)  # flat element whose copy-0 value sits at byte 2^31
    wins = [(0, 4096), (N - 4096, N), (e31 - 8192, e31 + 8192)]
    off = np.cumsum([0] + sizes)
    for o in off[1:-1]:
        a = max(0, (int(o) - 64) // 4 * 4)
        wins.append((a, min(N, a + 128)))
    rng = np.random.default_rng(seed)
    for a in rng.integers(0, N // 4 - 1024, 64):
        wins.append((4 * int(a), 4 * int(a) + 4096))
    return wins


def test_vgg16_k4_tensor_layout_full_size(orc):
    w = wl.WORKLOADS["vgg16_k4_easgd"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    assert N == 138_357_544 and N % 4 == 0
    tn = tc.tensor_numel(g, K)
    assert tn * 4 > (1 << 31)  # byte offsets beyond the signed 32-bit range

    gflat = wl.make_gradients(w, N, DEV)
    grads = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gflat])
    xs, xc = wl.make_state(w, N, DEV)

    # sampled positions for the oracle, taken before any kernel runs
    e31 = (1 << 31) // (4 * K)
    off = np.cumsum([0] + sizes)
    rng = np.random.default_rng(404)
    idx = np.unique(np.concatenate([
        rng.integers(0, N, 4_000_000),
        np.clip(np.concatenate([off[1:-1] - 2, off[1:-1] - 1, off[1:-1], off[1:-1] + 1]), 0, N - 1),
        np.arange(0, 4096), np.arange(N - 4096, N), np.arange(e31 - 4096, e31 + 4096)]))
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gflat]
    h_c = host_f32(xc[ti])
    wins = _windows(N, K, sizes, 405)
    h_gwin = [[host_stored(f[a:b]) for f in gflat] for a, b in wins]

    # separate buffers: the reference for bit identity
    gsep = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.pack(grads, gsep)
    gbar_s = torch.empty(N, device=DEV)
    tc.reduce(g, gsep, gbar_s, "avg")
    xs_s, xc_s = [t.clone() for t in xs], xc.clone()
    tc.easgd_step(g, xs_s, gsep, xc_s, w.eta, w.rho)
    par_s = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack(tc.TensorList(g, [wl.split_views(p, sizes) for p in par_s]), xs_s)
    torch.cuda.synchronize()
    for k in range(K):
        assert torch.equal(gsep[k], gflat[k]), f"tc_pack copy {k}"
        assert torch.equal(par_s[k], xs_s[k]), f"tc_unpack copy {k}"
    del xs_s, gflat

    # tensor layout, four calls
    X = torch.empty(tn, device=DEV)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    X0 = X.clone()
    G = torch.empty(tn, device=DEV)
    tc.pack_tensor(grads, G)
    gbar_t = torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, G, gbar_t, "avg")
    xc_t = xc.clone()
    tc.easgd_step_tensor(g, K, X, G, xc_t, w.eta, w.rho)
    par_t = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, [wl.split_views(p, sizes) for p in par_t]), X)
    torch.cuda.synchronize()
    assert torch.equal(_as_copies(G, K, N), torch.stack(gsep)), "tc_pack_tensor vs tc_pack"
    assert torch.equal(gbar_t, gbar_s), "tc_reduce_tensor vs tc_reduce"
    assert torch.equal(xc_t, xc_s), "center: easgd_step_tensor vs easgd_step"
    assert torch.equal(_as_copies(X, K, N), torch.stack(par_s)), "workers: easgd_step_tensor vs easgd_step"
    for k in range(K):
        assert torch.equal(par_t[k], par_s[k]), f"tc_unpack_tensor copy {k}"
    del gsep

    # the packed gradients against the oracle's index map, window by window
    for (a, b), hg in zip(wins, h_gwin):
        assert_bits_equal(host_stored(G[a * K:b * K]), orc.tensor_from_copies(hg, fill=0),
                          f"tc_pack_tensor window [{a}, {b})")

    # the same step as one launch
    Gp, gbar_p, xc_p = torch.empty(tn, device=DEV), torch.empty(N, device=DEV), xc.clone()
    par_p = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.easgd_pipeline_tensor(grads, tc.TensorList(g, [wl.split_views(p, sizes) for p in par_p]), Gp, gbar_p, X0,
                             xc_p, w.eta, w.rho)
    torch.cuda.synchronize()
    assert torch.equal(Gp, G), "pipeline: packed gradients"
    assert torch.equal(gbar_p, gbar_t), "pipeline: AVG"
    assert torch.equal(X0, X), "pipeline: workers"
    assert torch.equal(xc_p, xc_t), "pipeline: center"
    for k in range(K):
        assert torch.equal(par_p[k], par_t[k]), f"pipeline: parameters copy {k}"
    del Gp, gbar_p, xc_p, par_p, X0, G, X, grads

    # against the oracle on the sampled positions
    assert_close(host_f32(gbar_t[ti]), orc.reduce(h_g, oracle.AVG), reduce_mag(h_g, True), "vgg16 AVG")
    rx = [v.astype(np.float64) for v in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for k in range(K):
        assert_close(host_f32(par_t[k][ti]), rx[k], mx[k], f"vgg16 params[{k}]")
    assert_close(host_f32(xc_t[ti]), rc, mc, "vgg16 x_c")
