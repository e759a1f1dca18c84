"""Parity of the schedule and synchronous-SGD entry points (plain SGD, the
periodic elastic schedule, the asynchronous per-worker exchange, the
synchronous pushpull SGD step, broadcast) with the CPU oracle, on both
layouts, through the C ABI.  Tolerance as in tests/helpers.py."""

import numpy as np
import pytest
import torch

import paper_1801_03855_amd as tc
from paper_1801_03855_amd import workloads as wl
from tests.helpers import (TOL, assert_bits_equal, assert_close, assert_exact, easgd_mags, host_f32, host_stored,
                           widened)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _copies(N, K, dtype, seed, scale):
    gen = torch.Generator(device=DEV).manual_seed(seed)
    return [(torch.randn(N, generator=gen, device=DEV) * scale).to(dtype) for _ in range(K)]


def _tensor(orc, copies):
    h = orc.tensor_from_copies([host_stored(c) for c in copies], fill=0)
    if copies[0].dtype == torch.bfloat16:
        return torch.from_numpy(h.view(np.int16)).to(DEV).view(torch.bfloat16), h
    return torch.from_numpy(h).to(DEV), h


class Layout:
    """Runs one op on separate buffers or on the tensor layout and returns
    the workers (and gradients) as K host copies."""

    def __init__(self, orc, name, g, K, xs, gs=None, xc=None):
        self.orc, self.name, self.g, self.K = orc, name, g, K
        self.N = g.numel
        self.xs, self.gs, self.xc = xs, gs, xc
        if name == "tensor":
            self.X, _ = _tensor(orc, xs)
            self.G = _tensor(orc, gs)[0] if gs is not None else None

    def x_host(self):
        if self.name == "tensor":
            return self.orc.copies_from_tensor(host_f32(self.X), self.K, self.N)
        return [host_f32(t) for t in self.xs]

    def g_host(self):
        if self.name == "tensor":
            return self.orc.copies_from_tensor(host_stored(self.G), self.K, self.N)
        return [host_stored(t) for t in self.gs]


LAYOUTS = ["separate", "tensor"]


@pytest.mark.parametrize("layout", LAYOUTS)
# K not a power of two (3, 5, 12, 17, 33): the tensor layout's step maps
# lanes to pieces densely, for both gradient types; N = 3 and 5: that
# mapping with no whole slot, and with one whole slot and a ragged tail.
@pytest.mark.parametrize("K,gdt,N", [(1, torch.float32, 6007), (3, torch.float32, 6007), (8, torch.bfloat16, 6007),
                                     (16, torch.float32, 6007), (33, torch.float32, 6007),
                                     (5, torch.bfloat16, 6007), (12, torch.float32, 6007),
                                     (17, torch.bfloat16, 6007), (33, torch.bfloat16, 6007),
                                     (3, torch.float32, 3), (17, torch.bfloat16, 5)])
def test_sgd_step(orc, layout, K, gdt, N):
    g = tc.Group([N])
    xs, gs = _copies(N, K, torch.float32, K, 0.05), _copies(N, K, gdt, 50 + K, 0.01)
    L = Layout(orc, layout, g, K, xs, gs)
    h_x, h_g = L.x_host(), L.g_host()
    if layout == "tensor":
        tc.sgd_step_tensor(g, K, L.X, L.G, 0.05)
    else:
        tc.sgd_step(g, xs, gs, 0.05)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    orc.sgd_step(rx, h_g, 0.05)
    for i, got in enumerate(L.x_host()):
        mag = np.abs(h_x[i].astype(np.float64)) + 0.05 * np.abs(widened(h_g[i]))
        assert_close(got, rx[i], mag, f"{layout} K={K} x[{i}]")


@pytest.mark.parametrize("layout", LAYOUTS)
# K = 17, 20, 33 and 40: the exchange staged through LDS (and at K = 64 in
# the bit-identity and exact-regime tests)
@pytest.mark.parametrize("K", [1, 2, 5, 8, 16, 17, 20, 24, 33, 40])
def test_elastic_async(orc, layout, K):
    N = 4 * 1025 + 2
    g = tc.Group([N])
    xs = _copies(N, K, torch.float32, 100 + K, 0.05)
    xc = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(7), device=DEV) * 0.05
    L = Layout(orc, layout, g, K, xs)
    h_x, h_c = L.x_host(), host_f32(xc)
    order = list(np.random.default_rng(K).permutation(K))[: max(1, K - 1)]
    alpha = 0.1125
    if layout == "tensor":
        tc.elastic_async_tensor(g, K, L.X, xc, order, alpha)
    else:
        tc.elastic_async(g, xs, xc, order, alpha)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    orc.elastic_async(rx, rc, order, alpha)
    # magnitude: every quantity stays within the span of the inputs
    span = np.maximum.reduce([np.abs(a.astype(np.float64)) for a in h_x] + [np.abs(h_c.astype(np.float64))])
    got = L.x_host()
    for i in range(K):
        assert_close(got[i], rx[i], span, f"{layout} K={K} x[{i}]")
    assert_close(host_f32(xc), rc, span, f"{layout} K={K} x_c")


@pytest.mark.parametrize("K,R", [(3, 3), (4, 2), (8, 8), (16, 16), (17, 17), (20, 9), (33, 20), (48, 48), (56, 30), (64, 64)])
def test_elastic_async_layouts_bit_identical(orc, K, R):
    """The tensor-layout exchange runs the center's recurrence once per
    component (four lanes per slot) and hands each difference back through
    LDS; the separate-buffer kernel runs it per element.  Both take the same
    binary32 operations in the same order, so they agree bit for bit, every
    worker (exchanged or not) and the center, on several workgroups and a
    ragged tail."""
    N = 4 * 3001 + 3
    g = tc.Group([N])
    xs = _copies(N, K, torch.float32, 300 + K, 0.05)
    xc = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(8), device=DEV) * 0.05
    order = [int(w) for w in np.random.default_rng(50 + K).permutation(K)[:R]]
    Lt = Layout(orc, "tensor", g, K, xs)
    xc_t = xc.clone()
    tc.elastic_async_tensor(g, K, Lt.X, xc_t, order, 0.1125)
    xs_s, xc_s = [t.clone() for t in xs], xc.clone()
    tc.elastic_async(g, xs_s, xc_s, order, 0.1125)
    torch.cuda.synchronize()
    for i, got in enumerate(Lt.x_host()):
        assert_bits_equal(got, host_f32(xs_s[i]), f"K={K} R={R} x[{i}] tensor vs separate")
    assert_bits_equal(host_f32(xc_t), host_f32(xc_s), f"K={K} R={R} x_c tensor vs separate")


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("K", [1, 4, 8, 16, 64])
def test_elastic_async_exact_regime(orc, layout, K):
    """Integers and alpha = 1/4: exact in binary32, bit for bit."""
    N = 4 * 257 + 3
    g = tc.Group([N])
    xs = wl.integer_values(N, K, 1024, seed=900 + K, device=DEV)
    xc = wl.integer_values(N, 1, 1024, seed=950 + K, device=DEV)[0]
    L = Layout(orc, layout, g, K, xs)
    rx = [a.astype(np.float64) for a in L.x_host()]
    rc = host_f32(xc).astype(np.float64)
    order = list(reversed(range(K)))[: min(K, 6)]
    if layout == "tensor":
        tc.elastic_async_tensor(g, K, L.X, xc, order, 0.25)
    else:
        tc.elastic_async(g, xs, xc, order, 0.25)
    torch.cuda.synchronize()
    orc.elastic_async(rx, rc, order, 0.25)
    for i, got in enumerate(L.x_host()):
        assert_exact(got, rx[i], f"{layout} K={K} x[{i}]")
    assert_exact(host_f32(xc), rc, f"{layout} K={K} x_c")


@pytest.mark.parametrize("layout", LAYOUTS)
# K = 17, 20, 33, 48: the tensor layout's step staged through LDS
@pytest.mark.parametrize("K,gdt,bcast", [(1, torch.float32, True), (4, torch.float32, True), (8, torch.float32, False),
                                         (16, torch.bfloat16, False), (20, torch.float32, True),
                                         (17, torch.float32, False), (33, torch.bfloat16, False),
                                         (48, torch.float32, True)])
def test_sync_sgd(orc, layout, K, gdt, bcast):
    N = 4 * 2001 + 1
    g = tc.Group([N])
    x0 = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(K), device=DEV) * 0.05
    xs = [x0.clone() for _ in range(K)]
    gs = _copies(N, K, gdt, 200 + K, 0.01)
    L = Layout(orc, layout, g, K, xs, gs)
    h_x, h_g = L.x_host(), L.g_host()
    eta, rescale = 0.5, float(np.float32(1.0 / (K * 128)))
    if layout == "tensor":
        tc.sync_sgd_step_tensor(g, K, L.X, L.G, eta, rescale, bcast)
    else:
        tc.sync_sgd_step(g, xs, gs, eta, rescale, bcast)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    S = orc.sync_sgd(rx, h_g, eta, rescale)
    Smag = sum(np.abs(widened(a)) for a in h_g)
    got = L.x_host()
    for i in range(K):
        assert_close(got[i], rx[i], np.abs(h_x[i].astype(np.float64)) + eta * rescale * Smag, f"{layout} x[{i}]")
        assert np.array_equal(got[i], got[0]), "identical workers must stay identical"
    if bcast:
        for i, gi in enumerate(L.g_host()):
            assert_close(gi, S, Smag, f"{layout} broadcast g[{i}]")
    else:
        for a, b in zip(L.g_host(), h_g):
            assert_bits_equal(a, b, "gradients untouched")


@pytest.mark.parametrize("K", [8, 17, 33, 48])
def test_sync_sgd_tensor_sums_equal_the_reduction(orc, K):
    """The broadcast sums of the tensor-layout synchronous step (a full
    butterfly per slot group) equal tc_reduce_tensor's SUM (a split
    butterfly) bit for bit: both add a slot's copies in the pairwise tree
    over P terms, padded with +0.  From K = 17 on, both kernels are staged
    through LDS."""
    N = 4 * 3001 + 2
    g = tc.Group([N])
    gs = _copies(N, K, torch.float32, 300 + K, 0.01)
    xs = [torch.zeros(N, device=DEV) for _ in range(K)]
    L = Layout(orc, "tensor", g, K, xs, gs)
    ref = torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, L.G, ref, "sum")
    tc.sync_sgd_step_tensor(g, K, L.X, L.G, 0.5, 1.0, True)
    torch.cuda.synchronize()
    r = host_f32(ref)
    for i, gi in enumerate(L.g_host()):
        assert_bits_equal(gi, r, f"K={K} broadcast g[{i}] vs tc_reduce_tensor")


def test_sync_sgd_bf16_broadcast_unsupported():
    g = tc.Group([64])
    xs = [torch.zeros(64, device=DEV)]
    gs = [torch.zeros(64, device=DEV, dtype=torch.bfloat16)]
    with pytest.raises(tc.TCError) as e:
        tc.sync_sgd_step(g, xs, gs, 0.1, 1.0, broadcast=True)
    assert e.value.status == tc.TC_EUNSUPPORTED


@pytest.mark.parametrize("layout", LAYOUTS)
def test_period_schedule_matches_oracle(orc, layout):
    """tau = 4 over 10 iterations: elastic steps at 0, 4, 8 and SGD between,
    against the oracle's composition of the two steps."""
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    K, N, tau = 8, 4 * 4099 + 3, 4
    g = tc.Group([N])
    gs = wl.make_gradients(w, N, DEV)
    xs, xc = wl.make_state(w, N, DEV)
    L = Layout(orc, layout, g, K, xs, gs)
    h_x, h_g, h_c = L.x_host(), L.g_host(), host_f32(xc)
    for t in range(10):
        if layout == "tensor":
            tc.easgd_period_step_tensor(g, K, L.X, L.G, xc, w.eta, w.rho, t, tau)
        else:
            tc.easgd_period_step(g, xs, gs, xc, w.eta, w.rho, t, tau)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    # guard: each step's own magnitudes (elastic step: easgd_mags; SGD step:
    # |x_i| + eta |g_i|, the center untouched), taken at the largest value
    # each element reaches along the oracle's trajectory
    mx = [np.zeros_like(a) for a in rx]
    mc = np.zeros_like(rc)
    for t in range(10):
        if t % tau == 0:
            sx, sc = easgd_mags(rx, h_g, rc, w.eta, w.rho)
            orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
        else:
            sx = [np.abs(a) + w.eta * np.abs(widened(b)) for a, b in zip(rx, h_g)]
            sc = np.abs(rc)
            orc.sgd_step(rx, h_g, w.eta)
        mx = [np.maximum(a, b) for a, b in zip(mx, sx)]
        mc = np.maximum(mc, sc)
    for i, got in enumerate(L.x_host()):
        assert_close(got, rx[i], mx[i], f"{layout} x[{i}]")
    assert_close(host_f32(xc), rc, mc, f"{layout} x_c")


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
# (5, 17000003): the separate-buffer kernel's slot path then runs over
# several windows of source chunks, the last one partial, with copy groups
# of 4 and 1 and a ragged element tail, for both element sizes.  (1, 4),
# (1, 1000003): the plain copy kernel at K = 1, with exactly one slot, and
# with a partial last workgroup whose lanes past the end repeat the last
# slot and a ragged tail; (4, 4099): one copy group of four.  (17, 4099),
# (33, 100001): K just above a power of two, where the tensor layout's
# broadcast maps lanes to pieces densely; (3, 2): that mapping with no whole
# slot, the element tail alone.  (35, 4005), (33, 2): above K = 32, where
# 2-byte pieces go two to a lane, with an odd number of pieces (the last
# lane stores one), and with no whole slot.
@pytest.mark.parametrize("K,N", [(1, 7), (3, 4097), (8, 100003), (16, 5), (5, 17000003), (1, 4), (1, 1000003),
                                 (4, 4099), (17, 4099), (33, 100001), (3, 2), (35, 4005), (33, 2)])
def test_broadcast(orc, layout, dtype, K, N):
    g = tc.Group([N])
    src = torch.randn(N, device=DEV).to(dtype)
    if layout == "tensor":
        T = torch.zeros(tc.tensor_numel(g, K), device=DEV).to(dtype)
        tc.broadcast_tensor(g, K, src, T)
        torch.cuda.synchronize()
        outs = orc.copies_from_tensor(host_stored(T), K, N)
    else:
        dsts = [torch.zeros(N + 1, device=DEV).to(dtype)[1:] if K == 3 else torch.zeros(N, device=DEV).to(dtype)
                for _ in range(K)]
        tc.broadcast(g, src, dsts)
        torch.cuda.synchronize()
        outs = [host_stored(d) for d in dsts]
    ref = orc.broadcast(host_stored(src), K)
    for a, b in zip(outs, ref):
        assert_bits_equal(a, b, f"{layout} broadcast")


def test_schedule_argument_errors():
    g = tc.Group([32])
    xs = [torch.zeros(32, device=DEV) for _ in range(3)]
    xc = torch.zeros(32, device=DEV)
    with pytest.raises(tc.TCError):
        tc.elastic_async(g, xs, xc, [0, 0], 0.1)        # a worker twice
    with pytest.raises(tc.TCError):
        tc.elastic_async(g, xs, xc, [3], 0.1)           # outside [0, K)
    with pytest.raises(tc.TCError):
        tc.easgd_period_step(g, xs, xs, xc, 0.1, 0.5, 0, 0)  # tau = 0 (and grads alias workers)
    with pytest.raises(tc.TCError):
        tc.sgd_step(g, xs, xs, 0.1)                      # grad overlaps x
    tc.elastic_async(g, xs, xc, [], 0.1)                 # R = 0: no-op
    torch.cuda.synchronize()
