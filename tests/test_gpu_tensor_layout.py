"""Parity of the tensor-layout entry points (the K copies interleaved in one
buffer) with the CPU oracle, through the C ABI.

The oracle holds the layout's index map (oracle.tensor_from_copies /
copies_from_tensor, pinned against numpy's slot transpose); reduce and step
results are compared after converting the GPU's tensor back to K copies
with it.  Same tolerance as the separate-buffer tests (tests/helpers.py).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_1801_03855_amd as tc
from paper_1801_03855_amd import workloads as wl
from tests.helpers import (assert_bits_equal, assert_close, assert_exact, easgd_mags, host_f32, host_stored,
                           reduce_mag)

pytestmark = pytest.mark.gpu

DEV = "cuda"
SENTINEL_F32 = -12345.5


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _sentinel(dtype):
    return torch.tensor(SENTINEL_F32).to(dtype).item()


def _make_copies(N, K, dtype, seed, scale=1.0):
    gen = torch.Generator(device=DEV).manual_seed(seed)
    return [(torch.randn(N, generator=gen, device=DEV) * scale).to(dtype) for _ in range(K)]


def _to_tensor_layout(orc, copies, fill):
    """Host tensor-layout image of device copies (oracle index map)."""
    return orc.tensor_from_copies([host_stored(c) for c in copies], fill=fill)


def _device_tensor(host, dtype):
    if dtype == torch.bfloat16:
        return torch.from_numpy(host.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(host).to(DEV)


# -------------------------------------------------------------- pack/unpack

def _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=0, misalign=False, views=False):
    g = tc.Group(sizes)
    N = g.numel
    gen = torch.Generator(device=DEV).manual_seed(seed)
    tensors = []
    for _ in range(K):
        if views:
            buf = torch.randn(sum(sizes) + 3, generator=gen, device=DEV).to(dtype)
            copy, at = [], 3
            for s in sizes:
                copy.append(buf[at:at + s])
                at += s
        else:
            copy = [(torch.randn(s + 1, generator=gen, device=DEV).to(dtype)[1:] if misalign
                     else torch.randn(s, generator=gen, device=DEV).to(dtype)) for s in sizes]
        tensors.append(copy)
    tl = tc.TensorList(g, tensors)
    T = torch.full((tc.tensor_numel(g, K),), SENTINEL_F32, device=DEV).to(dtype)
    tc.pack_tensor(tl, T)
    torch.cuda.synchronize()
    flat = [orc.pack([host_stored(t) for t in copy]) for copy in tensors]
    ref = orc.tensor_from_copies(flat, fill=host_stored(torch.tensor([SENTINEL_F32]).to(dtype))[0])
    assert_bits_equal(host_stored(T), ref, f"pack_tensor K={K} {dtype}")  # padding untouched too
    outs = [[torch.full((s,), 7.0, device=DEV).to(dtype) for s in sizes] for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, outs), T)
    torch.cuda.synchronize()
    for k in range(K):
        for t, s in enumerate(sizes):
            if s:
                assert_bits_equal(host_stored(outs[k][t]), host_stored(tensors[k][t]), f"unpack_tensor ({k},{t})")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_resnet50(orc, dtype):
    _tensor_pack_roundtrip(orc, wl.group_sizes("resnet50"), 8, dtype, seed=1)


@pytest.mark.parametrize("K", [1, 3, 5, 9, 16, 17, 24, 31, 64])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_ragged_and_misaligned(orc, K, dtype):
    """Lengths not multiples of 4 (a partial last slot), tensors starting
    one element past their allocation, zero-size tensors; K = 9-31 take the
    copies in groups of one 128-byte line of each slot row (binary32 K > 8,
    bfloat16 K > 16), the last group partial."""
    sizes = [3, 0, 5, 4097, 1, 2, 0, 250, 7]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=K, misalign=True)


@pytest.mark.parametrize("K", [1, 2, 3, 4, 8, 12, 16, 32, 64])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_slot_aligned(orc, K, dtype):
    """Slot-multiple tensor lengths before a ragged last tensor, tensors in
    their own allocations: pack and unpack move each slot straight through
    registers (the last, partial slot element by element); the same sizes
    one element into their allocations take the tiles."""
    sizes = [4096, 8, 0, 12000, 516, 7]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=20 + K)
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=30 + K, misalign=True)


@pytest.mark.parametrize("K", [1, 2, 3, 4, 8, 16, 20])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_large_tensors_tiled(orc, K, dtype):
    """A group of large tensors (mean above 32,768 elements) whose tensors
    start one element into their allocations and whose length is not a
    multiple of 4: the tiles, across many chunk edges inside each tensor,
    in the unpack's shorter tensor-layout chunks at K >= 8."""
    sizes = [40001, 33335, 70002, 32769]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=60 + K, misalign=True)


@pytest.mark.parametrize("K", [1, 2])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("misalign", [False, True])
def test_pack_tensor_longer_chunks(orc, K, dtype, misalign):
    """At K <= 2 a group with enough chunks to fill the chip (here 4.7M
    elements of large tensors: 2,300 chunks of 2,048) packs and unpacks in
    the separate-buffer chunks, several tiles per chunk; slot-multiple
    sizes in their own allocations go straight through registers (but the
    binary32 unpack at K = 2 keeps the short chunks), the same sizes one
    element into their allocations through the tiles."""
    sizes = [1_500_000, 1_200_004, 2_000_000, 9] if not misalign else [1_500_001, 1_200_003, 2_000_002, 9]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=90 + K, misalign=misalign)


@pytest.mark.parametrize("K", [1, 2])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_longer_chunks_small_tensors(orc, K, dtype):
    """The same at K <= 2 for a group of small slot-multiple tensors (1,700
    log-uniform sizes rounded up to multiples of 4, 8.8M elements: 2,148
    chunks of 4,096), chunks holding many tensor boundaries."""
    sizes = [(v + 3) // 4 * 4 for v in wl.many_small_sizes(1700, seed=13)] + [5]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=95 + K)


@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_large_tensors_slot_aligned(orc, K, dtype):
    """Large slot-multiple tensors in their own allocations, ragged last
    tensor: straight through registers where a wave moves at least 256
    bytes of each copy (binary32 up to K = 4, bfloat16 up to K = 2), through
    the tiles otherwise (bfloat16 at K = 3, 4)."""
    sizes = [40000, 33336, 70004, 32768, 5]
    _tensor_pack_roundtrip(orc, sizes, K, dtype, seed=70 + K)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_tensor_views_and_many_small(orc, dtype):
    _tensor_pack_roundtrip(orc, [1, 2, 3, 5, 8, 13, 4099, 1, 7, 4096, 0, 9001], 4, dtype, seed=5, views=True)
    _tensor_pack_roundtrip(orc, wl.many_small_sizes(1500, seed=9), 16, dtype, seed=6, misalign=True)
    _tensor_pack_roundtrip(orc, wl.many_small_sizes(1500, seed=9), 2, dtype, seed=8, misalign=True)
    rng = np.random.default_rng(4)
    # tensors of 0 or 1 elements: about 2,000 per 1,024-element chunk, more than
    # the LDS tables hold, so the global-table search runs too
    _tensor_pack_roundtrip(orc, rng.integers(0, 2, 6000).tolist(), 2, dtype, seed=7)


# ------------------------------------------------------------------ reduce

@pytest.mark.parametrize("K", [1, 2, 3, 4, 7, 8, 16, 20, 33, 64])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_reduce_tensor(orc, K, dtype):
    N = 4 * 3001 + 3
    g = tc.Group([N])
    host = _to_tensor_layout(orc, _make_copies(N, K, dtype, seed=K), fill=0)
    T = _device_tensor(host, dtype)
    copies = orc.copies_from_tensor(host, K, N)
    for op, code in (("sum", oracle.SUM), ("avg", oracle.AVG)):
        out = torch.empty(N, device=DEV)
        tc.reduce_tensor(g, K, T, out, op)
        torch.cuda.synchronize()
        assert_close(host_f32(out), orc.reduce(copies, code), reduce_mag(copies, op == "avg"), f"K={K} {op}")


@pytest.mark.parametrize("K", [2, 3, 6, 10, 16, 18, 24, 33, 64])
def test_reduce_tensor_bf16_pairs(orc, K):
    """bfloat16 copies with K even are read two per lane, which adds each
    pair before the butterfly (the pairwise tree's first level); at K not a
    power of two (6, 10, 18, 24, 33) the copies are staged through LDS and
    paired there, odd K included.  Both layouts add in that tree, so the
    tensor layout's SUM and AVG equal the separate-buffer reduction bit for
    bit on general inputs; integers that bfloat16 holds exactly
    (|v| <= 256) give the oracle's sums exactly."""
    N = 4 * 2053 + 1
    g = tc.Group([N])
    for name, copies in (("general", _make_copies(N, K, torch.bfloat16, seed=40 + K)),
                         ("integer", [c.to(torch.bfloat16) for c in
                                      wl.integer_values(N, K, 256, seed=50 + K, device=DEV)])):
        host = _to_tensor_layout(orc, copies, fill=0)
        T = _device_tensor(host, torch.bfloat16)
        for op, code in (("sum", oracle.SUM), ("avg", oracle.AVG)):
            got, sep = torch.empty(N, device=DEV), torch.empty(N, device=DEV)
            tc.reduce_tensor(g, K, T, got, op)
            tc.reduce(g, copies, sep, op)
            torch.cuda.synchronize()
            assert_bits_equal(host_f32(got), host_f32(sep), f"K={K} {name} {op}: tensor vs separate")
            if name == "integer" and op == "sum":
                assert_exact(host_f32(got), orc.reduce(orc.copies_from_tensor(host, K, N), code), f"K={K} sum")


@pytest.mark.parametrize("K", [1, 3, 8, 16, 31, 64])
def test_tensor_integer_inputs_bit_exact(orc, K):
    """Exact regime (integers, eta = 1/8, rho = 1/2): bit for bit."""
    N = 4 * 1025 + 2
    g = tc.Group([N])
    xs = wl.integer_values(N, K, 1024, seed=500 + K, device=DEV)
    gs = wl.integer_values(N, K, 1024, seed=600 + K, device=DEV)
    xc = wl.integer_values(N, 1, 1024, seed=700 + K, device=DEV)[0]
    hx = _to_tensor_layout(orc, xs, 0)
    hg = _to_tensor_layout(orc, gs, 0)
    X, G = _device_tensor(hx, torch.float32), _device_tensor(hg, torch.float32)
    out = torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, G, out, "sum")
    tc.easgd_step_tensor(g, K, X, G, xc, 0.125, 0.5)
    torch.cuda.synchronize()
    gcopies = orc.copies_from_tensor(hg, K, N)
    assert_exact(host_f32(out), orc.reduce(gcopies, oracle.SUM), f"K={K} sum")
    rx = [a.astype(np.float64) for a in orc.copies_from_tensor(hx, K, N)]
    rc = host_f32(wl.integer_values(N, 1, 1024, seed=700 + K, device=DEV)[0]).astype(np.float64)
    orc.easgd_step(rx, gcopies, rc, 0.125, 0.5)
    got = orc.copies_from_tensor(host_f32(X), K, N)
    for i in range(K):
        assert_exact(got[i], rx[i], f"K={K} x[{i}]")
    assert_exact(host_f32(xc), rc, f"K={K} x_c")


@pytest.mark.parametrize("N", [1, 2, 3, 5, 7])
@pytest.mark.parametrize("K", [1, 3, 16])
def test_tensor_layout_groups_smaller_than_a_slot(orc, N, K):
    """Groups of at most one whole slot: the kernels' element-by-element
    tails alone (N < 4) or one slot and a tail.  Reduction and step against
    the oracle, pack and unpack bit for bit, in both gradient types."""
    g = tc.Group([N])
    for dtype in (torch.float32, torch.bfloat16):
        _tensor_pack_roundtrip(orc, [N], K, dtype, seed=N * 100 + K, misalign=True)
        gs = _make_copies(N, K, dtype, seed=N * 10 + K, scale=0.01)
        hg = _to_tensor_layout(orc, gs, 0)
        G = _device_tensor(hg, dtype)
        gcopies = orc.copies_from_tensor(hg, K, N)
        out = torch.empty(N, device=DEV)
        tc.reduce_tensor(g, K, G, out, "avg")
        xs = _make_copies(N, K, torch.float32, seed=N * 10 + K + 1, scale=0.05)
        hx = _to_tensor_layout(orc, xs, 0)
        X = _device_tensor(hx, torch.float32)
        xc = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(N + K), device=DEV) * 0.05
        h_c = host_f32(xc)
        tc.easgd_step_tensor(g, K, X, G, xc, 0.05, 2.25)
        torch.cuda.synchronize()
        assert_close(host_f32(out), orc.reduce(gcopies, oracle.AVG), reduce_mag(gcopies, True), f"N={N} K={K} avg")
        h_x = orc.copies_from_tensor(hx, K, N)
        rx = [a.astype(np.float64) for a in h_x]
        rc = h_c.astype(np.float64)
        mx, mc = easgd_mags(h_x, gcopies, h_c, 0.05, 2.25)
        orc.easgd_step(rx, gcopies, rc, 0.05, 2.25)
        got = orc.copies_from_tensor(host_f32(X), K, N)
        for i in range(K):
            assert_close(got[i], rx[i], mx[i], f"N={N} K={K} {dtype} x[{i}]")
        assert_close(host_f32(xc), rc, mc, f"N={N} K={K} {dtype} x_c")


# ------------------------------------------------------------------- easgd

@pytest.mark.parametrize("K,gdt", [(1, torch.float32), (2, torch.float32), (3, torch.bfloat16), (4, torch.float32),
                                   (5, torch.float32),
                                   (8, torch.float32), (16, torch.bfloat16), (24, torch.float32),
                                   (40, torch.float32), (64, torch.bfloat16)])
def test_easgd_tensor(orc, K, gdt):
    N = 4 * 2049 + 1
    g = tc.Group([N])
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    xs = _make_copies(N, K, torch.float32, seed=K, scale=0.05)
    gs = _make_copies(N, K, gdt, seed=100 + K, scale=0.01)
    xc = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(200 + K), device=DEV) * 0.05
    hx, hg = _to_tensor_layout(orc, xs, 0), _to_tensor_layout(orc, gs, 0)
    X, G = _device_tensor(hx, torch.float32), _device_tensor(hg, gdt)
    h_c = host_f32(xc)
    rho = 0.9 / (K * w.eta)
    tc.easgd_step_tensor(g, K, X, G, xc, w.eta, rho)
    torch.cuda.synchronize()
    h_x = orc.copies_from_tensor(hx, K, N)
    h_g = orc.copies_from_tensor(hg, K, N)
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, rho)
    orc.easgd_step(rx, h_g, rc, w.eta, rho)
    got = orc.copies_from_tensor(host_f32(X), K, N)
    for i in range(K):
        assert_close(got[i], rx[i], mx[i], f"K={K} x[{i}]")
    assert_close(host_f32(xc), rc, mc, f"K={K} x_c")


def test_resnet50_k8_tensor_step_and_layouts_agree(orc):
    """ResNet-50 group, K=8, one fused step on the tensor layout: every
    element against the oracle, and bit for bit equal to the separate-buffer
    kernel (power-of-two K: the same pairwise tree)."""
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    g = tc.Group(w.sizes())
    N, K = g.numel, w.K
    gs = wl.make_gradients(w, N, DEV)
    xs, xc = wl.make_state(w, N, DEV)
    h_x, h_g, h_c = [host_f32(t) for t in xs], [host_f32(t) for t in gs], host_f32(xc)
    X = torch.empty(tc.tensor_numel(g, K), device=DEV)
    G = torch.empty(tc.tensor_numel(g, K), device=DEV)
    # build the tensors on the GPU with the pack kernel from views of the copies
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, w.sizes()) for t in xs]), X)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, w.sizes()) for t in gs]), G)
    xc2 = xc.clone()
    gbar_t, gbar_s = torch.empty(N, device=DEV), torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, G, gbar_t, "avg")
    tc.reduce(g, gs, gbar_s, "avg")
    tc.easgd_step_tensor(g, K, X, G, xc, w.eta, w.rho)
    tc.easgd_step(g, xs, gs, xc2, w.eta, w.rho)
    torch.cuda.synchronize()
    assert torch.equal(gbar_t, gbar_s)
    assert torch.equal(xc, xc2)
    back = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, [wl.split_views(t, w.sizes()) for t in back]), X)
    torch.cuda.synchronize()
    for i in range(K):
        assert torch.equal(back[i], xs[i]), i
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for i in range(K):
        assert_close(host_f32(back[i]), rx[i], mx[i], f"x[{i}]")
    assert_close(host_f32(xc), rc, mc, "x_c")


def test_many_small_k16_bf16_tensor_pipeline(orc):
    """10,000 log-uniform tensors, K=16, bf16 gradients, on the tensor
    layout: pack_tensor of the gradient tensors, AVG reduce, one step,
    unpack_tensor of the workers; sampled positions plus tensor boundaries
    against the oracle, pack bit for bit in full."""
    w = wl.WORKLOADS["many_small_k16_bf16"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    gflat = wl.make_gradients(w, N, DEV)
    g_tl = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gflat])
    G = torch.empty(tc.tensor_numel(g, K), dtype=torch.bfloat16, device=DEV)
    tc.pack_tensor(g_tl, G)
    torch.cuda.synchronize()
    ref = orc.tensor_from_copies([host_stored(f) for f in gflat], fill=0)
    got = host_stored(G)
    S = (N + 3) // 4
    valid = np.ones((S, K, 4), dtype=bool)
    valid[S - 1, :, N - 4 * (S - 1):] = False if N % 4 else True
    valid = valid.reshape(-1)
    assert_bits_equal(got[valid], ref[valid], "pack_tensor many-small")
    del g_tl
    xs, xc = wl.make_state(w, N, DEV)
    X = torch.empty(tc.tensor_numel(g, K), device=DEV)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    off = np.cumsum([0] + sizes)
    rng = np.random.default_rng(66)
    idx = np.unique(np.concatenate([rng.integers(0, N, 1_000_000), np.clip(np.concatenate([off[1:-1] - 1, off[1:-1]]), 0, N - 1),
                                    np.arange(N - 64, N)]))
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gflat]
    h_c = host_f32(xc[ti])
    gbar = torch.empty(N, device=DEV)
    tc.reduce_tensor(g, K, G, gbar, "avg")
    tc.easgd_step_tensor(g, K, X, G, xc, w.eta, w.rho)
    outs = [[torch.empty(s, device=DEV) for s in sizes] for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, outs), X)
    torch.cuda.synchronize()
    assert_close(host_f32(gbar[ti]), orc.reduce(h_g, oracle.AVG), reduce_mag(h_g, True), "avg")
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for i in range(K):
        assert_close(host_f32(torch.cat(outs[i])[ti]), rx[i], mx[i], f"x[{i}]")
    assert_close(host_f32(xc[ti]), rc, mc, "x_c")


def test_tensor_argument_errors():
    g = tc.Group([16])
    L = tc.lib()
    s = torch.cuda.current_stream().cuda_stream
    X = torch.zeros(tc.tensor_numel(g, 2) + 4, device=DEV)
    G = torch.zeros(tc.tensor_numel(g, 2) + 4, device=DEV)
    xc = torch.zeros(20, device=DEV)
    assert L.easgd_step_tensor(g.handle, 2, X.data_ptr() + 4, G.data_ptr(), 0, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL
    assert "aligned" in tc.last_error()
    assert L.easgd_step_tensor(g.handle, 2, X.data_ptr(), X.data_ptr() + 64, 0, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL
    assert L.easgd_step_tensor(g.handle, 0, X.data_ptr(), G.data_ptr(), 0, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL
    assert L.tc_reduce_tensor(g.handle, 2, G.data_ptr(), G.data_ptr() + 16, 0, 0, s) == tc.TC_EINVAL  # overlap
    assert L.tc_reduce_tensor(g.handle, 65, G.data_ptr(), xc.data_ptr(), 0, 0, s) == tc.TC_EINVAL
    assert L.tc_tensor_numel(g.handle, 0) == -1 and L.tc_tensor_numel(g.handle, 3) == 48
    assert L.easgd_step_tensor(g.handle, 2, X.data_ptr(), G.data_ptr(), 0, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_OK
    torch.cuda.synchronize()
