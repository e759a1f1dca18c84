"""Parity of the one-pass pipeline (easgd_pipeline_tensor) with the CPU oracle
and with the four calls it fuses, through the C ABI.

Every case runs the pipeline and, on copies of the same inputs, the four
calls tc_pack_tensor, tc_reduce_tensor (AVG), easgd_step_tensor and
tc_unpack_tensor; all outputs must agree bit for bit.  Against the oracle
(pack, AVG reduce, the elastic step and unpack in binary64, from host copies
of the inputs): the packed gradients and the unpacked parameters bit for
bit, the AVG, the workers and the center within the guarded tolerance of
tests/helpers.py (exactly, in the integer regime).  The tensor-layout inputs
are built on the host with the oracle's index map, not by the GPU.
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
SENTINEL = -12345.5


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _upload(host, dtype):
    if dtype == torch.bfloat16:
        return torch.from_numpy(host.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(host).to(DEV)


def _lists(flat_host, sizes, dtype, misalign):
    """Per-layer device tensors holding consecutive pieces of a host copy;
    with misalign, every tensor starts one element into its allocation."""
    out, at = [], 0
    for s in sizes:
        piece = flat_host[at:at + s]
        at += s
        if misalign:
            buf = _upload(np.concatenate([flat_host[:1], piece]), dtype)
            out.append(buf[1:])
        else:
            out.append(_upload(piece.copy(), dtype))
    return out


def _sentinel_lists(sizes, K, misalign):
    out = []
    for _ in range(K):
        copy = []
        for s in sizes:
            buf = torch.full((s + (1 if misalign else 0),), SENTINEL, device=DEV)
            copy.append(buf[1:] if misalign else buf)
        out.append(copy)
    return out


def _inputs(sizes, K, gdt, seed, integer=False):
    rng = np.random.default_rng(seed)
    N = sum(sizes)
    if integer:
        gs = [rng.integers(-64, 65, N).astype(np.float32) for _ in range(K)]
        xs = [rng.integers(-512, 513, N).astype(np.float32) for _ in range(K)]
        xc = rng.integers(-512, 513, N).astype(np.float32)
    else:
        gs = [rng.normal(0, 1e-2, N).astype(np.float32) for _ in range(K)]
        xs = [rng.normal(0, 0.05, N).astype(np.float32) for _ in range(K)]
        xc = (np.mean(np.stack(xs).astype(np.float64), axis=0) + rng.normal(0, 1e-3, N)).astype(np.float32)
    if gdt == torch.bfloat16:
        gs = [host_stored(torch.from_numpy(g).to(torch.bfloat16)) for g in gs]
    return gs, xs, xc


def _binary32_quotient(q64):
    """The correctly rounded binary32 value of a quotient the oracle holds
    correctly rounded in binary64: rounding the binary64 value again is
    right unless it sits exactly on a binary32 midpoint, which is checked.
    (An AVG of integers is exact in binary32 only for power-of-two K.)"""
    f = q64.astype(np.float32)
    toward = np.where(q64 > f, np.float32(np.inf), np.float32(-np.inf))
    mid = (f.astype(np.float64) + np.nextafter(f, toward).astype(np.float64)) / 2
    assert not np.any((q64 != f) & (q64 == mid)), "binary64 quotient on a binary32 midpoint"
    return f


def _run(orc, sizes, K, gdt=torch.float32, seed=0, misalign=False, write_g=True, eta=0.05, rho=None,
         integer=False):
    rho = 0.9 / (K * eta) if rho is None else rho
    g = tc.Group(sizes)
    N = g.numel
    gs, xs, xc = _inputs(sizes, K, gdt, seed, integer)
    fill_g = host_stored(torch.tensor([SENTINEL]).to(gdt))[0]
    X_host = orc.tensor_from_copies(xs, fill=np.float32(SENTINEL))
    g_lists = [_lists(h, sizes, gdt, misalign) for h in gs]
    grads = tc.TensorList(g, g_lists)
    tn = tc.tensor_numel(g, K)

    def state():
        return (_upload(X_host.copy(), torch.float32), _upload(xc.copy(), torch.float32),
                torch.full((N,), SENTINEL, device=DEV), torch.full((tn,), SENTINEL, device=DEV).to(gdt))

    # the pipeline
    X1, c1, b1, G1 = state()
    p1 = _sentinel_lists(sizes, K, misalign)
    tc.easgd_pipeline_tensor(grads, tc.TensorList(g, p1), G1 if write_g else None, b1, X1, c1, eta, rho)
    # the four calls it fuses
    X2, c2, b2, G2 = state()
    p2 = _sentinel_lists(sizes, K, misalign)
    tc.pack_tensor(grads, G2)
    tc.reduce_tensor(g, K, G2, b2, "avg")
    tc.easgd_step_tensor(g, K, X2, G2, c2, eta, rho)
    tc.unpack_tensor(tc.TensorList(g, p2), X2)
    torch.cuda.synchronize()

    what = f"sizes[{len(sizes)}] N={N} K={K} {gdt} misalign={misalign} write_g={write_g}"
    for a, b, name in ((X1, X2, "x"), (c1, c2, "x_c"), (b1, b2, "gbar")):
        assert_bits_equal(host_stored(a), host_stored(b), f"{what}: {name} pipeline vs four calls")
    if write_g:
        assert_bits_equal(host_stored(G1), host_stored(G2), f"{what}: packed gradients pipeline vs four calls")
    else:
        assert bool((G1.float() == SENTINEL).all()), f"{what}: g_tensor written although not passed"
    for k in range(K):
        assert torch.equal(torch.cat(p1[k]), torch.cat(p2[k])), f"{what}: params of copy {k} pipeline vs four calls"

    # against the oracle
    packed = [orc.pack([host_stored(t) for t in copy]) for copy in g_lists]
    if write_g:
        assert_bits_equal(host_stored(G1), orc.tensor_from_copies(packed, fill=fill_g), f"{what}: packed gradients")
    avg = orc.reduce(packed, oracle.AVG)
    rx = [a.astype(np.float64) for a in xs]
    rc = xc.astype(np.float64)
    mx, mc = easgd_mags(xs, packed, xc, eta, rho)
    orc.easgd_step(rx, packed, rc, eta, rho)
    got_x = orc.copies_from_tensor(host_f32(X1), K, N)
    if integer:
        assert_bits_equal(host_f32(b1), _binary32_quotient(avg), f"{what}: gbar")
        for i in range(K):
            assert_exact(got_x[i], rx[i], f"{what}: x[{i}]")
        assert_exact(host_f32(c1), rc, f"{what}: x_c")
    else:
        assert_close(host_f32(b1), avg, reduce_mag(packed, True), f"{what}: gbar")
        for i in range(K):
            assert_close(got_x[i], rx[i], mx[i], f"{what}: x[{i}]")
        assert_close(host_f32(c1), rc, mc, f"{what}: x_c")
    for k in range(K):
        unpacked = np.concatenate(orc.unpack(got_x[k], sizes))
        assert_bits_equal(host_f32(torch.cat(p1[k])), unpacked, f"{what}: params of copy {k}")


def test_tiny_k2(orc):
    _run(orc, wl.tiny_sizes(), 2, eta=0.1, rho=0.5)


@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 8, 12, 16, 17, 20, 33, 64])
def test_k_and_ragged_tail(orc, K):
    """Several tiles and chunks, a group length that is not a multiple of 4,
    zero-size tensors, and tensors that end inside a slot.  At K = 12, 17,
    20 and 33 the four calls' step is the LDS-staged kernel, so this also
    holds it bit for bit to the pipelined kernel's own slot-group step."""
    sizes = [3000, 0, 5, 4096, 1, 0, 7, 9001, 2, 20003]
    _run(orc, sizes, K, seed=K)


@pytest.mark.parametrize("sizes", [[1], [3], [2, 1], [5], [4, 3]])
@pytest.mark.parametrize("K,gdt", [(1, torch.float32), (3, torch.bfloat16), (16, torch.float32)])
def test_groups_of_at_most_one_slot(orc, sizes, K, gdt):
    """Groups of at most one whole slot: the tail launch alone (N < 4) or
    one slot and a tail, on both paths (slot-aligned lists and lists one
    element into their allocations)."""
    _run(orc, sizes, K, gdt=gdt, seed=sum(sizes) * 10 + K)
    _run(orc, sizes, K, gdt=gdt, seed=sum(sizes) * 10 + K + 1, misalign=True)


@pytest.mark.parametrize("K,gdt", [(1, torch.float32), (2, torch.float32), (2, torch.bfloat16), (3, torch.float32),
                                   (8, torch.float32), (16, torch.bfloat16), (5, torch.bfloat16)])
def test_misaligned_tensors(orc, K, gdt):
    """Every per-layer tensor one element into its allocation: the gather
    reads unaligned windows, the scatter writes whole granules inside runs,
    with tile edges as run ends."""
    sizes = [513, 4099, 6, 70001, 3, 1030]
    _run(orc, sizes, K, gdt=gdt, seed=10 + K, misalign=True)


@pytest.mark.parametrize("K,gdt", [(1, torch.float32), (2, torch.float32), (3, torch.float32),
                                   (5, torch.float32), (8, torch.float32), (16, torch.float32),
                                   (33, torch.float32), (64, torch.float32), (2, torch.bfloat16),
                                   (4, torch.bfloat16), (8, torch.bfloat16), (16, torch.bfloat16)])
def test_slot_aligned_groups(orc, K, gdt):
    """Every tensor boundary before the last slot on a slot boundary and
    every tensor slot-aligned: while a wave still moves 128 contiguous bytes
    of each copy's gradients (K <= 8 binary32, K <= 4 bfloat16) the kernel
    moves each chunk straight between registers and the per-layer tensors,
    beyond that through the tiles; the last tensor ends inside a slot, which
    a launch of its own completes."""
    sizes = [4096, 8, 0, 12000, 516, 7]
    _run(orc, sizes, K, gdt=gdt, seed=70 + K)
    _run(orc, sizes, K, gdt=gdt, seed=80 + K, eta=0.125, rho=0.5, integer=True)


@pytest.mark.parametrize("K,gdt,misalign", [(1, torch.float32, False), (1, torch.bfloat16, True),
                                            (2, torch.bfloat16, False), (2, torch.float32, True),
                                            (2, torch.float32, False)])
def test_longer_chunks(orc, K, gdt, misalign):
    """A group with enough 1,024-element chunks to fill the chip (2.2M
    elements): at K = 1, and at K = 2 except binary32 gradients on the
    straight path (the last case, which keeps 512), the step takes those
    chunks, several tiles or straight steps per chunk."""
    sizes = [700_000, 900_004, 600_000, 7] if not misalign else [700_001, 900_003, 600_002, 7]
    _run(orc, sizes, K, gdt=gdt, seed=120 + K, misalign=misalign)


@pytest.mark.parametrize("K,gdt,misalign", [(5, torch.float32, False), (8, torch.float32, False),
                                            (8, torch.bfloat16, True), (16, torch.float32, True),
                                            (33, torch.bfloat16, False)])
def test_large_tensor_groups(orc, K, gdt, misalign):
    """A group of large tensors (2.2M elements in three tensors) at K >= 5,
    on the straight path (slot-aligned, binary32 up to K = 8) and through
    the tiles, with the chunking such groups take at these K."""
    sizes = [700_000, 900_004, 600_000, 7] if not misalign else [700_001, 900_003, 600_002, 7]
    _run(orc, sizes, K, gdt=gdt, seed=140 + K, misalign=misalign)


@pytest.mark.parametrize("gdt", [torch.float32, torch.bfloat16])
def test_slot_sizes_misaligned_pointers(orc, gdt):
    """Slot-multiple sizes but tensors one element into their allocations:
    the tiles and funnel shifts, not the straight path."""
    _run(orc, [4096, 8, 12000, 516], 8, gdt=gdt, seed=90, misalign=True)


@pytest.mark.parametrize("write_g", [True, False])
def test_without_packed_gradients(orc, write_g):
    _run(orc, [1000, 2051, 17, 40000], 8, seed=3, write_g=write_g)


def test_many_tensors_per_chunk(orc):
    """Thousands of tensors of 0 or 1 elements (about 2,000 per 1,024-element
    chunk): chunks touch more segments than the LDS tables hold, so the
    kernel reads the global tables."""
    rng = np.random.default_rng(9)
    sizes = [int(s) for s in rng.integers(0, 2, 6000)]
    _run(orc, sizes, 4, gdt=torch.bfloat16, seed=9, misalign=True)
    _run(orc, sizes, 2, gdt=torch.bfloat16, seed=29, misalign=True)
    _run(orc, sizes, 16, seed=19)


@pytest.mark.parametrize("K", [1, 3, 8, 16, 64])
def test_integer_regime_exact(orc, K):
    """Integer values with eta = 1/8, rho = 1/2: every result is exact in
    binary32, so the GPU must equal the oracle exactly."""
    _run(orc, [999, 4, 4097, 13, 2048], K, seed=40 + K, eta=0.125, rho=0.5, integer=True)


def _sample_index(sizes, N, seed):
    off = np.cumsum([0] + sizes)
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.integers(0, N, 500_000),
                                     np.clip(np.concatenate([off[1:-1] - 1, off[1:-1]]), 0, N - 1),
                                     np.arange(max(0, N - 64), N)]))


@pytest.mark.parametrize("wkey", ["resnet50_k8_easgd", "many_small_k16_bf16"])
def test_full_size(orc, wkey):
    """Full workload size in the configuration the bench times (gradients
    written): every output bit for bit equal to the four calls; sampled
    elements (random, every tensor boundary, the tail) against the oracle;
    the parameter tensors bit for bit equal to the workers."""
    w = wl.WORKLOADS[wkey]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    gflat = wl.make_gradients(w, N, DEV)
    grads = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gflat])
    xs, xc = wl.make_state(w, N, DEV)
    idx = _sample_index(sizes, N, 77)
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gflat]
    h_c = host_f32(xc[ti])
    X = torch.empty(tc.tensor_numel(g, K), device=DEV)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    del xs
    gdt = gflat[0].dtype
    del gflat
    res = {}
    for mode in ("pipeline", "four"):
        Xm, cm = X.clone(), xc.clone()
        G = torch.empty(tc.tensor_numel(g, K), dtype=gdt, device=DEV)
        gbar = torch.empty(N, device=DEV)
        params = [torch.empty(N, device=DEV) for _ in range(K)]
        ptl = tc.TensorList(g, [wl.split_views(p, sizes) for p in params])
        if mode == "pipeline":
            tc.easgd_pipeline_tensor(grads, ptl, G, gbar, Xm, cm, w.eta, w.rho)
        else:
            tc.pack_tensor(grads, G)
            tc.reduce_tensor(g, K, G, gbar, "avg")
            tc.easgd_step_tensor(g, K, Xm, G, cm, w.eta, w.rho)
            tc.unpack_tensor(ptl, Xm)
        torch.cuda.synchronize()
        res[mode] = (Xm, cm, G, gbar, params)
        del ptl
    a, b = res["pipeline"], res["four"]
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]) and torch.equal(a[3], b[3])
    assert torch.equal(a[2].view(torch.int16) if gdt == torch.bfloat16 else a[2],
                       b[2].view(torch.int16) if gdt == torch.bfloat16 else b[2])
    for k in range(K):
        assert torch.equal(a[4][k], b[4][k]), k
    del res["four"], b
    Xm, cm, G, gbar, params = a
    assert_close(host_f32(gbar[ti]), orc.reduce(h_g, oracle.AVG), reduce_mag(h_g, True), f"{wkey}: gbar")
    rx = [v.astype(np.float64) for v in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for k in range(K):
        assert_close(host_f32(params[k][ti]), rx[k], mx[k], f"{wkey}: params[{k}]")
    assert_close(host_f32(cm[ti]), rc, mc, f"{wkey}: x_c")
    # the workers' tensor layout holds the same values as the parameter copies
    back = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in back]), Xm)
    torch.cuda.synchronize()
    for k in range(K):
        assert torch.equal(back[k], params[k]), k


def test_pipeline_argument_errors():
    L = tc.lib()
    s = torch.cuda.current_stream().cuda_stream
    g, g2 = tc.Group([16, 5]), tc.Group([16, 5])
    K = 2
    mk = lambda grp, k, dt=torch.float32: tc.TensorList(grp, [[torch.zeros(n, device=DEV).to(dt) for n in (16, 5)]
                                                              for _ in range(k)])
    grads, params = mk(g, K), mk(g, K)
    tn = tc.tensor_numel(g, K)
    X, G = torch.zeros(tn + 4, device=DEV), torch.zeros(tn + 4, device=DEV)
    xc, gbar = torch.zeros(24, device=DEV), torch.zeros(24, device=DEV)
    P = lambda t: t.data_ptr()
    ok = (grads.handle, params.handle, P(G), P(gbar), P(X), P(xc), 0.1, 0.5, s)

    def call(**kw):
        args = list(ok)
        for k, v in kw.items():
            args[["grads", "params", "gt", "gbar", "x", "xc", "eta", "rho"].index(k)] = v
        return L.easgd_pipeline_tensor(*args)

    assert call(params=mk(g2, K).handle) == tc.TC_EINVAL and "groups" in tc.last_error()
    assert call(params=mk(g, 3).handle) == tc.TC_EINVAL and "K" in tc.last_error()
    assert call(params=mk(g, K, torch.bfloat16).handle) == tc.TC_EINVAL
    assert call(grads=None) == tc.TC_EINVAL
    assert call(gbar=None) == tc.TC_EINVAL
    assert call(x=P(X) + 4) == tc.TC_EINVAL and "aligned" in tc.last_error()
    assert call(xc=P(X) + 16) == tc.TC_EINVAL
    assert call(gt=P(X) + 64) == tc.TC_EINVAL
    assert call(eta=float("nan")) == tc.TC_EINVAL
    assert call() == tc.TC_OK
    assert call(gt=None) == tc.TC_OK
    torch.cuda.synchronize()


def test_resnet50_k8_100_iterations_every_path(orc):
    """ResNet-50 group, K = 8, 100 steps with fixed gradients on three paths
    at once: easgd_step on separate buffers, easgd_step_tensor, and the
    one-launch pipeline (packed gradients not written).  With a power-of-two
    K all three keep the same pairwise order, so the workers and the center
    stay bit-identical for all 100 steps; a sample of positions is followed
    by the oracle (the per-step bar on the largest guard magnitude each
    element reaches)."""
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    gs = wl.make_gradients(w, N, DEV)
    xs, xc = wl.make_state(w, N, DEV)
    idx = _sample_index(sizes, N, 91)[::5]
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gs]
    h_c = host_f32(xc[ti])
    X = torch.empty(tc.tensor_numel(g, K), device=DEV)
    G = torch.empty(tc.tensor_numel(g, K), device=DEV)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
    tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in gs]), G)
    Xp, xc_t, xc_p = X.clone(), xc.clone(), xc.clone()
    grads = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gs])
    params = [torch.empty(N, device=DEV) for _ in range(K)]
    ptl = tc.TensorList(g, [wl.split_views(p, sizes) for p in params])
    gbar = torch.empty(N, device=DEV)
    for _ in range(w.iterations):
        tc.easgd_step(g, xs, gs, xc, w.eta, w.rho)
        tc.easgd_step_tensor(g, K, X, G, xc_t, w.eta, w.rho)
        tc.easgd_pipeline_tensor(grads, ptl, None, gbar, Xp, xc_p, w.eta, w.rho)
    torch.cuda.synchronize()
    assert torch.equal(xc_t, xc) and torch.equal(xc_p, xc)
    assert torch.equal(X, Xp)
    back = [torch.empty(N, device=DEV) for _ in range(K)]
    tc.unpack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in back]), X)
    torch.cuda.synchronize()
    for k in range(K):
        assert torch.equal(back[k], xs[k]), k
        assert torch.equal(params[k], xs[k]), k
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    for _ in range(w.iterations):
        orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
        sx, sc = easgd_mags(rx, h_g, rc, w.eta, w.rho)
        mx = [np.maximum(a, b) for a, b in zip(mx, sx)]
        mc = np.maximum(mc, sc)
    for k in range(K):
        assert_close(host_f32(xs[k][ti]), rx[k], mx[k], f"x[{k}] after 100 steps")
    assert_close(host_f32(xc[ti]), rc, mc, "x_c after 100 steps")


@pytest.mark.parametrize("case", ["tiny_k2", "misaligned_k3_bf16"])
def test_steps_replay_from_a_hip_graph(case):
    """Every data entry point only launches kernels (no allocation, no
    synchronisation, no memset), so a step can be captured in a HIP graph.
    The four calls, the three calls with the reduction and the step as one
    (reduce_easgd_step_tensor), and the one-launch pipeline are captured once
    and replayed five times, with eager work and synchronisations between the
    replays; after every replay the state equals the same number of eager
    steps, bit for bit.  The tiny group takes the straight paths; the
    second case (lengths not multiples of 4, bfloat16 gradient tensors one
    element into their buffer, a ragged tail) the tiles, funnel shifts and
    the pipeline's tail launch."""
    if case == "tiny_k2":
        w = wl.WORKLOADS["tiny_k2"]
        sizes, K, gdt, eta, rho = w.sizes(), w.K, torch.float32, w.eta, w.rho
        g = tc.Group(sizes)
        N = g.numel
        gflat = wl.make_gradients(w, N, DEV)
        xs, xc = wl.make_state(w, N, DEV)
        grads = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gflat])
    else:
        sizes, K, gdt, eta, rho = [513, 4099, 6, 7001, 3], 3, torch.bfloat16, 0.05, 2.0
        g = tc.Group(sizes)
        N = g.numel
        gen = torch.Generator(device=DEV).manual_seed(77)
        gflat = [(torch.randn(N + 1, generator=gen, device=DEV) * 0.01).to(gdt)[1:] for _ in range(K)]
        xs = [torch.randn(N, generator=gen, device=DEV) * 0.05 for _ in range(K)]
        xc = torch.randn(N, generator=gen, device=DEV) * 0.05
        grads = tc.TensorList(g, [wl.split_views(f, sizes) for f in gflat])

    def make():
        # zeros: the padding of a partial last slot is never written
        X = torch.zeros(tc.tensor_numel(g, K), device=DEV)
        tc.pack_tensor(tc.TensorList(g, [wl.split_views(t, sizes) for t in xs]), X)
        G = torch.zeros(tc.tensor_numel(g, K), dtype=gdt, device=DEV)
        params = [torch.empty(N, device=DEV) for _ in range(K)]
        return dict(X=X, G=G, c=xc.clone(), gbar=torch.empty(N, device=DEV), params=params,
                    ptl=tc.TensorList(g, [wl.split_views(p, sizes) for p in params]))

    def four(st, s):
        tc.pack_tensor(grads, st["G"], s)
        tc.reduce_tensor(g, K, st["G"], st["gbar"], "avg", s)
        tc.easgd_step_tensor(g, K, st["X"], st["G"], st["c"], eta, rho, s)
        tc.unpack_tensor(st["ptl"], st["X"], s)

    def three(st, s):
        tc.pack_tensor(grads, st["G"], s)
        tc.reduce_easgd_step_tensor(g, K, st["X"], st["G"], st["c"], st["gbar"], eta, rho, "avg", s)
        tc.unpack_tensor(st["ptl"], st["X"], s)

    def one(st, s):
        tc.easgd_pipeline_tensor(grads, st["ptl"], st["G"], st["gbar"], st["X"], st["c"], eta, rho, s)

    for step in (four, three, one):
        eager, graphed = make(), make()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            step(graphed, side)  # recorded, not run
        torch.cuda.synchronize()
        for rep in range(5):
            graph.replay()
            step(eager, torch.cuda.current_stream())
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=DEV).sum()  # unrelated eager work between replays
            for key in ("X", "G", "c", "gbar"):
                assert torch.equal(graphed[key], eager[key]), (step.__name__, rep, key)
            for k in range(K):
                assert torch.equal(graphed["params"][k], eager["params"][k]), (step.__name__, rep, k)
            del scratch
        del graph


@pytest.mark.parametrize("fused", [False, True])
def test_separate_buffer_step_replays_from_a_hip_graph(fused):
    """The separate-buffer step (pack, AVG, fused step, unpack; or pack, the
    AVG and the step as one reduce_easgd_step call, unpack; the pointer
    arrays travel as launch arguments) captured once and replayed five times
    equals five eager steps bit for bit after every replay."""
    w = wl.WORKLOADS["tiny_k2"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N, K = g.numel, w.K
    gflat = wl.make_gradients(w, N, DEV)
    xs, xc = wl.make_state(w, N, DEV)
    grads = tc.TensorList(g, [wl.separate_tensors(f, sizes) for f in gflat])

    def make():
        st = dict(x=[t.clone() for t in xs], c=xc.clone(), gbar=torch.empty(N, device=DEV),
                  g=[torch.empty(N, device=DEV) for _ in range(K)], p=[torch.empty(N, device=DEV) for _ in range(K)])
        st["ptl"] = tc.TensorList(g, [wl.split_views(p, sizes) for p in st["p"]])
        return st

    def step(st, s):
        tc.pack(grads, st["g"], s)
        if fused:
            tc.reduce_easgd_step(g, st["x"], st["g"], st["c"], st["gbar"], w.eta, w.rho, "avg", s)
        else:
            tc.reduce(g, st["g"], st["gbar"], "avg", s)
            tc.easgd_step(g, st["x"], st["g"], st["c"], w.eta, w.rho, s)
        tc.unpack(st["ptl"], st["x"], s)

    eager, graphed = make(), make()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        step(graphed, side)
    torch.cuda.synchronize()
    for rep in range(5):
        graph.replay()
        step(eager, torch.cuda.current_stream())
        torch.cuda.synchronize()
        scratch = torch.randn(1 << 16, device=DEV).sum()
        assert torch.equal(graphed["c"], eager["c"]) and torch.equal(graphed["gbar"], eager["gbar"]), rep
        for k in range(K):
            for key in ("x", "g", "p"):
                assert torch.equal(graphed[key][k], eager[key][k]), (rep, key, k)
        del scratch
    del graph
