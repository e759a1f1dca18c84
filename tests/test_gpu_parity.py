"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Inputs come from the seeded generators in paper_1801_03855_amd.workloads,
on the GPU; the oracle works on host copies of the same inputs taken before
any kernel runs.  Floating-point results must be within the guarded 1e-5
tolerance of tests/helpers.py; integer-valued inputs, pack and unpack must
match bit for bit.
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_1801_03855_amd as tc
from paper_1801_03855_amd import workloads as wl
from tests.helpers import (assert_bits_equal, assert_close, assert_exact, easgd_mags, host_f32,
                           host_stored, reduce_mag, widened)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tc.lib()  # fails loudly if the HIP library is missing
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _reduce_check(orc, g, ins, op, what):
    out = torch.empty(g.numel, dtype=torch.float32, device=DEV)
    h_in = [host_stored(t) for t in ins]
    tc.reduce(g, ins, out, op)
    torch.cuda.synchronize()
    ref = orc.reduce(h_in, oracle.AVG if op == "avg" else oracle.SUM)
    return assert_close(host_f32(out), ref, reduce_mag(h_in, op == "avg"), what)


def _easgd_check(orc, g, xs, gs, xc, eta, rho, what, steps=1):
    h_x = [host_f32(t) for t in xs]
    h_g = [host_stored(t) for t in gs]
    h_c = host_f32(xc)
    for _ in range(steps):
        tc.easgd_step(g, xs, gs, xc, eta, rho)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, eta, rho)
    if steps > 1:
        mx = [m.copy() for m in mx]
        for _ in range(steps):
            orc.easgd_step(rx, h_g, rc, eta, rho)
            sx, sc = easgd_mags(rx, h_g, rc, eta, rho)
            mx = [np.maximum(a, b) for a, b in zip(mx, sx)]
            mc = np.maximum(mc, sc)
    else:
        orc.easgd_step(rx, h_g, rc, eta, rho)
    worst = 0.0
    for i, t in enumerate(xs):
        worst = max(worst, assert_close(host_f32(t), rx[i], mx[i], f"{what} x[{i}]"))
    worst = max(worst, assert_close(host_f32(xc), rc, mc, f"{what} x_c"))
    return worst


# ------------------------------------------------------------------ configs

def test_tiny_k2_reduce_and_step(orc):
    """Tiny group, K=2: AVG reduce of the gradients and one step."""
    w = wl.WORKLOADS["tiny_k2"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    assert g.numel == 7392
    gs = wl.make_gradients(w, g.numel, DEV)
    xs, xc = wl.make_state(w, g.numel, DEV)
    _reduce_check(orc, g, gs, "avg", "tiny avg")
    _easgd_check(orc, g, xs, gs, xc, w.eta, w.rho, "tiny step")


@pytest.mark.parametrize("op", ["sum", "avg"])
def test_resnet50_k4_reduce(orc, op):
    """ResNet-50 group (161 tensors, 25,557,032 elements), K=4, every element."""
    w = wl.WORKLOADS["resnet50_k4_reduce"]
    g = tc.Group(w.sizes())
    gs = wl.make_gradients(w, g.numel, DEV)
    _reduce_check(orc, g, gs, op, f"resnet50 {op}")


def test_resnet50_k8_one_step(orc):
    """ResNet-50 group, K=8, one fused step, every element."""
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    g = tc.Group(w.sizes())
    gs = wl.make_gradients(w, g.numel, DEV)
    xs, xc = wl.make_state(w, g.numel, DEV)
    _easgd_check(orc, g, xs, gs, xc, w.eta, w.rho, "resnet50 k8 step")


def _sample_index(N, count, seed, sizes):
    rng = np.random.default_rng(seed)
    idx = set(rng.integers(0, N, count).tolist())
    idx.update(range(0, min(N, 4096)))
    idx.update(range(max(0, N - 4096), N))
    off = np.cumsum([0] + list(sizes))
    for o in off[1:-1]:  # both sides of every tensor boundary
        idx.update(range(max(0, o - 2), min(N, o + 2)))
    return np.array(sorted(idx), dtype=np.int64)


def test_resnet50_k8_100_iterations(orc):
    """ResNet-50 group, K=8, 100 fused steps with fixed gradients; a sample of
    ~1M positions followed by the oracle for all 100 steps.  Tolerance: the
    per-step bar applied to the largest guard magnitude each element reaches
    along the oracle's trajectory."""
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    gs = wl.make_gradients(w, g.numel, DEV)
    xs, xc = wl.make_state(w, g.numel, DEV)
    idx = _sample_index(g.numel, 1_000_000, 33, sizes)
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gs]
    h_c = host_f32(xc[ti])
    for _ in range(w.iterations):
        tc.easgd_step(g, xs, gs, xc, w.eta, w.rho)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    for _ in range(w.iterations):
        orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
        sx, sc = easgd_mags(rx, h_g, rc, w.eta, w.rho)
        mx = [np.maximum(a, b) for a, b in zip(mx, sx)]
        mc = np.maximum(mc, sc)
    for i, t in enumerate(xs):
        assert_close(host_f32(t[ti]), rx[i], mx[i], f"x[{i}] after 100 steps")
    assert_close(host_f32(xc[ti]), rc, mc, "x_c after 100 steps")


def test_vgg16_k4_one_step_sampled(orc):
    """VGG-16 group (32 tensors, 138,357,544 elements), K=4, one fused step;
    ~4M sampled positions plus both sides of every tensor boundary and the
    first and last 4096 elements."""
    w = wl.WORKLOADS["vgg16_k4_easgd"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    assert g.numel == 138_357_544
    gs = wl.make_gradients(w, g.numel, DEV)
    xs, xc = wl.make_state(w, g.numel, DEV)
    idx = _sample_index(g.numel, 4_000_000, 44, sizes)
    ti = torch.from_numpy(idx).to(DEV)
    h_x = [host_f32(t[ti]) for t in xs]
    h_g = [host_stored(t[ti]) for t in gs]
    h_c = host_f32(xc[ti])
    tc.easgd_step(g, xs, gs, xc, w.eta, w.rho)
    torch.cuda.synchronize()
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for i, t in enumerate(xs):
        assert_close(host_f32(t[ti]), rx[i], mx[i], f"vgg16 x[{i}]")
    assert_close(host_f32(xc[ti]), rc, mc, "vgg16 x_c")


def test_many_small_k16_bf16(orc):
    """10,000 log-uniform tensors (59,303,476 elements), K=16, bfloat16
    gradients: pack of the gradient tensors, AVG reduce, one fused step and
    unpack of the workers, as one pipeline.  pack/unpack bit for bit on every
    element of copies 0 and 15 and against torch.cat for all copies; reduce
    and step on ~2M sampled positions plus tensor boundaries."""
    w = wl.WORKLOADS["many_small_k16_bf16"]
    sizes = w.sizes()
    g = tc.Group(sizes)
    N = g.numel
    assert N == 59_303_476
    gflat_src = wl.make_gradients(w, N, DEV)
    g_tensors = [wl.separate_tensors(f, sizes) for f in gflat_src]
    del gflat_src
    g_tl = tc.TensorList(g, g_tensors)
    gflat = [torch.empty(N, dtype=torch.bfloat16, device=DEV) for _ in range(w.K)]
    tc.pack(g_tl, gflat)
    torch.cuda.synchronize()
    for k in (0, w.K - 1):
        ref = orc.pack([host_stored(t) for t in g_tensors[k]])
        assert_bits_equal(host_stored(gflat[k]), ref, f"pack copy {k}")
    for k in range(w.K):
        assert torch.equal(gflat[k].view(torch.int16), torch.cat(g_tensors[k]).view(torch.int16)), k
    del g_tensors, g_tl

    xs, xc = wl.make_state(w, N, DEV)
    idx = _sample_index(N, 2_000_000, 55, sizes)
    ti = torch.from_numpy(idx).to(DEV)
    h_g = [host_stored(t[ti]) for t in gflat]
    h_x = [host_f32(t[ti]) for t in xs]
    h_c = host_f32(xc[ti])

    gbar = torch.empty(N, dtype=torch.float32, device=DEV)
    tc.reduce(g, gflat, gbar, "avg")
    tc.easgd_step(g, xs, gflat, xc, w.eta, w.rho)
    x_tensors = [[torch.empty(s, dtype=torch.float32, device=DEV) for s in sizes] for _ in range(2)]
    x_tl = tc.TensorList(g, x_tensors)
    tc.unpack(x_tl, [xs[0], xs[w.K - 1]])
    torch.cuda.synchronize()

    ref = orc.reduce(h_g, oracle.AVG)
    assert_close(host_f32(gbar[ti]), ref, reduce_mag(h_g, True), "many-small avg")
    rx = [a.astype(np.float64) for a in h_x]
    rc = h_c.astype(np.float64)
    mx, mc = easgd_mags(h_x, h_g, h_c, w.eta, w.rho)
    orc.easgd_step(rx, h_g, rc, w.eta, w.rho)
    for i, t in enumerate(xs):
        assert_close(host_f32(t[ti]), rx[i], mx[i], f"many-small x[{i}]")
    assert_close(host_f32(xc[ti]), rc, mc, "many-small x_c")
    for j, k in enumerate((0, w.K - 1)):
        parts = orc.unpack(host_f32(xs[k]), sizes)
        for t, (a, b) in enumerate(zip(x_tensors[j], parts)):
            if t % 97 == 0 or t == len(sizes) - 1:
                assert_bits_equal(host_f32(a), b, f"unpack copy {k} tensor {t}")
        assert torch.equal(torch.cat(x_tensors[j]), xs[k])


# ------------------------------------------------------- exact regimes

def test_golden_exact_regime():
    """Integer-valued fixture written by the oracle: bit-exact."""
    data = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "exact_regime.json")))
    N = data["N"]
    g = tc.Group([5, 0, 30, 2])
    assert g.numel == N
    for case in data["reduce"]:
        ins = [torch.tensor(a, dtype=torch.float32, device=DEV) for a in case["in"]]
        for op in ("sum", "avg"):
            if op not in case:
                continue
            out = torch.empty(N, dtype=torch.float32, device=DEV)
            tc.reduce(g, ins, out, op)
            assert_exact(host_f32(out), np.array(case[op]), f"golden {op} K={case['K']}")
    for case in data["easgd"]:
        xs = [torch.tensor(a, dtype=torch.float32, device=DEV) for a in case["x"]]
        gs = [torch.tensor(a, dtype=torch.float32, device=DEV) for a in case["g"]]
        xc = torch.tensor(case["xc"], dtype=torch.float32, device=DEV)
        tc.easgd_step(g, xs, gs, xc, case["eta"], case["rho"])
        for i, t in enumerate(xs):
            assert_exact(host_f32(t), np.array(case["x_out"][i]), f"golden x[{i}] K={case['K']}")
        assert_exact(host_f32(xc), np.array(case["xc_out"]), f"golden x_c K={case['K']}")


KS = list(range(1, 18)) + [31, 32, 33, 64]


@pytest.mark.parametrize("K", KS)
def test_integer_inputs_bit_exact(orc, K):
    """Integer-valued inputs (|v| <= 1024) and dyadic eta = 1/8, rho = 1/2:
    every intermediate is exact in binary32, so SUM, AVG and the step must
    equal the oracle bit for bit, for every K (specialised and generic
    kernels) and a ragged length (N = 4*4099 + 3)."""
    N = 4 * 4099 + 3
    g = tc.Group([1000, 0, N - 1000])
    ins = wl.integer_values(N, K, 1024, seed=100 + K, device=DEV)
    h_in = [host_f32(t) for t in ins]
    for op, code in (("sum", oracle.SUM), ("avg", oracle.AVG)):
        out = torch.empty(N, dtype=torch.float32, device=DEV)
        tc.reduce(g, ins, out, op)
        torch.cuda.synchronize()
        ref = orc.reduce(h_in, code)
        if op == "avg" and K & (K - 1):
            # sum/K is not a binary32 number: the result must be its correct
            # rounding (binary64 then binary32 rounds the same way here,
            # since no quotient of small integers by K <= 64 has a run of
            # 28 equal bits right after the 24th)
            ref = ref.astype(np.float32).astype(np.float64)
        assert_exact(host_f32(out), ref, f"K={K} {op}")
    xs = wl.integer_values(N, K, 1024, seed=200 + K, device=DEV)
    gs = wl.integer_values(N, K, 1024, seed=300 + K, device=DEV)
    xc = wl.integer_values(N, 1, 1024, seed=400 + K, device=DEV)[0]
    rx = [host_f32(t).astype(np.float64) for t in xs]
    h_g = [host_f32(t) for t in gs]
    rc = host_f32(xc).astype(np.float64)
    tc.easgd_step(g, xs, gs, xc, 0.125, 0.5)
    torch.cuda.synchronize()
    orc.easgd_step(rx, h_g, rc, 0.125, 0.5)
    for i, t in enumerate(xs):
        assert_exact(host_f32(t), rx[i], f"K={K} x[{i}]")
    assert_exact(host_f32(xc), rc, f"K={K} x_c")


def test_integer_inputs_bf16_bit_exact(orc):
    """bfloat16 integer gradients (|v| <= 128, exact in bfloat16)."""
    K, N = 16, 10007
    g = tc.Group([N])
    gs = [t.to(torch.bfloat16) for t in wl.integer_values(N, K, 128, seed=7, device=DEV)]
    h_g = [host_stored(t) for t in gs]
    out = torch.empty(N, dtype=torch.float32, device=DEV)
    tc.reduce(g, gs, out, "avg")
    torch.cuda.synchronize()
    assert_exact(host_f32(out), orc.reduce(h_g, oracle.AVG), "bf16 avg")
    xs = wl.integer_values(N, K, 1024, seed=8, device=DEV)
    xc = wl.integer_values(N, 1, 1024, seed=9, device=DEV)[0]
    rx = [host_f32(t).astype(np.float64) for t in xs]
    rc = host_f32(xc).astype(np.float64)
    tc.easgd_step(g, xs, gs, xc, 0.125, 0.5)
    torch.cuda.synchronize()
    orc.easgd_step(rx, h_g, rc, 0.125, 0.5)
    for i, t in enumerate(xs):
        assert_exact(host_f32(t), rx[i], f"bf16 x[{i}]")
    assert_exact(host_f32(xc), rc, "bf16 x_c")


# ---------------------------------------------------------- properties

@pytest.mark.parametrize("K", [2, 4, 8, 16, 32, 64])
def test_avg_of_identical_copies_is_the_copy(K):
    """Full ResNet-50 length: AVG of K identical copies returns the copy bit
    for bit (power-of-two K, pairwise tree)."""
    N = 25_557_032 if K <= 16 else 1_000_003
    g = tc.Group([N])
    v = torch.randn(N, generator=torch.Generator(device=DEV).manual_seed(K), device=DEV)
    out = torch.empty_like(v)
    tc.reduce(g, [v] * K, out, "avg")
    torch.cuda.synchronize()
    assert torch.equal(out, v)


def test_rho_zero_center_fixed_and_eta_zero_identity(orc):
    """rho = 0 leaves the center bit for bit; eta = 0 leaves everything."""
    K, N = 8, 1 << 20
    g = tc.Group([N])
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    gs = wl.make_gradients(w, N, DEV)
    xs, xc = wl.make_state(w, N, DEV)
    c0 = xc.clone()
    tc.easgd_step(g, xs, gs, xc, 0.05, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(xc, c0)
    x0 = [t.clone() for t in xs]
    tc.easgd_step(g, xs, gs, xc, 0.0, 2.25)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(xs, x0)) and torch.equal(xc, c0)


# -------------------------------------------------------------- edges

def test_unaligned_buffers_take_the_element_path(orc):
    """Buffers offset by one element (4-byte but not 16-byte aligned)."""
    K, N = 5, 70001
    g = tc.Group([N])
    w = wl.WORKLOADS["resnet50_k8_easgd"]
    base_g = wl.make_gradients(w, N + 1, DEV)[:K]
    base_x, base_c = wl.make_state(w, N + 1, DEV)
    gs = [t[1:] for t in base_g]
    xs = [t[1:] for t in base_x[:K]]
    xc = base_c[1:]
    _reduce_check(orc, g, gs, "avg", "unaligned avg")
    _easgd_check(orc, g, xs, gs, xc, 0.05, 0.9 / (K * 0.05), "unaligned step")


def test_in_place_reduce(orc):
    K, N = 4, 100003
    g = tc.Group([N])
    ins = [torch.randn(N, device=DEV) for _ in range(K)]
    h_in = [host_f32(t) for t in ins]
    tc.reduce(g, ins, ins[0], "avg")
    torch.cuda.synchronize()
    assert_close(host_f32(ins[0]), orc.reduce(h_in, oracle.AVG), reduce_mag(h_in, True), "in place")


@pytest.mark.parametrize("N", [0, 1, 2, 3, 4, 5, 1023, 1024, 1025])
def test_small_and_empty_lengths(orc, N):
    sizes = [N] if N else [0, 0]
    g = tc.Group(sizes)
    K = 3
    ins = [torch.randn(max(N, 1), device=DEV)[:N] for _ in range(K)]
    out = torch.empty(max(N, 1), device=DEV)[:N]
    tc.reduce(g, ins, out, "sum")
    xs = [torch.randn(max(N, 1), device=DEV)[:N] for _ in range(K)]
    xc = torch.randn(max(N, 1), device=DEV)[:N]
    h_x, h_g, h_c = [host_f32(t) for t in xs], [host_f32(t) for t in ins], host_f32(xc)
    tc.easgd_step(g, xs, ins, xc, 0.05, 1.0)
    torch.cuda.synchronize()
    if N:
        h_in = [host_f32(t) for t in ins]
        assert_close(host_f32(out), orc.reduce(h_in, oracle.SUM), reduce_mag(h_in, False), "sum")
        rx = [a.astype(np.float64) for a in h_x]
        rc = h_c.astype(np.float64)
        mx, mc = easgd_mags(h_x, h_g, h_c, 0.05, 1.0)
        orc.easgd_step(rx, h_g, rc, 0.05, 1.0)
        for i, t in enumerate(xs):
            assert_close(host_f32(t), rx[i], mx[i], f"x[{i}]")
        assert_close(host_f32(xc), rc, mc, "x_c")


def _pack_roundtrip(orc, sizes, K, dtype, misalign=False, seed=0, flat_shift=0, views=False):
    """pack then unpack through the C ABI, both checked bit for bit against
    the oracle.  misalign: every tensor starts one element past its
    allocation; views: the tensors of a copy are adjacent views of one
    buffer starting at an odd element (so neighbours share 16-byte
    granules); flat_shift: the flat buffers start that many elements past
    their allocation."""
    g = tc.Group(sizes)
    gen = torch.Generator(device=DEV).manual_seed(seed)
    tensors = []
    for _ in range(K):
        copy = []
        if views:
            buf = torch.randn(sum(sizes) + 3, generator=gen, device=DEV).to(dtype)
            at = 3
            for s in sizes:
                copy.append(buf[at:at + s])
                at += s
        for s in ([] if views else sizes):
            if misalign:
                t = torch.randn(s + 1, generator=gen, device=DEV).to(dtype)[1:]
            else:
                t = torch.randn(s, generator=gen, device=DEV).to(dtype)
            copy.append(t)
        tensors.append(copy)
    tl = tc.TensorList(g, tensors)
    flats = [torch.empty(g.numel + flat_shift + 1, dtype=dtype, device=DEV)[flat_shift:flat_shift + g.numel]
             for _ in range(K)]
    tc.pack(tl, flats)
    torch.cuda.synchronize()
    for k in range(K):
        ref = orc.pack([host_stored(t) for t in tensors[k]]) if g.numel else np.zeros(0)
        if g.numel:
            assert_bits_equal(host_stored(flats[k]), ref, f"pack copy {k}")
    if views:
        outs = []
        for _ in range(K):
            buf = torch.full((sum(sizes) + 5,), 7.0, device=DEV).to(dtype)
            at, copy = 5, []
            for s in sizes:
                copy.append(buf[at:at + s])
                at += s
            outs.append(copy)
    else:
        outs = [[torch.full((s,), 7.0, device=DEV).to(dtype) for s in sizes] for _ in range(K)]
    tl2 = tc.TensorList(g, outs)
    tc.unpack(tl2, flats)
    torch.cuda.synchronize()
    for k in range(K):
        parts = orc.unpack(host_stored(flats[k]), sizes) if g.numel else [np.zeros(0)] * len(sizes)
        for t in range(len(sizes)):
            if sizes[t]:
                assert_bits_equal(host_stored(outs[k][t]), parts[t], f"unpack ({k},{t})")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_resnet50_group(orc, dtype):
    _pack_roundtrip(orc, wl.group_sizes("resnet50"), 2, dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_misaligned_tensors(orc, dtype):
    """Tensors starting one element past an allocation: element path."""
    sizes = [1, 7, 4096, 3, 5000, 0, 4, 12345]
    _pack_roundtrip(orc, sizes, 3, dtype, misalign=True, seed=1)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_large_tensors_misaligned(orc, dtype):
    """A group of large tensors (mean above 32,768 elements: 2,048-element
    chunks, 4,096 for bfloat16), tensors one element into their allocations
    and flat buffers one element past a 16-byte boundary: chunk edges inside
    tensors, on both sides unaligned."""
    sizes = [40001, 33335, 70002, 32769, 3]
    _pack_roundtrip(orc, sizes, 3, dtype, misalign=True, seed=40)
    _pack_roundtrip(orc, sizes, 2, dtype, misalign=True, seed=41, flat_shift=1)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("flat_shift", [1, 2, 3])
def test_pack_misaligned_flat_buffers(orc, dtype, flat_shift):
    """Flat buffers 1-3 elements past a 16-byte boundary, tensors aligned and
    misaligned."""
    sizes = wl.many_small_sizes(300, seed=flat_shift)
    _pack_roundtrip(orc, sizes, 2, dtype, seed=10 + flat_shift, flat_shift=flat_shift)
    _pack_roundtrip(orc, sizes, 2, dtype, misalign=True, seed=20 + flat_shift, flat_shift=flat_shift)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_adjacent_views(orc, dtype):
    """Tensors that are adjacent views of one buffer at odd offsets: unpack
    writes neighbouring tensors' bytes within the same 16-byte granules from
    different lanes and workgroups."""
    sizes = [1, 2, 3, 5, 8, 13, 4099, 1, 7, 4096, 4097, 0, 6, 9000, 1, 1, 1, 33]
    _pack_roundtrip(orc, sizes, 3, dtype, seed=30, views=True)
    _pack_roundtrip(orc, wl.many_small_sizes(500, seed=31), 2, dtype, seed=31, views=True, flat_shift=1)


def test_pack_many_tiny_and_empty_tensors(orc):
    """5000 tensors of 0-3 elements: one chunk touches more tensors than fit
    in LDS, so the global-table search runs too."""
    rng = np.random.default_rng(3)
    sizes = rng.integers(0, 4, 5000).tolist()
    _pack_roundtrip(orc, sizes, 2, torch.float32, seed=2)
    _pack_roundtrip(orc, sizes, 2, torch.bfloat16, seed=3)


def test_pack_zero_total():
    g = tc.Group([0, 0, 0])
    tl = tc.TensorList(g, [[torch.empty(0, device=DEV)] * 3])
    tc.pack(tl, [torch.empty(0, device=DEV)])
    tc.unpack(tl, [torch.empty(0, device=DEV)])
    torch.cuda.synchronize()


def test_pack_many_small_group_smaller(orc):
    """2000 log-uniform tensors (the many-small distribution), K=4."""
    _pack_roundtrip(orc, wl.many_small_sizes(2000, seed=11), 4, torch.bfloat16, seed=4)
    _pack_roundtrip(orc, wl.many_small_sizes(2000, seed=12), 4, torch.float32, misalign=True, seed=5)


# ------------------------------------------------------------- errors

def test_argument_errors():
    g = tc.Group([16])
    a = [torch.zeros(16, device=DEV) for _ in range(3)]
    out = torch.zeros(16, device=DEV)
    L = tc.lib()
    from paper_1801_03855_amd import _ptr_array
    pa = _ptr_array([t.data_ptr() for t in a])
    s = torch.cuda.current_stream().cuda_stream
    assert L.tc_reduce(g.handle, 0, pa, out.data_ptr(), 0, s) == tc.TC_EINVAL
    assert L.tc_reduce(g.handle, 65, pa, out.data_ptr(), 0, s) == tc.TC_EINVAL
    assert L.tc_reduce(g.handle, 3, pa, out.data_ptr(), 7, s) == tc.TC_EINVAL
    assert L.tc_reduce(None, 3, pa, out.data_ptr(), 0, s) == tc.TC_EINVAL
    assert L.tc_reduce(g.handle, 3, pa, None, 0, s) == tc.TC_EINVAL
    assert L.tc_reduce(g.handle, 3, pa, a[1].data_ptr() + 4, 0, s) == tc.TC_EINVAL  # partial overlap
    assert "overlap" in tc.last_error()
    # bfloat16 inputs: out may not overlap an input at all, not even as the
    # same pointer (a binary32 output slot covers two input slots)
    big = torch.zeros(256, dtype=torch.bfloat16, device=DEV)
    h = [big[0:32], big[64:96]]
    hp = _ptr_array([t.data_ptr() for t in h])
    wide = torch.zeros(32, device=DEV)
    g32 = tc.Group([32])
    assert L.tc_reduce_ex(g32.handle, 2, hp, tc.TC_BF16, h[0].data_ptr(), 0, s) == tc.TC_EINVAL
    assert "bfloat16" in tc.last_error()
    assert L.tc_reduce_ex(g32.handle, 2, hp, tc.TC_BF16, big[80:].data_ptr(), 0, s) == tc.TC_EINVAL
    assert L.tc_reduce_ex(g32.handle, 2, hp, tc.TC_BF16, wide.data_ptr(), 0, s) == tc.TC_OK
    fp = _ptr_array([wide.data_ptr(), a[0].data_ptr()])
    assert L.tc_reduce_ex(tc.Group([16]).handle, 2, fp, tc.TC_F32, wide.data_ptr(), 0, s) == tc.TC_OK
    xc = torch.zeros(16, device=DEV)
    xp = _ptr_array([t.data_ptr() for t in a])
    gp = _ptr_array([t.data_ptr() for t in [out, out, out]])
    assert L.easgd_step(g.handle, 3, xp, gp, a[0].data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL  # x_c aliases x
    assert L.easgd_step(g.handle, 3, xp, xp, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL    # grad aliases x
    assert L.easgd_step(g.handle, 3, xp, gp, xc.data_ptr(), float("nan"), 0.5, s) == tc.TC_EINVAL
    assert L.easgd_step(g.handle, 3, xp, gp, xc.data_ptr(), 0.1, float("inf"), s) == tc.TC_EINVAL
    dup = _ptr_array([a[0].data_ptr(), a[0].data_ptr(), a[2].data_ptr()])
    assert L.easgd_step(g.handle, 3, dup, gp, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_EINVAL  # x not distinct
    assert L.easgd_step(g.handle, 3, xp, gp, xc.data_ptr(), 0.1, 0.5, s) == tc.TC_OK
    with pytest.raises(tc.TCError):
        tc.Group([3, -1])
    arr = tc._ptr_array([a[0].data_ptr()])
    assert not L.tc_tensorlist_create(g.handle, 0, arr, tc.TC_F32)   # K = 0
    assert not L.tc_tensorlist_create(g.handle, 1, arr, 9)           # unknown dtype
    null = tc._ptr_array([0])
    assert not L.tc_tensorlist_create(g.handle, 1, null, tc.TC_F32)  # NULL non-empty tensor
    assert "NULL" in tc.last_error()
    torch.cuda.synchronize()
