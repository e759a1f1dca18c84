"""Pins of the CPU oracle: checks against what the paper's definitions and
plain mathematics fix, independent of the oracle's own code.

Each pin is a function ``pin_*(orc)`` that raises AssertionError when the
oracle disagrees.  They are run on the real oracle (tests/test_oracle_pins.py)
and on deliberately broken copies of its source (tests/test_oracle_mutants.py),
where at least one pin must fail for every planted mistake.

Run as a script (``python -m tests.pins LIBRARY``) it loads the given oracle
library, runs every pin and prints the names of the failing ones as JSON.
"""

from __future__ import annotations

import json
import math
import sys
from fractions import Fraction

import numpy as np

# Known totals of the named groups: the parameter counts of ResNet-50 v1
# (25,557,032) and VGG-16 (138,357,544) as widely published for these
# architectures, and the sum of the tiny group's eight sizes.
KNOWN_TOTALS = {"tiny": 7_392, "resnet50": 25_557_032, "vgg16": 138_357_544}


def _rng(seed):
    return np.random.default_rng(seed)


def _f32(rng, n, lo_exp=-8, hi_exp=8):
    """Random binary32 values with exponents in [lo_exp, hi_exp)."""
    m = rng.uniform(1.0, 2.0, n)
    e = rng.integers(lo_exp, hi_exp, n)
    s = rng.choice([-1.0, 1.0], n)
    return (s * np.ldexp(m, e)).astype(np.float32)


# ---------------------------------------------------------------- offsets

def pin_offsets_cumsum(orc):
    """Offsets are the exclusive prefix sums of the sizes (numpy.cumsum)."""
    rng = _rng(1)
    for n in (1, 2, 7, 161, 1000):
        sizes = rng.integers(0, 5000, n)
        sizes[rng.random(n) < 0.1] = 0
        off = orc.offsets(sizes)
        assert off[0] == 0
        assert np.array_equal(off[1:], np.cumsum(sizes)), n


def pin_offsets_known_totals(orc):
    """The named groups' flat lengths equal their published parameter counts."""
    from paper_1801_03855_amd import workloads
    for name, total in KNOWN_TOTALS.items():
        off = orc.offsets(workloads.group_sizes(name))
        assert off[-1] == total, (name, off[-1])
    assert len(workloads.group_sizes("resnet50")) == 161
    assert len(workloads.group_sizes("vgg16")) == 32


# ----------------------------------------------------------- pack/unpack

def _tensors(rng, sizes, dtype):
    if dtype == np.float32:
        return [_f32(rng, s) for s in sizes]
    return [rng.integers(0, 1 << 16, s, dtype=np.uint16) for s in sizes]


def pin_pack_is_concatenation(orc):
    """pack == numpy.concatenate of the flattened tensors, bit for bit."""
    rng = _rng(2)
    for dtype in (np.float32, np.uint16):
        sizes = [5, 0, 1, 17, 0, 64, 3]
        ts = _tensors(rng, sizes, dtype)
        if dtype == np.float32:
            ts[0][:3] = [np.float32(-0.0), np.float32(np.nan), np.float32(np.inf)]
        flat = orc.pack(ts)
        ref = np.concatenate(ts)
        assert flat.dtype == ref.dtype
        assert np.array_equal(flat.view(np.uint8), ref.view(np.uint8))


def pin_unpack_is_split(orc):
    """unpack == numpy.split at the offsets, and unpack(pack(T)) == T."""
    rng = _rng(3)
    for dtype in (np.float32, np.uint16):
        sizes = [3, 0, 9, 1, 40]
        flat = _tensors(rng, [sum(sizes)], dtype)[0]
        parts = orc.unpack(flat, sizes)
        ref = np.split(flat, np.cumsum(sizes)[:-1])
        assert len(parts) == len(ref)
        for a, b in zip(parts, ref):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
        again = orc.unpack(orc.pack(parts), sizes)
        for a, b in zip(again, parts):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def pin_tensor_layout_is_slot_transpose(orc):
    """The tensor layout is numpy's (K, S, 4) -> (S, K, 4) transpose of the
    copies zero-padded to S = ceil(N/4) slots, bit for bit; padding keeps
    its fill; the inverse recovers the copies."""
    rng = _rng(19)
    for K, N in ((1, 9), (3, 10), (4, 16), (8, 37), (16, 1), (5, 4)):
        for dtype in (np.float32, np.uint16):
            copies = _tensors(rng, [N] * K, dtype)
            S = (N + 3) // 4
            padded = np.zeros((K, S * 4), dtype=dtype)
            for i, c in enumerate(copies):
                padded[i, :N] = c
            ref = padded.reshape(K, S, 4).transpose(1, 0, 2).reshape(-1)
            got = orc.tensor_from_copies(copies, fill=0)
            assert np.array_equal(got.view(np.uint8), ref.view(np.uint8)), (K, N, dtype)
            back = orc.copies_from_tensor(got, K, N)
            for a, b in zip(back, copies):
                assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (K, N)
            filled = orc.tensor_from_copies(copies, fill=7)
            mask = np.zeros((K, S * 4), dtype=bool)
            mask[:, N:] = True
            mask = mask.reshape(K, S, 4).transpose(1, 0, 2).reshape(-1)
            assert np.all(filled[mask] == 7) and np.array_equal(filled[~mask], ref[~mask])


# ----------------------------------------------------------------- bf16

def pin_bf16_decode_all_codes(orc):
    """Every one of the 65,536 bfloat16 codes decodes to torch's value."""
    import torch
    codes = np.arange(1 << 16, dtype=np.uint16)
    got = orc.widen(codes)
    ref = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))
    # a few codes by hand: 1.0, -2.0, 3.140625, smallest subnormal 2^-133
    for code, val in ((0x3F80, 1.0), (0xC000, -2.0), (0x4049, 3.140625), (0x0001, 2.0 ** -133)):
        assert orc.widen(np.array([code], dtype=np.uint16))[0] == val, hex(code)


def pin_f32_widen_exact(orc):
    rng = _rng(4)
    a = _f32(rng, 1000, -140, 120)
    assert np.array_equal(orc.widen(a), a.astype(np.float64))


# ---------------------------------------------------------------- reduce

def pin_reduce_k2_single_add(orc):
    """K=2: the sum of two binary32 numbers is exact in binary64 (when their
    exponents differ by < 29), so it equals the rational sum; AVG is half."""
    rng = _rng(5)
    a, b = _f32(rng, 2000), _f32(rng, 2000)
    s = orc.reduce([a, b], 0)
    m = orc.reduce([a, b], 1)
    for i in range(0, 2000, 7):
        exact = Fraction(float(a[i])) + Fraction(float(b[i]))
        assert Fraction(s[i]) == exact, i
        assert Fraction(m[i]) == exact / 2, i


def pin_reduce_integer_exact(orc):
    """Integer-valued inputs: SUM is the int64 sum in any order; AVG is the
    correctly rounded quotient sum/K."""
    rng = _rng(6)
    for K in (1, 2, 3, 4, 5, 7, 8, 16, 33, 64):
        ins = [rng.integers(-1024, 1025, 257).astype(np.float32) for _ in range(K)]
        isum = np.sum(np.stack([x.astype(np.int64) for x in ins]), axis=0)
        s = orc.reduce(ins, 0)
        assert np.array_equal(s, isum.astype(np.float64)), K
        m = orc.reduce(ins, 1)
        ref = np.array([float(Fraction(int(v), K)) for v in isum])
        assert np.array_equal(m, ref), K
        perm = list(rng.permutation(K))
        assert np.array_equal(orc.reduce([ins[p] for p in perm], 0), s), K


def pin_reduce_identical_copies(orc):
    """AVG of K identical copies is the copy; SUM is K times it."""
    rng = _rng(7)
    v = _f32(rng, 999)
    for K in (1, 2, 3, 4, 6, 8, 16, 64):
        assert np.array_equal(orc.reduce([v] * K, 1), v.astype(np.float64)), K
        assert np.array_equal(orc.reduce([v] * K, 0), K * v.astype(np.float64)), K


def pin_reduce_rational_bound(orc):
    """General inputs: within binary64 rounding of the rational sum."""
    rng = _rng(8)
    for K in (3, 5, 16):
        ins = [_f32(rng, 64, -30, 30) for _ in range(K)]
        s = orc.reduce(ins, 0)
        m = orc.reduce(ins, 1)
        for j in range(64):
            vals = [Fraction(float(x[j])) for x in ins]
            exact = sum(vals, Fraction(0))
            mag = sum(abs(v) for v in vals)
            bound = K * mag * Fraction(1, 2 ** 52)
            assert abs(Fraction(s[j]) - exact) <= bound, (K, j)
            assert abs(Fraction(m[j]) - exact / K) <= bound / K + abs(exact / K) * Fraction(1, 2 ** 52), (K, j)


def pin_reduce_bf16_equals_widened(orc):
    """A bfloat16 reduction equals the reduction of the same values stored
    as binary32 (decoding is exact)."""
    import torch
    rng = _rng(9)
    K = 16
    f = [_f32(rng, 300) for _ in range(K)]
    codes = [torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16) for x in f]
    back = [torch.from_numpy(c.view(np.int16)).view(torch.bfloat16).float().numpy() for c in codes]
    for op in (0, 1):
        assert np.array_equal(orc.reduce(codes, op), orc.reduce(back, op))


# ------------------------------------------------------------ easgd step

def _state(rng, K, n, scale=0.05):
    xs = [rng.normal(0, scale, n).astype(np.float32).astype(np.float64) for _ in range(K)]
    xc = rng.normal(0, scale, n).astype(np.float32).astype(np.float64)
    gs = [rng.normal(0, 0.01, n).astype(np.float32) for _ in range(K)]
    return xs, xc, gs


def _close(a, b, rel=1e-13, mag=None):
    mag = np.maximum(np.abs(b), 1e-300) if mag is None else mag
    return np.all(np.abs(a - b) <= rel * mag)


def pin_easgd_rho0_is_sgd(orc):
    """rho = 0: each worker takes the plain SGD step w - eta*g (Sec. 2.1,
    Eq. 1 with dw = -eta*g) and the center does not move."""
    rng = _rng(10)
    for K in (1, 2, 8):
        xs, xc, gs = _state(rng, K, 500)
        x0 = [x.copy() for x in xs]
        c0 = xc.copy()
        eta = 0.05
        orc.easgd_step(xs, gs, xc, eta, 0.0)
        for x, x_old, g in zip(xs, x0, gs):
            assert np.array_equal(x, x_old - eta * g.astype(np.float64)), K
        assert np.array_equal(xc, c0), K


def pin_easgd_eta0_identity(orc):
    rng = _rng(11)
    xs, xc, gs = _state(rng, 4, 300)
    x0 = [x.copy() for x in xs]
    c0 = xc.copy()
    orc.easgd_step(xs, gs, xc, 0.0, 2.5)
    assert all(np.array_equal(a, b) for a, b in zip(xs, x0))
    assert np.array_equal(xc, c0)


def pin_easgd_consensus_fixed_point(orc):
    """All workers at the center and zero gradients: nothing moves."""
    rng = _rng(12)
    c = rng.normal(0, 1, 200).astype(np.float32).astype(np.float64)
    for K in (1, 3, 16):
        xs = [c.copy() for _ in range(K)]
        xc = c.copy()
        gs = [np.zeros(200, np.float32) for _ in range(K)]
        orc.easgd_step(xs, gs, xc, 0.05, 0.9 / (K * 0.05))
        assert all(np.array_equal(x, c) for x in xs) and np.array_equal(xc, c), K


def pin_easgd_conservation(orc):
    """Zero gradients: sum_i x_i + x_c is invariant, because every worker's
    elastic move is matched by an equal and opposite move of the center."""
    rng = _rng(13)
    for K in (1, 2, 5, 8, 16):
        xs, xc, _ = _state(rng, K, 400)
        gs = [np.zeros(400, np.float32) for _ in range(K)]
        before = sum(xs) + xc
        mag = sum(np.abs(x) for x in xs) + np.abs(xc)
        orc.easgd_step(xs, gs, xc, 0.05, 0.9 / (K * 0.05))
        after = sum(xs) + xc
        assert _close(after, before, 1e-13, mag), K


def pin_easgd_disagreement_decay(orc):
    """Zero gradients: the difference of two workers shrinks by (1 - eta*rho)."""
    rng = _rng(14)
    K, eta, rho = 6, 0.05, 3.0
    xs, xc, _ = _state(rng, K, 400)
    gs = [np.zeros(400, np.float32) for _ in range(K)]
    d0 = [xs[i] - xs[0] for i in range(K)]
    mag = sum(np.abs(x) for x in xs)
    orc.easgd_step(xs, gs, xc, eta, rho)
    for i in range(1, K):
        assert _close(xs[i] - xs[0], (1 - eta * rho) * d0[i], 1e-13, mag), i


def pin_easgd_center_gap(orc):
    """Zero gradients: with m the workers' mean, the gap m - x_c shrinks by
    (1 - eta*rho - K*eta*rho): each worker moves alpha of the gap toward the
    center, the center moves K*alpha of it toward the workers."""
    rng = _rng(15)
    for K, eta, rho in ((1, 0.05, 2.0), (4, 0.05, 4.5), (8, 0.05, 2.25), (16, 0.1, 0.3)):
        xs, xc, _ = _state(rng, K, 400)
        gs = [np.zeros(400, np.float32) for _ in range(K)]
        e0 = sum(xs) / K - xc
        mag = sum(np.abs(x) for x in xs) + np.abs(xc)
        orc.easgd_step(xs, gs, xc, eta, rho)
        e1 = sum(xs) / K - xc
        a = eta * rho
        assert _close(e1, (1 - a - K * a) * e0, 1e-12, mag), K


def pin_easgd_gradient_term(orc):
    """The gradient enters worker i only, as -eta*g_i (Sec. 2.1), and does
    not move the center."""
    rng = _rng(16)
    K, eta, rho = 4, 0.05, 4.5
    xs, xc, gs = _state(rng, K, 300)
    xa, ca = [x.copy() for x in xs], xc.copy()
    zeros = [np.zeros(300, np.float32) for _ in range(K)]
    orc.easgd_step(xs, gs, xc, eta, rho)
    orc.easgd_step(xa, zeros, ca, eta, rho)
    mag = sum(np.abs(x) for x in xa) + 1e-3
    for i in range(K):
        assert _close(xs[i] - xa[i], -eta * gs[i].astype(np.float64), 1e-12, mag), i
    assert np.array_equal(xc, ca)


def pin_easgd_iterated_closed_form(orc):
    """Identical workers, zero gradients, T steps: x - x_c = (1 - a - K a)^T
    times its start; the mean of x and the center obey the 2x2 linear map."""
    rng = _rng(17)
    K, eta, rho, T = 4, 0.05, 1.0, 10
    x = rng.normal(0, 0.05, 100)
    xs = [x.copy() for _ in range(K)]
    xc = rng.normal(0, 0.05, 100)
    e0 = x - xc
    gs = [np.zeros(100, np.float32) for _ in range(K)]
    orc.easgd_step(xs, gs, xc, eta, rho, steps=T)
    a = eta * rho
    assert _close(xs[0] - xc, (1 - a - K * a) ** T * e0, 1e-9, np.abs(e0) + 1e-300)


def pin_easgd_bf16_equals_widened(orc):
    """A step with bfloat16 gradients equals the step with the same values
    stored as binary32."""
    import torch
    rng = _rng(18)
    K = 16
    xs, xc, gs = _state(rng, K, 250)
    codes = [torch.from_numpy(g).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16) for g in gs]
    back = [torch.from_numpy(c.view(np.int16)).view(torch.bfloat16).float().numpy() for c in codes]
    xa, ca = [x.copy() for x in xs], xc.copy()
    orc.easgd_step(xs, codes, xc, 0.05, 1.125)
    orc.easgd_step(xa, back, ca, 0.05, 1.125)
    assert all(np.array_equal(a, b) for a, b in zip(xs, xa)) and np.array_equal(xc, ca)


# ------------------------------------------------- schedules and sync SGD

def pin_sgd_step_is_textbook(orc):
    """sgd_step is w - eta*g per worker (Sec. 2.1, Eq. 1), and equals the
    elastic step with rho = 0 on the workers."""
    rng = _rng(20)
    K = 5
    xs, xc, gs = _state(rng, K, 300)
    x0 = [x.copy() for x in xs]
    orc.sgd_step(xs, gs, 0.05)
    for x, x_old, g in zip(xs, x0, gs):
        assert np.array_equal(x, x_old - 0.05 * g.astype(np.float64))
    xe = [x.copy() for x in x0]
    orc.easgd_step(xe, gs, xc.copy(), 0.05, 0.0)
    assert all(np.array_equal(a, b) for a, b in zip(xs, xe))


def pin_elastic_async_conserves_pairs(orc):
    """Each exchange moves worker and center by equal and opposite amounts:
    sum_i x_i + x_c is invariant; the exchanged worker's gap to the center
    shrinks by (1 - 2 alpha)."""
    rng = _rng(21)
    K, alpha = 6, 0.1
    xs, xc, _ = _state(rng, K, 400)
    before = sum(xs) + xc
    mag = sum(np.abs(x) for x in xs) + np.abs(xc)
    order = [3, 0, 5, 3, 1]
    orc.elastic_async(xs, xc, order, alpha)
    assert _close(sum(xs) + xc, before, 1e-13, mag)
    # a single exchange, checked in closed form
    xs2, xc2, _ = _state(rng, K, 400)
    gap = xs2[2] - xc2
    x2, c2 = xs2[2].copy(), xc2.copy()
    orc.elastic_async(xs2, xc2, [2], alpha)
    assert _close(xs2[2] - xc2, (1 - 2 * alpha) * gap, 1e-13, np.abs(x2) + np.abs(c2))
    assert _close(xc2, c2 + alpha * gap, 1e-13, np.abs(x2) + np.abs(c2))


def pin_elastic_async_is_sequential(orc):
    """Exchanges see the center left by the earlier ones: two exchanges of
    the same worker equal the single-exchange map applied twice, and an
    empty order changes nothing."""
    rng = _rng(22)
    xs, xc, _ = _state(rng, 3, 200)
    xa, ca = [x.copy() for x in xs], xc.copy()
    orc.elastic_async(xa, ca, [1, 1], 0.2)
    xb, cb = [x.copy() for x in xs], xc.copy()
    orc.elastic_async(xb, cb, [1], 0.2)
    orc.elastic_async(xb, cb, [1], 0.2)
    assert all(np.array_equal(a, b) for a, b in zip(xa, xb)) and np.array_equal(ca, cb)
    xe, ce = [x.copy() for x in xs], xc.copy()
    orc.elastic_async(xe, ce, [], 0.2)
    assert all(np.array_equal(a, b) for a, b in zip(xe, xs)) and np.array_equal(ce, xc)
    # order matters once two different workers exchange
    xo, co = [x.copy() for x in xs], xc.copy()
    orc.elastic_async(xo, co, [2, 1], 0.2)
    assert not np.allclose(co, ca)


def pin_sync_sgd_identical_steps(orc):
    """Synchronous SGD: every worker takes the same step -eta*rescale*S with
    S the reduce-SUM of the gradients; identical workers stay identical;
    with rescale = 1/K it is SGD with the average gradient."""
    rng = _rng(23)
    K = 4
    x = rng.normal(0, 0.05, 300)
    xs = [x.copy() for _ in range(K)]
    gs = [rng.normal(0, 0.01, 300).astype(np.float32) for _ in range(K)]
    S = orc.sync_sgd(xs, gs, 0.05, 1.0 / K)
    assert np.array_equal(S, orc.reduce(gs, 0))
    assert all(np.array_equal(a, xs[0]) for a in xs)
    avg = orc.reduce(gs, 1)
    assert _close(xs[0], x - 0.05 * avg, 1e-14, np.abs(x) + 0.05 * np.abs(avg))
    # integer gradients: exact
    gi = [rng.integers(-100, 101, 300).astype(np.float32) for _ in range(K)]
    xi = [np.zeros(300) for _ in range(K)]
    S = orc.sync_sgd(xi, gi, 1.0, 1.0)
    assert np.array_equal(xi[1], -np.sum(np.stack([g.astype(np.int64) for g in gi]), axis=0).astype(np.float64))


def pin_broadcast_copies(orc):
    rng = _rng(24)
    for dtype in (np.float32, np.uint16):
        src = _tensors(rng, [77], dtype)[0]
        outs = orc.broadcast(src, 5)
        assert len(outs) == 5 and all(np.array_equal(o.view(np.uint8), src.view(np.uint8)) for o in outs)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]


def run_all(orc):
    """Names of the pins that fail (an exception counts as a failure)."""
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except Exception:  # noqa: BLE001 - any exception is a failed pin
            failed.append(pin.__name__)
    return failed


if __name__ == "__main__":
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from oracle import Oracle
    print(json.dumps(run_all(Oracle(sys.argv[1]))))
