"""Tensor-group collectives and the fused elastic-averaging SGD step on
AMD MI355X (gfx950).

A thin ctypes binding of the C ABI declared in ``include/tc.h``: every
function here marshals torch tensors into device pointers, sizes and the
current HIP stream, and calls the library of the same name.  All arithmetic
runs in the library's HIP kernels; there is no CPU or PyTorch fallback, and
loading fails loudly when the library has not been built.

    g = Group(sizes)                        # tc_group_create
    tl = TensorList(g, [[t00, t01, ...], [t10, ...]])   # tc_tensorlist_create
    pack(tl, flats); unpack(tl, flats)      # tc_pack / tc_unpack
    reduce(g, ins, out, "avg")              # tc_reduce / tc_reduce_ex
    easgd_step(g, xs, gs, xc, eta, rho)     # easgd_step / easgd_step_ex

Schedules and synchronous SGD (separate buffers; *_tensor on the tensor layout):
    sgd_step(g, xs, gs, eta)                # sgd_step
    easgd_period_step(g, xs, gs, xc, eta, rho, t, tau)  # easgd_period_step
    elastic_async(g, xs, xc, order, alpha)  # elastic_async
    sync_sgd_step(g, xs, gs, eta, rescale, broadcast)   # sync_sgd_step
    broadcast(g, src, dsts)                 # tc_broadcast

Tensor layout (the K copies interleaved in one buffer):
    n = tensor_numel(g, K)                  # tc_tensor_numel
    pack_tensor(tl, T); unpack_tensor(tl, T)            # tc_pack_tensor / tc_unpack_tensor
    reduce_tensor(g, K, T, out, "avg")      # tc_reduce_tensor
    easgd_step_tensor(g, K, X, G, xc, eta, rho)         # easgd_step_tensor
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

from .build import LIBRARY

TC_SUM, TC_AVG = 0, 1
TC_F32, TC_BF16 = 0, 1
TC_OK, TC_EINVAL, TC_ENOMEM, TC_EHIP, TC_EUNSUPPORTED = 0, -1, -2, -3, -4
TC_MAX_K = 64

_OPS = {"sum": TC_SUM, "avg": TC_AVG, TC_SUM: TC_SUM, TC_AVG: TC_AVG}
_DTYPES = {torch.float32: TC_F32, torch.bfloat16: TC_BF16}


class TCError(RuntimeError):
    """A C-ABI call returned an error status."""

    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status


_VP = ctypes.c_void_p
_VPP = ctypes.POINTER(ctypes.c_void_p)
_lib = None


def lib(path: str = LIBRARY) -> ctypes.CDLL:
    """The loaded HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library {path} is not built; run __graft_entry__.build() "
                           f"or python -m paper_1801_03855_amd.build")
    L = ctypes.CDLL(path)
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    sig = {
        "tc_last_error": (ctypes.c_char_p, []),
        "tc_version": (i32, []),
        "tc_group_create": (_VP, [ctypes.POINTER(i64), i32]),
        "tc_group_destroy": (None, [_VP]),
        "tc_group_numel": (i64, [_VP]),
        "tc_group_ntensors": (i32, [_VP]),
        "tc_group_offsets": (i32, [_VP, ctypes.POINTER(i64)]),
        "tc_tensorlist_create": (_VP, [_VP, i32, _VPP, i32]),
        "tc_tensorlist_destroy": (None, [_VP]),
        "tc_pack": (i32, [_VP, _VPP, _VP]),
        "tc_unpack": (i32, [_VP, _VPP, _VP]),
        "tc_reduce": (i32, [_VP, i32, _VPP, _VP, i32, _VP]),
        "tc_reduce_ex": (i32, [_VP, i32, _VPP, i32, _VP, i32, _VP]),
        "easgd_step": (i32, [_VP, i32, _VPP, _VPP, _VP, f32, f32, _VP]),
        "easgd_step_ex": (i32, [_VP, i32, _VPP, _VPP, i32, _VP, f32, f32, _VP]),
        "reduce_easgd_step": (i32, [_VP, i32, _VPP, _VPP, i32, _VP, _VP, i32, f32, f32, _VP]),
        "tc_tensor_numel": (i64, [_VP, i32]),
        "tc_pack_tensor": (i32, [_VP, _VP, _VP]),
        "tc_unpack_tensor": (i32, [_VP, _VP, _VP]),
        "tc_reduce_tensor": (i32, [_VP, i32, _VP, i32, _VP, i32, _VP]),
        "easgd_step_tensor": (i32, [_VP, i32, _VP, _VP, i32, _VP, f32, f32, _VP]),
        "reduce_easgd_step_tensor": (i32, [_VP, i32, _VP, _VP, i32, _VP, _VP, i32, f32, f32, _VP]),
        "sgd_step": (i32, [_VP, i32, _VPP, _VPP, i32, f32, _VP]),
        "sgd_step_tensor": (i32, [_VP, i32, _VP, _VP, i32, f32, _VP]),
        "easgd_period_step": (i32, [_VP, i32, _VPP, _VPP, i32, _VP, f32, f32, i64, i32, _VP]),
        "easgd_period_step_tensor": (i32, [_VP, i32, _VP, _VP, i32, _VP, f32, f32, i64, i32, _VP]),
        "elastic_async": (i32, [_VP, i32, _VPP, _VP, ctypes.POINTER(i32), i32, f32, _VP]),
        "elastic_async_tensor": (i32, [_VP, i32, _VP, _VP, ctypes.POINTER(i32), i32, f32, _VP]),
        "sync_sgd_step": (i32, [_VP, i32, _VPP, _VPP, i32, f32, f32, i32, _VP]),
        "sync_sgd_step_tensor": (i32, [_VP, i32, _VP, _VP, i32, f32, f32, i32, _VP]),
        "tc_broadcast": (i32, [_VP, i32, _VP, _VPP, i32, _VP]),
        "tc_broadcast_tensor": (i32, [_VP, i32, _VP, _VP, i32, _VP]),
        "easgd_pipeline_tensor": (i32, [_VP, _VP, _VP, _VP, _VP, _VP, f32, f32, _VP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def last_error() -> str:
    return lib().tc_last_error().decode()


def _check(status: int) -> None:
    if status != TC_OK:
        raise TCError(status, last_error())


def _ptr_array(ptrs: Sequence[Optional[int]]):
    arr = (ctypes.c_void_p * max(1, len(ptrs)))()
    for i, p in enumerate(ptrs):
        arr[i] = p if p else None
    return arr


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t: torch.Tensor, n: int, dtypes=(torch.float32,), what: str = "tensor") -> int:
    if not t.is_cuda:
        raise ValueError(f"{what} must be a GPU tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{what} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous() or t.numel() < n:
        raise ValueError(f"{what} must be contiguous with at least {n} elements (has {t.numel()})")
    return t.data_ptr()


class Group:
    """A tensor group: n layer sizes, one flat index space of N elements."""

    def __init__(self, sizes: Sequence[int]):
        arr = (ctypes.c_int64 * len(sizes))(*[int(s) for s in sizes])
        h = lib().tc_group_create(arr, len(sizes))
        if not h:
            raise TCError(TC_EINVAL, last_error())
        self._h = h
        self.sizes = [int(s) for s in sizes]
        self.n = lib().tc_group_ntensors(h)
        self.numel = lib().tc_group_numel(h)

    @property
    def handle(self):
        return self._h

    def offsets(self):
        out = (ctypes.c_int64 * (self.n + 1))()
        _check(lib().tc_group_offsets(self._h, out))
        return list(out)

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.tc_group_destroy(h)


class TensorList:
    """K copies of a group as separate tensors: tensors[k][t] is tensor t of
    copy k (a contiguous GPU tensor of sizes[t] elements)."""

    def __init__(self, group: Group, tensors: Sequence[Sequence[torch.Tensor]]):
        K = len(tensors)
        if K < 1:
            raise ValueError("a tensor list needs at least one copy")
        dt = None
        ptrs = []
        for k, copy in enumerate(tensors):
            if len(copy) != group.n:
                raise ValueError(f"copy {k} has {len(copy)} tensors, the group has {group.n}")
            for t, (x, s) in enumerate(zip(copy, group.sizes)):
                dt = dt or x.dtype
                if x.dtype != dt or x.dtype not in _DTYPES:
                    raise TypeError(f"tensor ({k},{t}) has dtype {x.dtype}")
                if x.numel() != s:
                    raise ValueError(f"tensor ({k},{t}) has {x.numel()} elements, expected {s}")
                ptrs.append(_dev_ptr(x, s, (dt,), f"tensor ({k},{t})") if s else 0)
        self.group, self.K, self.dtype = group, K, dt
        self._keep = [list(c) for c in tensors]
        h = lib().tc_tensorlist_create(group.handle, K, _ptr_array(ptrs), _DTYPES[dt])
        if not h:
            raise TCError(TC_EINVAL, last_error())
        self._h = h

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.tc_tensorlist_destroy(h)


def _flat_ptrs(tl: TensorList, flats: Sequence[torch.Tensor]):
    if len(flats) != tl.K:
        raise ValueError(f"need {tl.K} flat buffers, got {len(flats)}")
    n = tl.group.numel
    return _ptr_array([_dev_ptr(f, n, (tl.dtype,), f"flat[{k}]") for k, f in enumerate(flats)])


def pack(tl: TensorList, flats: Sequence[torch.Tensor], stream=None) -> None:
    """flats[k][offsets[t] + e] = tensors[k][t][e] (tc_pack)."""
    _check(lib().tc_pack(tl.handle, _flat_ptrs(tl, flats), _stream(stream)))


def unpack(tl: TensorList, flats: Sequence[torch.Tensor], stream=None) -> None:
    """tensors[k][t][e] = flats[k][offsets[t] + e] (tc_unpack)."""
    _check(lib().tc_unpack(tl.handle, _flat_ptrs(tl, flats), _stream(stream)))


def reduce(group: Group, ins: Sequence[torch.Tensor], out: torch.Tensor, op="avg", stream=None) -> None:
    """out = sum (or average) of the K flat copies ins (tc_reduce_ex)."""
    n = group.numel
    dt = ins[0].dtype
    if dt not in _DTYPES:
        raise TypeError(f"inputs have dtype {dt}")
    p = _ptr_array([_dev_ptr(t, n, (dt,), f"in[{i}]") for i, t in enumerate(ins)])
    _check(lib().tc_reduce_ex(group.handle, len(ins), p, _DTYPES[dt],
                              _dev_ptr(out, n, (torch.float32,), "out"), _OPS[op], _stream(stream)))


def easgd_step(group: Group, xs: Sequence[torch.Tensor], gs: Sequence[torch.Tensor], xc: torch.Tensor,
               eta: float, rho: float, stream=None) -> None:
    """One fused elastic-averaging SGD step, in place on xs and xc
    (easgd_step_ex)."""
    n = group.numel
    if len(xs) != len(gs):
        raise ValueError("need one gradient per worker")
    gdt = gs[0].dtype
    if gdt not in _DTYPES:
        raise TypeError(f"gradients have dtype {gdt}")
    xp = _ptr_array([_dev_ptr(t, n, (torch.float32,), f"x[{i}]") for i, t in enumerate(xs)])
    gp = _ptr_array([_dev_ptr(t, n, (gdt,), f"grad[{i}]") for i, t in enumerate(gs)])
    _check(lib().easgd_step_ex(group.handle, len(xs), xp, gp, _DTYPES[gdt],
                               _dev_ptr(xc, n, (torch.float32,), "x_c"), float(eta), float(rho),
                               _stream(stream)))


def reduce_easgd_step(group: Group, xs: Sequence[torch.Tensor], gs: Sequence[torch.Tensor], xc: torch.Tensor,
                      out: torch.Tensor, eta: float, rho: float, op="avg", stream=None) -> None:
    """The sum (or average) of the gradients into out and the fused step on
    xs and xc, in one pass (reduce_easgd_step)."""
    n = group.numel
    if len(xs) != len(gs):
        raise ValueError("need one gradient per worker")
    gdt = gs[0].dtype
    if gdt not in _DTYPES:
        raise TypeError(f"gradients have dtype {gdt}")
    xp = _ptr_array([_dev_ptr(t, n, (torch.float32,), f"x[{i}]") for i, t in enumerate(xs)])
    gp = _ptr_array([_dev_ptr(t, n, (gdt,), f"grad[{i}]") for i, t in enumerate(gs)])
    _check(lib().reduce_easgd_step(group.handle, len(xs), xp, gp, _DTYPES[gdt],
                                   _dev_ptr(xc, n, (torch.float32,), "x_c"),
                                   _dev_ptr(out, n, (torch.float32,), "out"), _OPS[op], float(eta), float(rho),
                                   _stream(stream)))


# --------------------------------------------------------------- tensor layout

def tensor_numel(group: Group, K: int) -> int:
    n = lib().tc_tensor_numel(group.handle, K)
    if n < 0:
        raise TCError(TC_EINVAL, f"bad K = {K}")
    return n


def pack_tensor(tl: TensorList, tensor: torch.Tensor, stream=None) -> None:
    """K copies' separate tensors -> one tensor-layout buffer (tc_pack_tensor)."""
    n = tensor_numel(tl.group, tl.K)
    _check(lib().tc_pack_tensor(tl.handle, _dev_ptr(tensor, n, (tl.dtype,), "tensor"), _stream(stream)))


def unpack_tensor(tl: TensorList, tensor: torch.Tensor, stream=None) -> None:
    """One tensor-layout buffer -> the K copies' separate tensors (tc_unpack_tensor)."""
    n = tensor_numel(tl.group, tl.K)
    _check(lib().tc_unpack_tensor(tl.handle, _dev_ptr(tensor, n, (tl.dtype,), "tensor"), _stream(stream)))


def reduce_tensor(group: Group, K: int, tensor: torch.Tensor, out: torch.Tensor, op="avg", stream=None) -> None:
    """out = sum (or average) of the K copies in a tensor-layout buffer (tc_reduce_tensor)."""
    dt = tensor.dtype
    if dt not in _DTYPES:
        raise TypeError(f"input has dtype {dt}")
    p = _dev_ptr(tensor, tensor_numel(group, K), (dt,), "in")
    _check(lib().tc_reduce_tensor(group.handle, K, p, _DTYPES[dt], _dev_ptr(out, group.numel, (torch.float32,), "out"),
                                  _OPS[op], _stream(stream)))


def easgd_step_tensor(group: Group, K: int, x: torch.Tensor, g: torch.Tensor, xc: torch.Tensor,
                      eta: float, rho: float, stream=None) -> None:
    """One fused elastic-averaging SGD step on tensor-layout workers x and
    gradients g, in place on x and xc (easgd_step_tensor)."""
    n = tensor_numel(group, K)
    gdt = g.dtype
    if gdt not in _DTYPES:
        raise TypeError(f"gradients have dtype {gdt}")
    _check(lib().easgd_step_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"),
                                   _dev_ptr(g, n, (gdt,), "grad"), _DTYPES[gdt],
                                   _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), float(eta), float(rho),
                                   _stream(stream)))


def reduce_easgd_step_tensor(group: Group, K: int, x: torch.Tensor, g: torch.Tensor, xc: torch.Tensor,
                             out: torch.Tensor, eta: float, rho: float, op="avg", stream=None) -> None:
    """reduce_easgd_step on tensor-layout workers x and gradients g
    (reduce_easgd_step_tensor)."""
    n = tensor_numel(group, K)
    gdt = g.dtype
    if gdt not in _DTYPES:
        raise TypeError(f"gradients have dtype {gdt}")
    _check(lib().reduce_easgd_step_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"),
                                          _dev_ptr(g, n, (gdt,), "grad"), _DTYPES[gdt],
                                          _dev_ptr(xc, group.numel, (torch.float32,), "x_c"),
                                          _dev_ptr(out, group.numel, (torch.float32,), "out"), _OPS[op],
                                          float(eta), float(rho), _stream(stream)))


# ----------------------------------------------- schedules and synchronous SGD

def _gdt(gs_or_g) -> torch.dtype:
    dt = gs_or_g[0].dtype if isinstance(gs_or_g, (list, tuple)) else gs_or_g.dtype
    if dt not in _DTYPES:
        raise TypeError(f"gradients have dtype {dt}")
    return dt


def _workers(group: Group, xs):
    return _ptr_array([_dev_ptr(t, group.numel, (torch.float32,), f"x[{i}]") for i, t in enumerate(xs)])


def _grads(group: Group, gs, dt):
    return _ptr_array([_dev_ptr(t, group.numel, (dt,), f"grad[{i}]") for i, t in enumerate(gs)])


def sgd_step(group: Group, xs, gs, eta: float, stream=None) -> None:
    """x_i -= eta * g_i for every worker, in place (sgd_step)."""
    dt = _gdt(gs)
    _check(lib().sgd_step(group.handle, len(xs), _workers(group, xs), _grads(group, gs, dt), _DTYPES[dt],
                          float(eta), _stream(stream)))


def sgd_step_tensor(group: Group, K: int, x, g, eta: float, stream=None) -> None:
    dt = _gdt(g)
    n = tensor_numel(group, K)
    _check(lib().sgd_step_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"), _dev_ptr(g, n, (dt,), "grad"),
                                 _DTYPES[dt], float(eta), _stream(stream)))


def easgd_period_step(group: Group, xs, gs, xc, eta: float, rho: float, iteration: int, tau: int, stream=None) -> None:
    """The elastic step when iteration % tau == 0, plain SGD otherwise."""
    dt = _gdt(gs)
    _check(lib().easgd_period_step(group.handle, len(xs), _workers(group, xs), _grads(group, gs, dt), _DTYPES[dt],
                                   _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), float(eta), float(rho),
                                   int(iteration), int(tau), _stream(stream)))


def easgd_period_step_tensor(group: Group, K: int, x, g, xc, eta: float, rho: float, iteration: int, tau: int,
                             stream=None) -> None:
    dt = _gdt(g)
    n = tensor_numel(group, K)
    _check(lib().easgd_period_step_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"),
                                          _dev_ptr(g, n, (dt,), "grad"), _DTYPES[dt],
                                          _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), float(eta), float(rho),
                                          int(iteration), int(tau), _stream(stream)))


def _order(order):
    o = [int(v) for v in order]
    return (ctypes.c_int32 * max(1, len(o)))(*o), len(o)


def elastic_async(group: Group, xs, xc, order, alpha: float, stream=None) -> None:
    """Elastic exchanges of the workers in `order`, one at a time (elastic_async)."""
    arr, R = _order(order)
    _check(lib().elastic_async(group.handle, len(xs), _workers(group, xs),
                               _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), arr, R, float(alpha),
                               _stream(stream)))


def elastic_async_tensor(group: Group, K: int, x, xc, order, alpha: float, stream=None) -> None:
    arr, R = _order(order)
    n = tensor_numel(group, K)
    _check(lib().elastic_async_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"),
                                      _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), arr, R, float(alpha),
                                      _stream(stream)))


def sync_sgd_step(group: Group, xs, gs, eta: float, rescale: float, broadcast: bool = False, stream=None) -> None:
    """Synchronous SGD through pushpull (sync_sgd_step)."""
    dt = _gdt(gs)
    _check(lib().sync_sgd_step(group.handle, len(xs), _workers(group, xs), _grads(group, gs, dt), _DTYPES[dt],
                               float(eta), float(rescale), int(bool(broadcast)), _stream(stream)))


def sync_sgd_step_tensor(group: Group, K: int, x, g, eta: float, rescale: float, broadcast: bool = False,
                         stream=None) -> None:
    dt = _gdt(g)
    n = tensor_numel(group, K)
    _check(lib().sync_sgd_step_tensor(group.handle, K, _dev_ptr(x, n, (torch.float32,), "x"),
                                      _dev_ptr(g, n, (dt,), "grad"), _DTYPES[dt], float(eta), float(rescale),
                                      int(bool(broadcast)), _stream(stream)))


def broadcast(group: Group, src, dsts, stream=None) -> None:
    """dsts[i] = src for every copy (tc_broadcast)."""
    dt = _gdt(src)
    p = _ptr_array([_dev_ptr(t, group.numel, (dt,), f"dst[{i}]") for i, t in enumerate(dsts)])
    _check(lib().tc_broadcast(group.handle, len(dsts), _dev_ptr(src, group.numel, (dt,), "src"), p, _DTYPES[dt],
                              _stream(stream)))


def broadcast_tensor(group: Group, K: int, src, dst, stream=None) -> None:
    dt = _gdt(src)
    _check(lib().tc_broadcast_tensor(group.handle, K, _dev_ptr(src, group.numel, (dt,), "src"),
                                     _dev_ptr(dst, tensor_numel(group, K), (dt,), "dst"), _DTYPES[dt],
                                     _stream(stream)))


# ----------------------------------------------------------------- pipeline

def easgd_pipeline_tensor(grads: TensorList, params: TensorList, g_tensor: Optional[torch.Tensor],
                          gbar: torch.Tensor, x: torch.Tensor, xc: torch.Tensor, eta: float, rho: float,
                          stream=None) -> None:
    """The whole step in one pass (easgd_pipeline_tensor): pack the gradient
    lists into g_tensor (skipped when None), gbar = their AVG, the fused
    elastic step on the tensor-layout workers x and the center xc, and the
    new workers unpacked into the parameter lists."""
    if grads.group is not params.group:
        raise ValueError("the gradient and parameter lists must share one group")
    group, K = grads.group, grads.K
    n = tensor_numel(group, K)
    gt = _dev_ptr(g_tensor, n, (grads.dtype,), "g_tensor") if g_tensor is not None else None
    _check(lib().easgd_pipeline_tensor(grads.handle, params.handle, gt,
                                       _dev_ptr(gbar, group.numel, (torch.float32,), "gbar"),
                                       _dev_ptr(x, n, (torch.float32,), "x"),
                                       _dev_ptr(xc, group.numel, (torch.float32,), "x_c"), float(eta), float(rho),
                                       _stream(stream)))
