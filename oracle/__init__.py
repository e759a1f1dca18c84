"""CPU oracle (test infrastructure only).

A plain, slow, binary64 C statement of what the tensor-group reduction and the
synchronous elastic-averaging SGD step compute (the source in
``tc_oracle.c`` cites the passages of the paper it follows), plus this ctypes
wrapper.  Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline leg may import it; the product library never does, and the two share
no code.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "tc_oracle.c")
LIBRARY = os.path.join(HERE, "libtc_oracle.so")

F32, BF16 = 0, 1
SUM, AVG = 0, 1

# No contraction of a*b+c into fused operations, no fast-math: the binary64
# arithmetic is exactly what the source says.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(source: str = SOURCE, output: str = LIBRARY, extra: Sequence[str] = ()) -> str:
    """Compile the oracle with gcc into a shared library; returns its path."""
    cmd = ["gcc", *CFLAGS, *extra, "-o", output, source, "-lm"]
    subprocess.run(cmd, check=True)
    return output


_DP = ctypes.POINTER(ctypes.c_double)
_VP = ctypes.c_void_p
_I64P = ctypes.POINTER(ctypes.c_int64)


class Oracle:
    """ctypes view of one compiled oracle library."""

    def __init__(self, path: str = LIBRARY):
        if not os.path.exists(path):
            raise FileNotFoundError(f"oracle library not built: {path}")
        self.path = path
        lib = ctypes.CDLL(path)
        lib.oracle_widen.argtypes = [_VP, ctypes.c_int32, ctypes.c_int64, _DP]
        lib.oracle_widen.restype = None
        lib.oracle_group_offsets.argtypes = [_I64P, ctypes.c_int32, _I64P]
        lib.oracle_group_offsets.restype = ctypes.c_int64
        lib.oracle_pack.argtypes = [ctypes.c_int32, _I64P, ctypes.POINTER(_VP), ctypes.c_int32, _VP]
        lib.oracle_pack.restype = None
        lib.oracle_unpack.argtypes = [ctypes.c_int32, _I64P, _VP, ctypes.c_int32, ctypes.POINTER(_VP)]
        lib.oracle_unpack.restype = None
        lib.oracle_reduce.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_VP),
                                      ctypes.c_int32, ctypes.c_int32, _DP]
        lib.oracle_reduce.restype = None
        lib.oracle_easgd_step.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_DP),
                                          ctypes.POINTER(_VP), ctypes.c_int32, _DP,
                                          ctypes.c_double, ctypes.c_double]
        lib.oracle_easgd_step.restype = None
        lib.oracle_sgd_step.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_DP),
                                        ctypes.POINTER(_VP), ctypes.c_int32, ctypes.c_double]
        lib.oracle_sgd_step.restype = None
        lib.oracle_elastic_async.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_DP), _DP,
                                             ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_double]
        lib.oracle_elastic_async.restype = None
        lib.oracle_sync_sgd.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_DP),
                                        ctypes.POINTER(_VP), ctypes.c_int32, ctypes.c_double,
                                        ctypes.c_double, _DP]
        lib.oracle_sync_sgd.restype = None
        lib.oracle_broadcast.argtypes = [ctypes.c_int32, ctypes.c_int64, _VP, ctypes.c_int32,
                                         ctypes.POINTER(_VP)]
        lib.oracle_broadcast.restype = None
        lib.oracle_tensor_from_copies.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_VP),
                                                  ctypes.c_int32, _VP]
        lib.oracle_tensor_from_copies.restype = None
        lib.oracle_copies_from_tensor.argtypes = [ctypes.c_int32, ctypes.c_int64, _VP, ctypes.c_int32,
                                                  ctypes.POINTER(_VP)]
        lib.oracle_copies_from_tensor.restype = None
        self.lib = lib

    # -- helpers --------------------------------------------------------
    @staticmethod
    def _dtype_code(a: np.ndarray) -> int:
        if a.dtype == np.float32:
            return F32
        if a.dtype == np.uint16:
            return BF16
        raise TypeError(f"stored arrays are float32 or uint16 (bfloat16 codes), got {a.dtype}")

    @staticmethod
    def _ptrs(arrays: Sequence[np.ndarray]):
        arr = (_VP * max(1, len(arrays)))()
        for i, a in enumerate(arrays):
            arr[i] = a.ctypes.data if a.size else None
        return arr

    # -- operations -----------------------------------------------------
    def widen(self, a: np.ndarray) -> np.ndarray:
        a = np.ascontiguousarray(a)
        out = np.empty(a.size, dtype=np.float64)
        self.lib.oracle_widen(a.ctypes.data, self._dtype_code(a), a.size,
                              out.ctypes.data_as(_DP))
        return out

    def offsets(self, sizes: Sequence[int]) -> np.ndarray:
        s = np.ascontiguousarray(np.asarray(sizes, dtype=np.int64))
        off = np.empty(len(s) + 1, dtype=np.int64)
        self.lib.oracle_group_offsets(s.ctypes.data_as(_I64P), len(s), off.ctypes.data_as(_I64P))
        return off

    def pack(self, tensors: Sequence[np.ndarray]) -> np.ndarray:
        tensors = [np.ascontiguousarray(t).reshape(-1) for t in tensors]
        dt = tensors[0].dtype
        sizes = np.array([t.size for t in tensors], dtype=np.int64)
        flat = np.empty(int(sizes.sum()), dtype=dt)
        self.lib.oracle_pack(len(tensors), sizes.ctypes.data_as(_I64P), self._ptrs(tensors),
                             dt.itemsize, flat.ctypes.data)
        return flat

    def unpack(self, flat: np.ndarray, sizes: Sequence[int]) -> List[np.ndarray]:
        flat = np.ascontiguousarray(flat)
        s = np.asarray(sizes, dtype=np.int64)
        outs = [np.empty(int(v), dtype=flat.dtype) for v in s]
        self.lib.oracle_unpack(len(outs), s.ctypes.data_as(_I64P), flat.ctypes.data,
                               flat.dtype.itemsize, self._ptrs(outs))
        return outs

    def reduce(self, ins: Sequence[np.ndarray], op: int) -> np.ndarray:
        ins = [np.ascontiguousarray(a) for a in ins]
        n = ins[0].size
        assert all(a.size == n and a.dtype == ins[0].dtype for a in ins)
        out = np.empty(n, dtype=np.float64)
        self.lib.oracle_reduce(len(ins), n, self._ptrs(ins), self._dtype_code(ins[0]), op,
                               out.ctypes.data_as(_DP))
        return out

    def easgd_step(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray], xc: np.ndarray,
                   eta: float, rho: float, steps: int = 1) -> None:
        """Advance binary64 state (xs, xc) in place by ``steps`` steps with
        the stored gradients gs (float32 arrays or uint16 bfloat16 codes)."""
        K = len(xs)
        n = xc.size
        for a in xs:
            assert a.dtype == np.float64 and a.flags.c_contiguous and a.size == n
        assert xc.dtype == np.float64 and xc.flags.c_contiguous
        gs = [np.ascontiguousarray(a) for a in gs]
        assert len(gs) == K and all(a.size == n for a in gs)
        xp = (_DP * K)(*[a.ctypes.data_as(_DP) for a in xs])
        gp = self._ptrs(gs)
        for _ in range(steps):
            self.lib.oracle_easgd_step(K, n, xp, gp, self._dtype_code(gs[0]),
                                       xc.ctypes.data_as(_DP), float(eta), float(rho))


    # -- schedules and synchronous SGD ---------------------------------------
    @staticmethod
    def _state_ptrs(xs):
        for a in xs:
            assert a.dtype == np.float64 and a.flags.c_contiguous
        return (_DP * len(xs))(*[a.ctypes.data_as(_DP) for a in xs])

    def sgd_step(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray], eta: float) -> None:
        """x_i -= eta * g_i in place (binary64 state, stored gradients)."""
        gs = [np.ascontiguousarray(a) for a in gs]
        self.lib.oracle_sgd_step(len(xs), xs[0].size, self._state_ptrs(xs), self._ptrs(gs),
                                 self._dtype_code(gs[0]), float(eta))

    def elastic_async(self, xs: Sequence[np.ndarray], xc: np.ndarray, order: Sequence[int], alpha: float) -> None:
        """Per-worker elastic exchanges in the given order, in place."""
        assert xc.dtype == np.float64 and xc.flags.c_contiguous
        o = np.ascontiguousarray(np.asarray(order, dtype=np.int32))
        assert len(o) == 0 or (o.min() >= 0 and o.max() < len(xs))
        self.lib.oracle_elastic_async(len(xs), xc.size, self._state_ptrs(xs), xc.ctypes.data_as(_DP),
                                      o.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(o), float(alpha))

    def sync_sgd(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray], eta: float, rescale: float):
        """x_i -= eta * rescale * sum_j g_j in place; returns the sum."""
        gs = [np.ascontiguousarray(a) for a in gs]
        out = np.empty(xs[0].size, dtype=np.float64)
        self.lib.oracle_sync_sgd(len(xs), xs[0].size, self._state_ptrs(xs), self._ptrs(gs),
                                 self._dtype_code(gs[0]), float(eta), float(rescale), out.ctypes.data_as(_DP))
        return out

    def broadcast(self, src: np.ndarray, K: int) -> List[np.ndarray]:
        src = np.ascontiguousarray(src)
        outs = [np.empty_like(src) for _ in range(K)]
        self.lib.oracle_broadcast(K, src.size, src.ctypes.data, src.dtype.itemsize, self._ptrs(outs))
        return outs

    # -- tensor layout ------------------------------------------------------
    @staticmethod
    def tensor_numel(N: int, K: int) -> int:
        return (N + 3) // 4 * 4 * K

    def tensor_from_copies(self, copies: Sequence[np.ndarray], fill=0) -> np.ndarray:
        """One buffer holding the K copies in the tensor layout; padding
        positions keep the value ``fill``."""
        copies = [np.ascontiguousarray(c) for c in copies]
        K, N, dt = len(copies), copies[0].size, copies[0].dtype
        out = np.full(self.tensor_numel(N, K), fill, dtype=dt)
        self.lib.oracle_tensor_from_copies(K, N, self._ptrs(copies), dt.itemsize, out.ctypes.data)
        return out

    def copies_from_tensor(self, tensor: np.ndarray, K: int, N: int) -> List[np.ndarray]:
        tensor = np.ascontiguousarray(tensor)
        outs = [np.empty(N, dtype=tensor.dtype) for _ in range(K)]
        self.lib.oracle_copies_from_tensor(K, N, tensor.ctypes.data, tensor.dtype.itemsize, self._ptrs(outs))
        return outs


_DEFAULT: Optional[Oracle] = None


def load() -> Oracle:
    """The oracle built from ``tc_oracle.c`` (compiled on first use)."""
    global _DEFAULT
    if _DEFAULT is None:
        if not os.path.exists(LIBRARY) or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE):
            build()
        _DEFAULT = Oracle(LIBRARY)
    return _DEFAULT
