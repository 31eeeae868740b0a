"""CPU oracle for the sparse-convolution layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does.

Thin numpy wrappers over ``oracle.cpp`` (a hash-map kernel map and float64
per-offset sums written straight from Eq. 1-3 of the paper).  Each function
names the passage it follows.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

SUBM, DOWN, UP = 0, 1, 2
_MODES = {"subm": SUBM, "down": DOWN, "up": UP}

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
        lib = ctypes.CDLL(path)
        i32p = ctypes.POINTER(ctypes.c_int32)
        i64p = ctypes.POINTER(ctypes.c_int64)
        f64p = ctypes.POINTER(ctypes.c_double)
        lib.orc_offsets.argtypes = [ctypes.c_int, ctypes.c_int, i32p]
        lib.orc_offsets.restype = ctypes.c_int
        lib.orc_out_coords.argtypes = [i32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, i32p]
        lib.orc_out_coords.restype = ctypes.c_int64
        lib.orc_kernel_map.argtypes = [i32p, ctypes.c_int64, i32p, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, i64p, i32p, i32p, ctypes.c_int64]
        lib.orc_kernel_map.restype = ctypes.c_int64
        lib.orc_features.argtypes = [f64p, ctypes.c_int64, ctypes.c_int, f64p, ctypes.c_int,
                                     ctypes.c_int, i64p, i32p, i32p, ctypes.c_int64, i64p,
                                     ctypes.c_int64, f64p, ctypes.c_int]
        lib.orc_features.restype = ctypes.c_int
        lib.orc_max_threads.argtypes = []
        lib.orc_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: status {status}")
        self.status = status


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype)) if a is not None else None


def _mode(mode) -> int:
    return _MODES[mode] if isinstance(mode, str) else int(mode)


def max_threads() -> int:
    return _load().orc_max_threads()


def offsets(K: int, t: int = 1) -> np.ndarray:
    """Delta(K, t) as int32 [K^3][3] (Section 2.1, the weight-offset set after Eq. 2)."""
    out = np.zeros((K ** 3, 3), dtype=np.int32)
    r = _load().orc_offsets(K, t, _p(out, ctypes.c_int32))
    if r < 0:
        raise OracleError(r, "offsets")
    return out


def out_coords(coords: np.ndarray, s: int, t: int = 1) -> np.ndarray:
    """Eq. 1 output coordinates, deduplicated and sorted by signed (b, x, y, z)."""
    c = np.ascontiguousarray(coords, dtype=np.int32).reshape(-1, 4)
    out = np.zeros_like(c)
    n = _load().orc_out_coords(_p(c, ctypes.c_int32), c.shape[0], s, t, _p(out, ctypes.c_int32))
    if n < 0:
        raise OracleError(n, "out_coords")
    return out[:n].copy()


class KernelMap:
    """Eq. 3 kernel map as per-offset pair lists (input row, output row),
    each list in ascending output row."""

    def __init__(self, counts, pin, pout, n_in, n_out, K):
        self.counts = counts
        self.pin = pin
        self.pout = pout
        self.n_in = n_in
        self.n_out = n_out
        self.K = K
        self.ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)

    @property
    def K3(self):
        return self.counts.shape[0]

    def pairs(self, k: int):
        a, b = self.ptr[k], self.ptr[k + 1]
        return self.pin[a:b], self.pout[a:b]

    def as_sets(self):
        return [set(zip(*map(np.ndarray.tolist, self.pairs(k)))) for k in range(self.K3)]


def kernel_map(in_coords: np.ndarray, out_coords_: np.ndarray | None, K: int, t: int, mode) -> KernelMap:
    """Eq. 3 via a hash table over the input coordinates (Section 2.2, Step 1)."""
    m = _mode(mode)
    ic = np.ascontiguousarray(in_coords, dtype=np.int32).reshape(-1, 4)
    if m == SUBM:
        oc = ic
    else:
        oc = np.ascontiguousarray(out_coords_, dtype=np.int32).reshape(-1, 4)
    k3 = K ** 3
    counts = np.zeros(k3, dtype=np.int64)
    cap = max(1, k3 * oc.shape[0])
    pin = np.zeros(cap, dtype=np.int32)
    pout = np.zeros(cap, dtype=np.int32)
    lib = _load()
    n = lib.orc_kernel_map(_p(ic, ctypes.c_int32), ic.shape[0], _p(oc, ctypes.c_int32), oc.shape[0],
                           K, t, m, _p(counts, ctypes.c_int64), _p(pin, ctypes.c_int32),
                           _p(pout, ctypes.c_int32), cap)
    if n < 0:
        raise OracleError(n, "kernel_map")
    return KernelMap(counts, pin[:n].copy(), pout[:n].copy(), ic.shape[0], oc.shape[0], K)


def features(x: np.ndarray, w: np.ndarray, kmap: KernelMap, rows: np.ndarray | None = None,
             nthreads: int = 0) -> np.ndarray:
    """Eq. 2 in float64 (sum over k ascending, then input channel ascending).

    ``x`` [n_in][c_in] and ``w`` [K^3][c_in][c_out] are widened exactly to float64.
    ``rows`` selects output rows (default: all).  Returns float64 [n_rows][c_out].
    """
    xd = np.ascontiguousarray(x, dtype=np.float64)
    wd = np.ascontiguousarray(w, dtype=np.float64)
    n_in, cin = xd.shape
    k3, cin2, cout = wd.shape
    if cin2 != cin or k3 != kmap.K3 or n_in != kmap.n_in:
        raise ValueError("shape mismatch")
    if rows is None:
        rr = None
        n_rows = kmap.n_out
    else:
        rr = np.ascontiguousarray(rows, dtype=np.int64)
        n_rows = rr.shape[0]
    y = np.zeros((n_rows, cout), dtype=np.float64)
    r = _load().orc_features(_p(xd, ctypes.c_double), n_in, cin, _p(wd, ctypes.c_double), cout, k3,
                             _p(kmap.counts, ctypes.c_int64), _p(kmap.pin, ctypes.c_int32),
                             _p(kmap.pout, ctypes.c_int32), kmap.n_out, _p(rr, ctypes.c_int64),
                             n_rows, _p(y, ctypes.c_double), nthreads)
    if r < 0:
        raise OracleError(r, "features")
    return y


def conv(in_coords, x, w, K, stride=1, t=1, mode="subm", out_coords_=None, rows=None, nthreads=0):
    """One sparse-conv layer: output coordinates (Eq. 1), kernel map (Eq. 3), features (Eq. 2).

    Returns (out_coords, kernel_map, y).  For ``up`` the fine output coordinates
    must be given; for ``down`` they are computed by Eq. 1.
    """
    m = _mode(mode)
    if m == SUBM:
        oc = np.ascontiguousarray(in_coords, dtype=np.int32)
    elif m == DOWN:
        oc = out_coords(in_coords, stride, t)
    else:
        oc = np.ascontiguousarray(out_coords_, dtype=np.int32)
    km = kernel_map(in_coords, oc, K, t, m)
    y = features(x, w, km, rows=rows, nthreads=nthreads)
    return oc, km, y
