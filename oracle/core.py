"""ctypes view of the oracle's C loops (float64 in, float64 out).

Test infrastructure only; see ``oracle/__init__.py``.
"""
from __future__ import annotations

import ctypes as C
from typing import Tuple

import numpy as np

from .build import ensure_built

_lib = None
_dp = C.POINTER(C.c_double)


def lib():
    global _lib
    if _lib is None:
        L = C.CDLL(ensure_built())
        L.or_out_extent.restype = C.c_int
        L.or_out_extent.argtypes = [C.c_int] * 4
        L.or_conv.restype = None
        L.or_conv.argtypes = [_dp, _dp] + [C.c_int] * 9 + [_dp]
        L.or_conv_points.restype = None
        L.or_conv_points.argtypes = [_dp, _dp] + [C.c_int] * 9 + [C.POINTER(C.c_int32), C.c_long, _dp]
        L.or_block_sums.restype = None
        L.or_block_sums.argtypes = [_dp, C.c_long, C.c_long, C.c_double, _dp, _dp]
        L.or_num_threads.restype = C.c_int
        L.or_num_threads.argtypes = []
        _lib = L
    return _lib


def _f64(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def out_extent(h: int, r: int, u: int, p: int) -> int:
    """Output extent of one axis, floor((H + 2P - R)/U) + 1 (eq. 1 plus zero padding)."""
    return lib().or_out_extent(h, r, u, p)


def conv(D: np.ndarray, W: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """Direct convolution of eq. (1), float64: D [N][C][H][W] (x) W [M][C][R][S] -> [N][M][E][F]."""
    D = _f64(D)
    W = _f64(W)
    N, Ch, H, Wd = D.shape
    M, Ch2, R, S = W.shape
    assert Ch == Ch2, (D.shape, W.shape)
    E, F = out_extent(H, R, stride, pad), out_extent(Wd, S, stride, pad)
    O = np.empty((N, M, E, F), dtype=np.float64)
    lib().or_conv(_p(D), _p(W), N, Ch, H, Wd, M, R, S, stride, pad, _p(O))
    return O


def conv_points(D: np.ndarray, W: np.ndarray, stride: int, pad: int, pts: np.ndarray) -> np.ndarray:
    """Eq. (1) at the coordinates pts[q] = (n, m, x, y)."""
    D = _f64(D)
    W = _f64(W)
    N, Ch, H, Wd = D.shape
    M, _, R, S = W.shape
    pts = np.ascontiguousarray(pts, dtype=np.int32).reshape(-1, 4)
    out = np.empty(len(pts), dtype=np.float64)
    lib().or_conv_points(_p(D), _p(W), N, Ch, H, Wd, M, R, S, stride, pad,
                         pts.ctypes.data_as(C.POINTER(C.c_int32)), len(pts), _p(out))
    return out


def block_sums(X: np.ndarray, base: float = 0.0) -> Tuple[np.ndarray, np.ndarray]:
    """Sec. 3.2 input checksums of a stack of blocks: (sum_r X_r, sum_r (r+base) X_r)."""
    X = _f64(X)
    rows = X.shape[0]
    cols = int(np.prod(X.shape[1:]))
    c1 = np.empty(cols, dtype=np.float64)
    c2 = np.empty(cols, dtype=np.float64)
    lib().or_block_sums(_p(X), rows, cols, float(base), _p(c1), _p(c2))
    return c1.reshape(X.shape[1:]), c2.reshape(X.shape[1:])


def num_threads() -> int:
    return lib().or_num_threads()
