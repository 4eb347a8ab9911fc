"""CPU oracle for the im2win transform and convolution (arXiv 2306.14320).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP library and never imports it.

Every function wraps a plain C loop nest in ``oracle.c`` (fp64 arithmetic for
floating point, no fast-math).  Arrays are numpy, C-contiguous.  The shape of a
problem is a ``Shape``: input N x C x H x W, filter K x C x Fh x Fw, stride
(sh, sw) and symmetric zero padding (ph, pw).
"""
import ctypes
import os
from dataclasses import dataclass

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_out_extent.restype = i64
        lib.oracle_out_extent.argtypes = [i64, i64, i64, i64]
        lib.oracle_im2win_elems.restype = i64
        lib.oracle_im2win_elems.argtypes = [p, ctypes.c_int]
        lib.oracle_row_width.restype = i64
        lib.oracle_row_width.argtypes = [p, ctypes.c_int]
        lib.oracle_im2col_elems.restype = i64
        lib.oracle_im2col_elems.argtypes = [p]
        lib.oracle_im2win.restype = None
        lib.oracle_im2win.argtypes = [p, p, p, ctypes.c_int, ctypes.c_int]
        lib.oracle_direct_conv.restype = None
        lib.oracle_direct_conv.argtypes = [p, p, p, p, p]
        lib.oracle_direct_conv_at.restype = None
        lib.oracle_direct_conv_at.argtypes = [p, p, p, p, i64, p, p]
        lib.oracle_window_conv.restype = None
        lib.oracle_window_conv.argtypes = [p, p, p, p, ctypes.c_int]
        lib.oracle_im2col.restype = None
        lib.oracle_im2col.argtypes = [p, p, p]
        _lib = lib
    return _lib


@dataclass(frozen=True)
class Shape:
    n: int
    c: int
    h: int
    w: int
    k: int
    fh: int
    fw: int
    sh: int = 1
    sw: int = 1
    ph: int = 0
    pw: int = 0

    def vec(self) -> np.ndarray:
        return np.array([self.n, self.c, self.h, self.w, self.k, self.fh, self.fw,
                         self.sh, self.sw, self.ph, self.pw], dtype=np.int64)

    @property
    def ho(self) -> int:
        return out_extent(self.h, self.fh, self.sh, self.ph)

    @property
    def wo(self) -> int:
        return out_extent(self.w, self.fw, self.sw, self.pw)

    @property
    def wp(self) -> int:
        return self.w + 2 * self.pw

    @property
    def wt(self) -> int:
        """Trimmed row width: the columns some window reads."""
        return int(_load().oracle_row_width(_ptr(self.vec()), 1))

    def win_shape_of(self, trimmed: bool):
        return (self.n, self.c, self.ho, (self.wt if trimmed else self.wp) * self.fh)

    @property
    def out_shape(self):
        return (self.n, self.k, self.ho, self.wo)

    @property
    def win_shape(self):
        return (self.n, self.c, self.ho, self.wp * self.fh)


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def out_extent(size: int, f: int, s: int, pad: int) -> int:
    """floor((size + 2*pad - f) / s) + 1, or 0 when the filter does not fit."""
    return int(_load().oracle_out_extent(size, f, s, pad))


def im2win_elems(shp: Shape, trimmed: bool = False) -> int:
    """Elements of the window tensor N x C x Ho x (Wr*Fh), Wr = Wp or the trimmed width."""
    v = shp.vec()
    return int(_load().oracle_im2win_elems(_ptr(v), int(trimmed)))


def im2col_elems(shp: Shape) -> int:
    """Elements of the im2col matrix N x (Ho*Wo) x (C*Fh*Fw)."""
    v = shp.vec()
    return int(_load().oracle_im2col_elems(_ptr(v)))


def im2win(shp: Shape, x: np.ndarray, trimmed: bool = False) -> np.ndarray:
    """Window tensor of x (2-, 4- or 8-byte elements, copied bit for bit), with
    rows of the padded width Wp, or of the trimmed width when asked."""
    x = np.ascontiguousarray(x)
    assert x.shape == (shp.n, shp.c, shp.h, shp.w), x.shape
    assert x.itemsize in (2, 4, 8)
    out = np.empty(shp.win_shape_of(trimmed), dtype=x.dtype)
    v = shp.vec()
    _load().oracle_im2win(_ptr(v), _ptr(x), _ptr(out), x.itemsize, int(trimmed))
    return out


def _f64(a: np.ndarray) -> np.ndarray:
    assert a.dtype == np.float64, a.dtype
    return np.ascontiguousarray(a)


def direct_conv(shp: Shape, x: np.ndarray, w: np.ndarray, with_abs: bool = False):
    """fp64 direct convolution; returns y (and sum |x*w| per output if asked)."""
    x, w = _f64(x), _f64(w)
    assert x.shape == (shp.n, shp.c, shp.h, shp.w)
    assert w.shape == (shp.k, shp.c, shp.fh, shp.fw)
    y = np.empty(shp.out_shape, dtype=np.float64)
    ya = np.empty(shp.out_shape, dtype=np.float64) if with_abs else None
    v = shp.vec()
    _load().oracle_direct_conv(_ptr(v), _ptr(x), _ptr(w), _ptr(y),
                               _ptr(ya) if with_abs else None)
    return (y, ya) if with_abs else y


def direct_conv_at(shp: Shape, x: np.ndarray, w: np.ndarray, idx: np.ndarray):
    """fp64 convolution at flat NCHW output indices; returns (y, sum |x*w|)."""
    x, w = _f64(x), _f64(w)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    total = shp.n * shp.k * shp.ho * shp.wo
    assert idx.size == 0 or (idx.min() >= 0 and idx.max() < total)
    y = np.empty(idx.shape, dtype=np.float64)
    ya = np.empty(idx.shape, dtype=np.float64)
    v = shp.vec()
    _load().oracle_direct_conv_at(_ptr(v), _ptr(x), _ptr(w), _ptr(idx), idx.size,
                                  _ptr(y), _ptr(ya))
    return y, ya


def window_conv(shp: Shape, win: np.ndarray, w: np.ndarray, trimmed: bool = False) -> np.ndarray:
    """Alg. 2 (basic im2win-based convolution) over a window tensor, fp64."""
    win, w = _f64(win), _f64(w)
    assert win.shape == shp.win_shape_of(trimmed)
    y = np.empty(shp.out_shape, dtype=np.float64)
    v = shp.vec()
    _load().oracle_window_conv(_ptr(v), _ptr(win), _ptr(w), _ptr(y), int(trimmed))
    return y


def im2col(shp: Shape, x: np.ndarray) -> np.ndarray:
    """Brute-force im2col matrices, N x (Ho*Wo) x (C*Fh*Fw), fp64."""
    x = _f64(x)
    cols = np.empty((shp.n, shp.ho * shp.wo, shp.c * shp.fh * shp.fw), dtype=np.float64)
    v = shp.vec()
    _load().oracle_im2col(_ptr(v), _ptr(x), _ptr(cols))
    return cols


def num_threads() -> int:
    """Threads the OpenMP runtime will use for the oracle's parallel loops."""
    env = os.environ.get("OMP_NUM_THREADS")
    if env:
        try:
            return max(1, int(env.split(",")[0]))
        except ValueError:
            pass
    return len(os.sched_getaffinity(0))
