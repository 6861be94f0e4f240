"""Oracle for im2win convolution -- TEST INFRASTRUCTURE ONLY.

A ctypes wrapper over ``oracle.c``: a plain fp64 CPU reference of the paper's
definitions (Sec. III-A Eq. 1, Sec. III-B Eq. 2, Sec. III-C Eq. 3).  Only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  It shares no code with the GPU library and never
imports it.

Layouts: input NHWC ``[N][H_i][W_i][C_i]``, filter ``[K_h][K_w][C_i][C_o]``,
output NHWC ``[N][H_o][W_o][C_o]``, window tensor ``[N][H_o][W_i*K_h][C_i]``
(with filter dilation d: ``[N][H_o][d*ceil(W/d)*K_h][C_i]``, strip columns
grouped by residue mod d; see ``oracle.c``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "_oracle.so")

_i64 = ctypes.c_int64
_dp = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` with gcc (fp64, no contraction, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
            "-std=c99", "-Wall", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_out_extent.restype = _i64
        lib.oracle_out_extent.argtypes = [_i64, _i64, _i64]
        lib.oracle_threads.restype = ctypes.c_int
        lib.oracle_set_threads.restype = None
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_conv_f64.restype = ctypes.c_int
        lib.oracle_conv_f64.argtypes = [_i64] * 8 + [_dp, _dp, _dp, _dp]
        lib.oracle_conv_f64_points.restype = ctypes.c_int
        lib.oracle_conv_f64_points.argtypes = [_i64] * 8 + [_dp, _dp, _i64,
                                                           ctypes.POINTER(_i64), _dp, _dp]
        lib.oracle_window_elems.restype = _i64
        lib.oracle_window_elems.argtypes = [_i64] * 6
        lib.oracle_im2col_elems.restype = _i64
        lib.oracle_im2col_elems.argtypes = [_i64] * 7
        lib.oracle_im2win.restype = ctypes.c_int
        lib.oracle_im2win.argtypes = [_i64] * 7 + [_vp, _vp]
        lib.oracle_windowed_conv_f64.restype = ctypes.c_int
        lib.oracle_windowed_conv_f64.argtypes = [_i64] * 8 + [_dp, _dp, _dp]
        lib.oracle_conv_pad_f64.restype = ctypes.c_int
        lib.oracle_conv_pad_f64.argtypes = [_i64] * 10 + [_dp, _dp, _dp, _dp]
        lib.oracle_im2win_pad.restype = ctypes.c_int
        lib.oracle_im2win_pad.argtypes = [_i64] * 9 + [_vp, _vp]
        lib.oracle_conv_dil_f64.restype = ctypes.c_int
        lib.oracle_conv_dil_f64.argtypes = [_i64] * 11 + [_dp, _dp, _dp, _dp]
        lib.oracle_dil_group_cols.restype = _i64
        lib.oracle_dil_group_cols.argtypes = [_i64, _i64]
        lib.oracle_dil_window_col.restype = _i64
        lib.oracle_dil_window_col.argtypes = [_i64] * 4
        lib.oracle_im2win_dil.restype = ctypes.c_int
        lib.oracle_im2win_dil.argtypes = [_i64] * 10 + [_vp, _vp]
        lib.oracle_windowed_conv_dil_f64.restype = ctypes.c_int
        lib.oracle_windowed_conv_dil_f64.argtypes = [_i64] * 9 + [_dp, _dp, _dp]
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def out_extent(n_in: int, k: int, s: int) -> int:
    """H_o (or W_o) = floor((n_in - k) / s) + 1; -1 if the filter does not fit."""
    return int(_load().oracle_out_extent(n_in, k, s))


def threads() -> int:
    """OpenMP threads the oracle runs with."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Run the oracle's parallel loops on `n` threads (timing only)."""
    _load().oracle_set_threads(int(n))


def conv(x, w, stride: int, with_abs: bool = False):
    """Eq. (1) in fp64. ``x``: NHWC input, ``w``: [K_h][K_w][C_i][C_o].

    Returns O (and A = sum |x||w| per output, if ``with_abs``)."""
    x = _f64(x)
    w = _f64(w)
    N, Hi, Wi, Ci = x.shape
    Kh, Kw, Ci2, Co = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho, Wo = out_extent(Hi, Kh, stride), out_extent(Wi, Kw, stride)
    if Ho < 0 or Wo < 0:
        raise ValueError("filter does not fit")
    out = np.empty((N, Ho, Wo, Co), np.float64)
    ab = np.empty_like(out) if with_abs else None
    rc = _load().oracle_conv_f64(N, Ci, Hi, Wi, Co, Kh, Kw, stride, _ptr(x), _ptr(w),
                                 _ptr(out), _ptr(ab) if with_abs else None)
    if rc != 0:
        raise ValueError("oracle_conv_f64 rejected its arguments")
    return (out, ab) if with_abs else out


def conv_points(x, w, stride: int, pts):
    """Eq. (1) at output coordinates ``pts`` (an [P, 4] int array of i, m, n, j).

    Returns (O, A) as two length-P fp64 arrays."""
    x = _f64(x)
    w = _f64(w)
    N, Hi, Wi, Ci = x.shape
    Kh, Kw, Ci2, Co = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    pts = np.ascontiguousarray(pts, dtype=np.int64).reshape(-1, 4)
    out = np.empty(len(pts), np.float64)
    ab = np.empty(len(pts), np.float64)
    rc = _load().oracle_conv_f64_points(N, Ci, Hi, Wi, Co, Kh, Kw, stride, _ptr(x), _ptr(w),
                                        len(pts), pts.ctypes.data_as(ctypes.POINTER(_i64)),
                                        _ptr(out), _ptr(ab))
    if rc != 0:
        raise ValueError("oracle_conv_f64_points rejected its arguments")
    return out, ab


def im2win(x, k_h: int, stride: int) -> np.ndarray:
    """Eq. (2): the window tensor [N][H_o][W_i*K_h][C_i], bit-exact, any dtype."""
    x = np.ascontiguousarray(x)
    N, Hi, Wi, Ci = x.shape
    Ho = out_extent(Hi, k_h, stride)
    if Ho < 0:
        raise ValueError("filter does not fit")
    out = np.empty((N, Ho, Wi * k_h, Ci), x.dtype)
    rc = _load().oracle_im2win(N, Ci, Hi, Wi, k_h, stride, x.dtype.itemsize,
                               x.ctypes.data_as(_vp), out.ctypes.data_as(_vp))
    if rc != 0:
        raise ValueError("oracle_im2win rejected its arguments")
    return out


def windowed_conv(win, w, h_i: int, w_i: int, stride: int):
    """Eq. (3): the convolution computed from the window tensor, fp64."""
    win = _f64(win)
    w = _f64(w)
    N, Ho_, _, Ci = win.shape
    Kh, Kw, Ci2, Co = w.shape
    Ho, Wo = out_extent(h_i, Kh, stride), out_extent(w_i, Kw, stride)
    if Ci2 != Ci or Ho != Ho_ or win.shape[2] != w_i * Kh:
        raise ValueError("window tensor does not match the layer")
    out = np.empty((N, Ho, Wo, Co), np.float64)
    rc = _load().oracle_windowed_conv_f64(N, Ci, h_i, w_i, Co, Kh, Kw, stride,
                                          _ptr(win), _ptr(w), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_windowed_conv_f64 rejected its arguments")
    return out


def window_elems(N: int, Ci: int, Hi: int, Wi: int, Kh: int, stride: int) -> int:
    return int(_load().oracle_window_elems(N, Ci, Hi, Wi, Kh, stride))


def im2col_elems(N: int, Ci: int, Hi: int, Wi: int, Kh: int, Kw: int, stride: int) -> int:
    return int(_load().oracle_im2col_elems(N, Ci, Hi, Wi, Kh, Kw, stride))


def conv_pad(x, w, stride: int, pad_h: int, pad_w: int, with_abs: bool = False):
    """Eq. (1) on the input zero-padded by ``pad_h`` rows above and below and
    ``pad_w`` columns left and right (an extension: the paper's layers have no
    padding).  Returns O (and A = sum |x||w|, if ``with_abs``)."""
    x = _f64(x)
    w = _f64(w)
    N, Hi, Wi, Ci = x.shape
    Kh, Kw, Ci2, Co = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho, Wo = out_extent(Hi + 2 * pad_h, Kh, stride), out_extent(Wi + 2 * pad_w, Kw, stride)
    if Ho < 0 or Wo < 0 or pad_h < 0 or pad_w < 0:
        raise ValueError("filter does not fit")
    out = np.empty((N, Ho, Wo, Co), np.float64)
    ab = np.empty_like(out) if with_abs else None
    rc = _load().oracle_conv_pad_f64(N, Ci, Hi, Wi, Co, Kh, Kw, stride, pad_h, pad_w, _ptr(x), _ptr(w),
                                     _ptr(out), _ptr(ab) if with_abs else None)
    if rc != 0:
        raise ValueError("oracle_conv_pad_f64 rejected its arguments")
    return (out, ab) if with_abs else out


def im2win_pad(x, k_h: int, stride: int, pad_h: int, pad_w: int) -> np.ndarray:
    """Eq. (2) on the zero-padded input: [N][H_o][(W_i+2 pad_w)*K_h][C_i],
    bit-exact, zero bytes at padded positions."""
    x = np.ascontiguousarray(x)
    N, Hi, Wi, Ci = x.shape
    Ho = out_extent(Hi + 2 * pad_h, k_h, stride)
    if Ho < 0 or pad_h < 0 or pad_w < 0:
        raise ValueError("filter does not fit")
    Wp = Wi + 2 * pad_w
    out = np.empty((N, Ho, Wp * k_h, Ci), x.dtype)
    rc = _load().oracle_im2win_pad(N, Ci, Hi, Wi, k_h, stride, pad_h, pad_w, x.dtype.itemsize,
                                   x.ctypes.data_as(_vp), out.ctypes.data_as(_vp))
    if rc != 0:
        raise ValueError("oracle_im2win_pad rejected its arguments")
    return out


def dil_extent(n: int, k: int, stride: int, dilation: int) -> int:
    """Output extent with filter dilation: floor((n - (k-1)*d - 1) / s) + 1,
    or -1 when the dilated filter does not fit."""
    if dilation <= 0 or k <= 0:
        return -1
    return out_extent(n, (k - 1) * dilation + 1, stride)


def conv_dil(x, w, stride: int, pad_h: int, pad_w: int, dilation: int, with_abs: bool = False):
    """Eq. (1) with filter dilation on the zero-padded input (an extension):
    tap (u, v) reads padded row m*s + u*d and column n*s + v*d.  Returns O
    (and A = sum |x||w|, if ``with_abs``)."""
    x = _f64(x)
    w = _f64(w)
    N, Hi, Wi, Ci = x.shape
    Kh, Kw, Ci2, Co = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho = dil_extent(Hi + 2 * pad_h, Kh, stride, dilation)
    Wo = dil_extent(Wi + 2 * pad_w, Kw, stride, dilation)
    if Ho < 0 or Wo < 0 or pad_h < 0 or pad_w < 0:
        raise ValueError("filter does not fit")
    out = np.empty((N, Ho, Wo, Co), np.float64)
    ab = np.empty_like(out) if with_abs else None
    rc = _load().oracle_conv_dil_f64(N, Ci, Hi, Wi, Co, Kh, Kw, stride, pad_h, pad_w, dilation, _ptr(x),
                                     _ptr(w), _ptr(out), _ptr(ab) if with_abs else None)
    if rc != 0:
        raise ValueError("oracle_conv_dil_f64 rejected its arguments")
    return (out, ab) if with_abs else out


def dil_group_cols(wp: int, dilation: int) -> int:
    """Columns per residue group of a dilated strip, ceil(Wp / d)."""
    return int(_load().oracle_dil_group_cols(wp, dilation))


def dil_window_col(n: int, stride: int, dilation: int, wq: int) -> int:
    """Strip position (in columns) where the window of output column n starts."""
    return int(_load().oracle_dil_window_col(n, stride, dilation, wq))


def im2win_dil(x, k_h: int, stride: int, pad_h: int, pad_w: int, dilation: int) -> np.ndarray:
    """Eq. (2) with dilation on the zero-padded input: [N][H_o][d*Wq*K_h][C_i],
    strip columns grouped by residue mod d, bit-exact, zero bytes at padded
    and filler positions."""
    x = np.ascontiguousarray(x)
    N, Hi, Wi, Ci = x.shape
    Ho = dil_extent(Hi + 2 * pad_h, k_h, stride, dilation)
    if Ho < 0 or pad_h < 0 or pad_w < 0:
        raise ValueError("filter does not fit")
    Wq = dil_group_cols(Wi + 2 * pad_w, dilation)
    out = np.empty((N, Ho, dilation * Wq * k_h, Ci), x.dtype)
    rc = _load().oracle_im2win_dil(N, Ci, Hi, Wi, k_h, stride, pad_h, pad_w, dilation, x.dtype.itemsize,
                                   x.ctypes.data_as(_vp), out.ctypes.data_as(_vp))
    if rc != 0:
        raise ValueError("oracle_im2win_dil rejected its arguments")
    return out


def windowed_conv_dil(win, w, hp: int, wp: int, stride: int, dilation: int) -> np.ndarray:
    """Eq. (3) with dilation: the convolution read out of ``im2win_dil``'s
    window tensor (padded extents ``hp`` x ``wp``)."""
    win = _f64(win)
    w = _f64(w)
    N, Ho = win.shape[0], win.shape[1]
    Ci = win.shape[3]
    Kh, Kw, Ci2, Co = w.shape
    Wo = dil_extent(wp, Kw, stride, dilation)
    if Ci2 != Ci or Wo < 0:
        raise ValueError("shape mismatch")
    out = np.empty((N, Ho, Wo, Co), np.float64)
    rc = _load().oracle_windowed_conv_dil_f64(N, Ci, hp, wp, Co, Kh, Kw, stride, dilation, _ptr(win), _ptr(w),
                                              _ptr(out))
    if rc != 0:
        raise ValueError("oracle_windowed_conv_dil_f64 rejected its arguments")
    return out
