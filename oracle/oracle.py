"""ctypes binding of the oracle's C library (TEST INFRASTRUCTURE ONLY).

Argument marshalling only: every value is computed in ``oracle.c``.  The
library is built by ``oracle/build.py`` (gcc, -O2, OpenMP) on first use if it
is not there yet.
"""
import ctypes
import os
from typing import NamedTuple

import numpy as np

from . import build as _build

_lib = None

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_int = ctypes.c_int


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    lib.oracle_num_threads.restype = _int
    lib.oracle_set_num_threads.argtypes = [_int]
    lib.oracle_filter_norms.argtypes = [_f64p, _int, _int, _int, _int, _f64p]
    lib.oracle_filter_perm.argtypes = [_f64p, _int, _int, _int, _int, _int, _i32p]
    lib.oracle_apply_perm.argtypes = [_f64p, _int, _int, _int, _int, _i32p, _f64p]
    lib.oracle_block_scores.argtypes = [_f64p, _int, _int, _int, _int, _int, _f64p]
    lib.oracle_kept_count.argtypes = [ctypes.c_int64, ctypes.c_double]
    lib.oracle_kept_count.restype = ctypes.c_int64
    lib.oracle_select.argtypes = [_f64p, ctypes.c_int64, ctypes.c_double, _u8p]
    lib.oracle_select.restype = ctypes.c_int64
    lib.oracle_masked_weight.argtypes = [_f64p, _u8p, _int, _int, _int, _int, _int, _f64p]
    lib.oracle_pack.argtypes = [_f64p, _u8p, _int, _int, _int, _int, _int, _i32p, _i32p, _f64p]
    lib.oracle_pack.restype = ctypes.c_int64
    lib.oracle_conv2d.argtypes = [_f64p, _f64p] + [_int] * 11 + [_f64p]
    lib.oracle_conv2d_at.argtypes = [_f64p, _f64p] + [_int] * 11 + [_i64p, ctypes.c_int64, _f64p]
    lib.oracle_epilogue.argtypes = [_f64p, _int, _int, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p, _int]
    lib.oracle_conv2d_bwd_data.argtypes = [_f64p, _f64p] + [_int] * 11 + [_f64p]
    lib.oracle_conv2d_bwd_weight.argtypes = [_f64p, _f64p, _u8p] + [_int] * 12 + [_f64p]
    lib.oracle_decode.argtypes = [_f64p, _i32p, _i32p, _f64p] + [_int] * 12 + [_f64p]
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def num_threads() -> int:
    return _load().oracle_num_threads()


def set_num_threads(k: int) -> None:
    """Threads of the oracle's parallel loops from now on (for timing it)."""
    _load().oracle_set_num_threads(int(k))


def filter_norms(w):
    w = _f64(w)
    n, m, h, wd = w.shape
    out = np.empty(n, np.float64)
    _load().oracle_filter_norms(w, n, m, h, wd, out)
    return out


def filter_perm(w, rearrange=True):
    w = _f64(w)
    n, m, h, wd = w.shape
    perm = np.empty(n, np.int32)
    _load().oracle_filter_perm(w, n, m, h, wd, int(bool(rearrange)), perm)
    return perm


def apply_perm(w, perm):
    w = _f64(w)
    n, m, h, wd = w.shape
    out = np.empty_like(w)
    _load().oracle_apply_perm(w, n, m, h, wd, np.ascontiguousarray(perm, np.int32), out)
    return out


def block_scores(wt, N):
    wt = _f64(wt)
    n, m, h, wd = wt.shape
    G = -(-n // N)
    S = np.empty((m, G), np.float64)
    _load().oracle_block_scores(wt, n, m, h, wd, int(N), S)
    return S


def kept_count(K, p):
    return int(_load().oracle_kept_count(int(K), float(p)))


def select(S, p):
    S = _f64(S)
    T = np.empty(S.shape, np.uint8)
    t = _load().oracle_select(S.reshape(-1), S.size, float(p), T.reshape(-1))
    return T, int(t)


def masked_weight(wt, T, N):
    wt = _f64(wt)
    n, m, h, wd = wt.shape
    out = np.empty_like(wt)
    _load().oracle_masked_weight(wt, np.ascontiguousarray(T, np.uint8), n, m, h, wd, int(N), out)
    return out


def pack(wt, T, N):
    wt = _f64(wt)
    n, m, h, wd = wt.shape
    T = np.ascontiguousarray(T, np.uint8)
    G = -(-n // N)
    t = int(T.sum())
    P = np.empty(G + 1, np.int32)
    I = np.empty(max(t, 1), np.int32)
    D = np.empty((max(t, 1), N, h, wd), np.float64)
    z = _load().oracle_pack(wt, T, n, m, h, wd, int(N), P, I, D)
    assert z == t
    return P, I[:t].copy(), D[:t].copy()


def _out_hw(H, W, h, wd, stride, pad):
    return (H + 2 * pad[0] - h) // stride[0] + 1, (W + 2 * pad[1] - wd) // stride[1] + 1


def conv2d(x, wbar, stride=(1, 1), pad=(0, 0)):
    """Eq. 7, NCHW x[B][m][H][W], weight wbar[n][m][h][w] -> y[B][n][Ho][Wo] (fp64)."""
    x, wbar = _f64(x), _f64(wbar)
    B, m, H, W = x.shape
    n, m2, h, wd = wbar.shape
    assert m == m2
    Ho, Wo = _out_hw(H, W, h, wd, stride, pad)
    y = np.empty((B, n, Ho, Wo), np.float64)
    _load().oracle_conv2d(x, wbar, B, m, H, W, n, h, wd, stride[0], stride[1], pad[0], pad[1], y)
    return y


def conv2d_at(x, wbar, idx, stride=(1, 1), pad=(0, 0)):
    """Eq. 7 evaluated only at the flat NCHW output indices ``idx``."""
    x, wbar = _f64(x), _f64(wbar)
    B, m, H, W = x.shape
    n, _, h, wd = wbar.shape
    idx = np.ascontiguousarray(idx, np.int64)
    out = np.empty(idx.size, np.float64)
    _load().oracle_conv2d_at(x, wbar, B, m, H, W, n, h, wd, stride[0], stride[1], pad[0], pad[1],
                             idx, idx.size, out)
    return out


def conv2d_bwd_data(dy, wbar, input_hw, stride=(1, 1), pad=(0, 0)):
    """dL/dX of Eq. 7: dy[B][n][Ho][Wo], wbar[n][m][h][w] -> dx[B][m][H][W] (fp64)."""
    dy, wbar = _f64(dy), _f64(wbar)
    B, n = dy.shape[0], dy.shape[1]
    _, m, h, wd = wbar.shape
    H, W = input_hw
    assert (dy.shape[2], dy.shape[3]) == _out_hw(H, W, h, wd, stride, pad)
    dx = np.empty((B, m, H, W), np.float64)
    _load().oracle_conv2d_bwd_data(dy, wbar, B, m, H, W, n, h, wd, stride[0], stride[1], pad[0],
                                   pad[1], dx)
    return dx


def conv2d_bwd_weight(x, dy, T, N, kernel_hw, stride=(1, 1), pad=(0, 0)):
    """dL/dW of Eq. 7 on the kept 1xN blocks of mask T[m][G] (0 elsewhere):
    x[B][m][H][W], dy[B][n][Ho][Wo] -> dw[n][m][h][w] (fp64, rearranged rows)."""
    x, dy = _f64(x), _f64(dy)
    B, m, H, W = x.shape
    n = dy.shape[1]
    h, wd = kernel_hw
    assert (dy.shape[2], dy.shape[3]) == _out_hw(H, W, h, wd, stride, pad)
    T = np.ascontiguousarray(T, np.uint8)
    assert T.shape == (m, -(-n // N))
    dw = np.empty((n, m, h, wd), np.float64)
    _load().oracle_conv2d_bwd_weight(x, dy, T, B, m, H, W, n, h, wd, int(N), stride[0], stride[1],
                                     pad[0], pad[1], dw)
    return dw


_ACTS = {"none": 0, "relu": 1, "relu6": 2}


def epilogue(y, scale=None, bias=None, act="none"):
    """act(scale[o] * y + bias[o]) per output channel o of y[B][n][Ho][Wo]
    (a new fp64 array); None means scale 1 / bias 0."""
    y = np.array(y, dtype=np.float64, order="C", copy=True)
    B, n = y.shape[0], y.shape[1]
    hw = int(np.prod(y.shape[2:])) if y.ndim > 2 else 1
    s = None if scale is None else _f64(scale)
    b = None if bias is None else _f64(bias)
    for v in (s, b):
        assert v is None or v.size == n
    _load().oracle_epilogue(y, B, n, hw, None if s is None else s.ctypes.data,
                            None if b is None else b.ctypes.data, _ACTS[act])
    return y


def decode(x, P, I, D, n, stride=(1, 1), pad=(0, 0)):
    """Eq. 8 over the BSR arrays; same output as ``conv2d``."""
    x = _f64(x)
    B, m, H, W = x.shape
    t, N, h, wd = D.shape if len(I) else (0,) + tuple(D.shape[1:])
    Ho, Wo = _out_hw(H, W, h, wd, stride, pad)
    y = np.zeros((B, n, Ho, Wo), np.float64)
    Dd = _f64(D) if len(I) else np.zeros((1, N, h, wd))
    Ii = np.ascontiguousarray(I, np.int32) if len(I) else np.zeros(1, np.int32)
    _load().oracle_decode(x, np.ascontiguousarray(P, np.int32), Ii, Dd, B, m, H, W, n, h, wd,
                          int(N), stride[0], stride[1], pad[0], pad[1], y)
    return y


class Pruned(NamedTuple):
    perm: np.ndarray      # int32[n]
    T: np.ndarray         # uint8[m][G]
    t: int
    wt: np.ndarray        # rearranged weight, fp64 [n][m][h][w]
    wbar: np.ndarray      # masked rearranged weight (Eq. 6), fp64
    P: np.ndarray         # int32[G+1]
    I: np.ndarray         # int32[t]
    D: np.ndarray         # fp64[t][N][h][w]


def prune(w, N, p, rearrange):
    """Offline steps in the paper's order: rearrange (Sec. 3.3), score blocks (Eq. 5),
    keep the top-(1-p) (Eq. 1), mask (Eq. 6), encode (Sec. 3.4)."""
    perm = filter_perm(w, rearrange)
    wt = apply_perm(w, perm)
    S = block_scores(wt, N)
    T, t = select(S, p)
    wbar = masked_weight(wt, T, N)
    P, I, D = pack(wt, T, N)
    return Pruned(perm, T, t, wt, wbar, P, I, D)
