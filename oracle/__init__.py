"""fp64 CPU oracle for the WTConv operator -- TEST INFRASTRUCTURE ONLY.

This package is the correctness reference the GPU library is checked against.
Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it; the product path never does. It shares no code
with the GPU path. See ``wtconv_oracle.c`` for what each function computes and
which passage of the paper it follows.

All arrays are numpy float64, C-contiguous. Layouts:
  x, y, dy, dx: [B, C, H, W]; base_w: [C, k, k]; base_scale: [C];
  level_w: [L, 4C, k, k] (row 4c+q, q = LL, LH, HL, HH); level_scale: [L, 4C].
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None
_D = ctypes.POINTER(ctypes.c_double)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    i, d, l = ctypes.c_int, ctypes.c_double, ctypes.c_long
    lib.oracle_haar_analysis.argtypes = [i, i, _D, _D]
    lib.oracle_haar_synthesis.argtypes = [i, i, _D, _D]
    lib.oracle_corr_same.argtypes = [i, i, i, _D, _D, _D]
    lib.oracle_pyramid_size.argtypes = [i, i, i]
    lib.oracle_pyramid_size.restype = l
    lib.oracle_plane_pyramid.argtypes = [i, i, i, _D, _D]
    lib.oracle_plane_forward.argtypes = [i, i, i, i, _D, _D, d, _D, _D, d, _D, _D]
    lib.oracle_closed_form_synthesis.argtypes = [i, i, i, _D, _D]
    lib.oracle_cascade_synthesis.argtypes = [i, i, i, _D, _D]
    lib.oracle_plane_backward.argtypes = [i, i, i, i, _D, _D, _D, d, _D, _D, d, _D, _D, _D, _D, _D, _D]
    lib.oracle_forward.argtypes = [i] * 6 + [_D] * 7
    lib.oracle_backward.argtypes = [i] * 6 + [_D] * 13
    lib.oracle_num_threads.restype = i
    lib.oracle_set_num_threads.argtypes = [i]
    _lib = lib
    return lib


def _p(a):
    return a.ctypes.data_as(_D)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP thread count of the whole-tensor entry points."""
    _load().oracle_set_num_threads(int(n))


def level_shape(H: int, W: int, l: int):
    """Grid size of level l: ceil(H / 2^l) x ceil(W / 2^l)."""
    for _ in range(l):
        H, W = (H + 1) // 2, (W + 1) // 2
    return H, W


def haar_analysis(X):
    """One Haar analysis level with bottom/right zero padding: [h, w] -> [4, ceil(h/2), ceil(w/2)]."""
    X = _f64(X)
    h, w = X.shape
    Y = np.empty((4, (h + 1) // 2, (w + 1) // 2))
    _load().oracle_haar_analysis(h, w, _p(X), _p(Y))
    return Y


def haar_synthesis(Y, h: int, w: int):
    """One Haar synthesis level cropped to [h, w]."""
    Y = _f64(Y)
    assert Y.shape == (4, (h + 1) // 2, (w + 1) // 2)
    X = np.empty((h, w))
    _load().oracle_haar_synthesis(h, w, _p(Y), _p(X))
    return X


def corr_same(u, wk):
    u, wk = _f64(u), _f64(wk)
    h, w = u.shape
    k = wk.shape[0]
    out = np.empty((h, w))
    _load().oracle_corr_same(h, w, k, _p(u), _p(wk), _p(out))
    return out


def _split_pyramid(flat, H, W, L):
    out, off = [], 0
    for l in range(1, L + 1):
        h, w = level_shape(H, W, l)
        out.append(flat[off:off + 4 * h * w].reshape(4, h, w))
        off += 4 * h * w
    return out


def _join_pyramid(levels):
    return _f64(np.concatenate([np.asarray(z, dtype=np.float64).ravel() for z in levels])) \
        if levels else np.zeros(1)


def plane_pyramid(x, L: int):
    """Unfiltered Haar pyramid [Y_1, ..., Y_L] of one plane (raw LL carried)."""
    x = _f64(x)
    H, W = x.shape
    n = int(_load().oracle_pyramid_size(H, W, L))
    flat = np.zeros(max(n, 1))
    _check(_load().oracle_plane_pyramid(H, W, L, _p(x), _p(flat)), "plane_pyramid")
    return _split_pyramid(flat, H, W, L)


def plane_forward(x, w0, s0, wl, sl, return_z=False, b0=0.0):
    """Alg. 1 on one plane. wl: [L, 4, k, k], sl: [L, 4], b0: base bias. Returns y (and [Z_1..Z_L])."""
    x, w0 = _f64(x), _f64(w0)
    H, W = x.shape
    k = w0.shape[0]
    wl = _f64(np.asarray(wl).reshape(-1, 4, k, k)) if np.size(wl) else np.zeros((0, 4, k, k))
    L = wl.shape[0]
    sl = _f64(np.asarray(sl).reshape(L, 4)) if L else np.zeros((1,))
    wl_p = wl if L else np.zeros(1)
    y = np.empty((H, W))
    n = int(_load().oracle_pyramid_size(H, W, L))
    z = np.zeros(max(n, 1))
    _check(_load().oracle_plane_forward(H, W, k, L, _p(x), _p(w0), float(s0), _p(wl_p), _p(sl), float(b0), _p(y),
                                        _p(z)), "plane_forward")
    if return_z:
        return y, _split_pyramid(z, H, W, L)
    return y


def closed_form_synthesis(levels, H: int, W: int):
    """Proposition 2 evaluated per pixel from a list of 4-band level arrays."""
    L = len(levels)
    flat = _join_pyramid(levels)
    R = np.empty((H, W))
    _load().oracle_closed_form_synthesis(H, W, L, _p(flat), _p(R))
    return R


def plane_backward(x, dy, w0, s0, wl, sl, b0=0.0):
    """Reverse mode through plane_forward. Returns dx, dw0, ds0, dwl [L,4,k,k], dsl [L,4], db0."""
    x, dy, w0 = _f64(x), _f64(dy), _f64(w0)
    H, W = x.shape
    k = w0.shape[0]
    wl = _f64(np.asarray(wl).reshape(-1, 4, k, k)) if np.size(wl) else np.zeros((0, 4, k, k))
    L = wl.shape[0]
    sl = _f64(np.asarray(sl).reshape(L, 4)) if L else np.zeros((1,))
    dx = np.empty((H, W))
    dw0 = np.empty((k, k))
    ds0 = np.empty(1)
    db0 = np.empty(1)
    dwl = np.zeros((max(L, 1), 4, k, k))
    dsl = np.zeros((max(L, 1), 4))
    wl_p = wl if L else np.zeros(1)
    _check(_load().oracle_plane_backward(H, W, k, L, _p(x), _p(dy), _p(w0), float(s0), _p(wl_p), _p(sl), float(b0),
                                         _p(dx), _p(dw0), _p(ds0), _p(db0), _p(dwl), _p(dsl)), "plane_backward")
    return dx, dw0, float(ds0[0]), dwl[:L], dsl[:L], float(db0[0])


def _stack_levels(level_w, level_scale, C, k):
    L = len(level_w)
    if L == 0:
        return np.zeros(1), np.zeros(1)
    lw = _f64(np.stack([np.asarray(w, dtype=np.float64).reshape(4 * C, k, k) for w in level_w]))
    ls = _f64(np.stack([np.asarray(s, dtype=np.float64).reshape(4 * C) for s in level_scale]))
    return lw, ls


def forward(x, base_w, base_scale, level_w, level_scale, base_bias=None):
    """Whole-tensor forward. level_w / level_scale: lists of L arrays [4C,k,k] / [4C];
    base_bias: [C] or None (zero)."""
    x = _f64(x)
    B, C, H, W = x.shape
    base_w = _f64(base_w)
    k = base_w.shape[-1]
    L = len(level_w)
    lw, ls = _stack_levels(level_w, level_scale, C, k)
    bias = _f64(base_bias) if base_bias is not None else None
    y = np.empty_like(x)
    _check(_load().oracle_forward(B, C, H, W, k, L, _p(x), _p(base_w), _p(_f64(base_scale)),
                                  _p(bias) if bias is not None else None, _p(lw), _p(ls), _p(y)), "forward")
    return y


def backward(x, dy, base_w, base_scale, level_w, level_scale, base_bias=None):
    """Whole-tensor backward. Returns dict with dx, d_base_w, d_base_scale, d_base_bias,
    d_level_w, d_level_scale."""
    x, dy = _f64(x), _f64(dy)
    B, C, H, W = x.shape
    base_w = _f64(base_w)
    k = base_w.shape[-1]
    L = len(level_w)
    lw, ls = _stack_levels(level_w, level_scale, C, k)
    bias = _f64(base_bias) if base_bias is not None else None
    dx = np.empty_like(x)
    dbw = np.empty((C, k, k))
    dbs = np.empty(C)
    dbb = np.empty(C)
    dlw = np.zeros((max(L, 1), 4 * C, k, k))
    dls = np.zeros((max(L, 1), 4 * C))
    _check(_load().oracle_backward(B, C, H, W, k, L, _p(x), _p(dy), _p(base_w), _p(_f64(base_scale)),
                                   _p(bias) if bias is not None else None, _p(lw), _p(ls), _p(dx), _p(dbw),
                                   _p(dbs), _p(dbb), _p(dlw), _p(dls)), "backward")
    return {"dx": dx, "d_base_w": dbw, "d_base_scale": dbs, "d_base_bias": dbb,
            "d_level_w": [dlw[l] for l in range(L)], "d_level_scale": [dls[l] for l in range(L)]}


def cascade_synthesis(levels, H: int, W: int):
    """Upward half of Alg. 1 (sequential synthesis cascade) from [Z_1..Z_L]."""
    L = len(levels)
    flat = _join_pyramid(levels)
    R = np.empty((H, W))
    _check(_load().oracle_cascade_synthesis(H, W, L, _p(flat), _p(R)), "cascade_synthesis")
    return R
