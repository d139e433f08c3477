"""CPU oracle for KGS-sparse 3-D convolution -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It wraps ``rt3d_oracle.c`` (plain C, float64
arithmetic) through ctypes and shares nothing with the GPU library.

Array conventions follow the paper's notation (Section 3):
  x [n][c_in][t][h][w], w [c_out][c_in][kt][kh][kw] (kt = kernel depth K_d),
  mask [P][Q][kt*kh*kw] with P = ceil(c_out/g_m), Q = ceil(c_in/g_n)
  (Section 4), y [n][c_out][to][ho][wo].
"""
import ctypes
import os

import numpy as np

from .build_oracle import LIB, build_oracle

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build_oracle(force=True)
        lib = ctypes.CDLL(LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        i = ctypes.c_int
        lib.oracle_conv3d_dense.argtypes = [i] * 15 + [dp, dp, dp, dp, i, dp]
        lib.oracle_conv3d_kgs.argtypes = [i] * 17 + [dp, dp, ctypes.c_void_p, dp, dp, i, dp]
        lib.oracle_kgs_pack.argtypes = [i] * 8 + [ctypes.c_void_p] * 8
        lib.oracle_maxpool3d.argtypes = [i] * 14 + [dp, dp]
        lib.oracle_conv3d_points.argtypes = ([i] * 17 + [dp, dp, ctypes.c_void_p, dp, dp, i,
                                              ctypes.c_long, ctypes.c_void_p, dp])
        lib.oracle_group_reweight.argtypes = ([i] * 7 + [dp, dp] + [ctypes.c_double] * 4 +
                                              [dp, dp, dp, ctypes.c_void_p, dp, dp])
        lib.oracle_num_threads.argtypes = []
        lib.oracle_set_threads.argtypes = [i]
        lib.oracle_set_threads.restype = None
        for f in (lib.oracle_conv3d_dense, lib.oracle_conv3d_kgs, lib.oracle_kgs_pack,
                  lib.oracle_maxpool3d, lib.oracle_conv3d_points, lib.oracle_num_threads,
                  lib.oracle_group_reweight):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().oracle_num_threads())


def set_threads(n: int) -> None:
    """Set the thread count of the oracle's OpenMP loops (for timing)."""
    _load().oracle_set_threads(int(n))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def out_shape(t, h, w, k, stride, pad):
    """Output (to, ho, wo) of a zero-padded strided correlation."""
    return tuple((i + 2 * p - kk) // s + 1 for i, kk, s, p in zip((t, h, w), k, stride, pad))


def _conv_common(x, w, bias, residual, stride, pad):
    x = _f64(x)
    w = _f64(w)
    n, c_in, t, h, ww = x.shape
    c_out, c_in2, kt, kh, kw = w.shape
    if c_in2 != c_in:
        raise ValueError("channel mismatch")
    to, ho, wo = out_shape(t, h, ww, (kt, kh, kw), stride, pad)
    y = np.empty((n, c_out, to, ho, wo), dtype=np.float64)
    b = None if bias is None else _f64(bias)
    r = None if residual is None else _f64(residual)
    if b is not None and b.shape != (c_out,):
        raise ValueError("bias shape")
    if r is not None and r.shape != y.shape:
        raise ValueError("residual shape")
    geo = [n, c_in, c_out, t, h, ww, kt, kh, kw, *stride, *pad]
    return x, w, b, r, y, geo


def conv3d_dense(x, w, bias=None, residual=None, stride=(1, 1, 1), pad=(0, 0, 0), relu=False):
    """Dense 3-D CONV, float64 (Section 3)."""
    x, w, b, r, y, geo = _conv_common(x, w, bias, residual, stride, pad)
    rc = _load().oracle_conv3d_dense(*geo, _ptr(x), _ptr(w), _ptr(b), _ptr(r), int(relu), _ptr(y))
    if rc:
        raise ValueError("oracle_conv3d_dense rejected its arguments")
    return y


def conv3d_kgs(x, w, mask, g_m, g_n, bias=None, residual=None, stride=(1, 1, 1), pad=(0, 0, 0),
               relu=False):
    """KGS-sparse 3-D CONV, float64 (Section 3, Fig. 1(b))."""
    x, w, b, r, y, geo = _conv_common(x, w, bias, residual, stride, pad)
    c_out, c_in, kt, kh, kw = w.shape
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    p_groups, q_groups = -(-c_out // g_m), -(-c_in // g_n)
    if m.shape != (p_groups, q_groups, kt * kh * kw):
        raise ValueError("mask shape %s, want %s" % (m.shape, (p_groups, q_groups, kt * kh * kw)))
    rc = _load().oracle_conv3d_kgs(*geo, g_m, g_n, _ptr(x), _ptr(w), m.ctypes.data, _ptr(b),
                                   _ptr(r), int(relu), _ptr(y))
    if rc:
        raise ValueError("oracle_conv3d_kgs rejected its arguments")
    return y


def conv3d_points(x, w, idx, mask=None, g_m=4, g_n=4, bias=None, residual=None,
                  stride=(1, 1, 1), pad=(0, 0, 0), relu=False):
    """Selected outputs of the KGS layer (dense when mask is None).

    ``idx`` holds flat indices into the [n][c_out][to][ho][wo] output; the
    result holds the same values the full layer would produce there.
    """
    x = _f64(x)
    w = _f64(w)
    n, c_in, t, h, ww = x.shape
    c_out, _, kt, kh, kw = w.shape
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape[0], dtype=np.float64)
    b = None if bias is None else _f64(bias)
    r = None if residual is None else _f64(residual)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if m is not None and m.shape != (-(-c_out // g_m), -(-c_in // g_n), kt * kh * kw):
        raise ValueError("mask shape")
    geo = [n, c_in, c_out, t, h, ww, kt, kh, kw, *stride, *pad, g_m, g_n]
    rc = _load().oracle_conv3d_points(*geo, _ptr(x), _ptr(w), None if m is None else m.ctypes.data,
                                      _ptr(b), _ptr(r), int(relu), idx.shape[0], idx.ctypes.data,
                                      _ptr(out))
    if rc:
        raise ValueError("oracle_conv3d_points rejected its arguments")
    return out


def kgs_pack(w, mask, g_m, g_n):
    """Compact per-group format (Section 3, reshaping paragraph).

    ``w`` may be any numpy dtype; its element bytes are copied verbatim.
    Returns (group_ptr u32, pos u16, val_ptr u64, vals with w's dtype).
    """
    w = np.ascontiguousarray(w)
    c_out, c_in, kt, kh, kw = w.shape
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    p_groups, q_groups = -(-c_out // g_m), -(-c_in // g_n)
    if m.shape != (p_groups, q_groups, kt * kh * kw):
        raise ValueError("mask shape")
    lib = _load()
    npos = ctypes.c_uint64()
    nval = ctypes.c_uint64()
    geo = [c_out, c_in, kt, kh, kw, g_m, g_n, w.itemsize]
    rc = lib.oracle_kgs_pack(*geo, w.ctypes.data, m.ctypes.data, None, None, None, None,
                             ctypes.addressof(npos), ctypes.addressof(nval))
    if rc:
        raise ValueError("oracle_kgs_pack rejected its arguments")
    group_ptr = np.zeros(p_groups * q_groups + 1, dtype=np.uint32)
    pos = np.zeros(max(npos.value, 1), dtype=np.uint16)
    val_ptr = np.zeros(p_groups * q_groups + 1, dtype=np.uint64)
    vals = np.zeros(max(nval.value, 1), dtype=w.dtype)
    rc = lib.oracle_kgs_pack(*geo, w.ctypes.data, m.ctypes.data, group_ptr.ctypes.data,
                             pos.ctypes.data, val_ptr.ctypes.data, vals.ctypes.data, None, None)
    if rc:
        raise ValueError("oracle_kgs_pack rejected its arguments")
    return group_ptr, pos[:npos.value], val_ptr, vals[:nval.value]


def maxpool3d(x, k, stride, pad=(0, 0, 0)):
    """3-D max pooling, floor output size; padded positions take no part."""
    x = _f64(x)
    n, c, t, h, w = x.shape
    to, ho, wo = out_shape(t, h, w, k, stride, pad)
    y = np.empty((n, c, to, ho, wo), dtype=np.float64)
    rc = _load().oracle_maxpool3d(n, c, t, h, w, *k, *stride, *pad, _ptr(x), _ptr(y))
    if rc:
        raise ValueError("oracle_maxpool3d rejected its arguments")
    return y


def group_reweight(w, g_m, g_n, norm=2, scope=0, pen=None, lam=1.0, eps=1e-6, tau=0.0, step=1.0,
                   grad=None):
    """Group norms and the reweighted group-lasso penalty, float64 (Section 4).

    ``w`` is [c_out][c_in][kt][kh][kw].  scope 0 takes one norm per kernel
    position of each kernel group (KGS), scope 1 one norm per whole group
    (vanilla).  ``pen`` holds the current penalty factors, one per norm
    (None = all ones).  ``grad`` (float64, w's shape) is accumulated into
    in place when given.  Returns a dict with ``norms`` and ``pen_next``
    ([P][Q][ks] or [P][Q]), ``reg`` (float), ``mask`` (uint8 [P][Q][ks]) and
    ``w_prox`` (w's shape).
    """
    w = _f64(w)
    c_out, c_in = w.shape[0], w.shape[1]
    ks = int(np.prod(w.shape[2:]))
    p_groups, q_groups = -(-c_out // g_m), -(-c_in // g_n)
    ushape = (p_groups, q_groups, ks) if scope == 0 else (p_groups, q_groups)
    p = None if pen is None else _f64(pen)
    if p is not None and p.shape != ushape:
        raise ValueError("pen shape %s, want %s" % (p.shape, ushape))
    if grad is not None and (grad.dtype != np.float64 or grad.shape != w.shape
                             or not grad.flags["C_CONTIGUOUS"]):
        raise ValueError("grad must be a C-contiguous float64 array of w's shape")
    norms = np.empty(ushape, dtype=np.float64)
    pen_next = np.empty(ushape, dtype=np.float64)
    mask = np.empty((p_groups, q_groups, ks), dtype=np.uint8)
    w_prox = np.empty(w.shape, dtype=np.float64)
    reg = ctypes.c_double()
    rc = _load().oracle_group_reweight(
        c_out, c_in, ks, g_m, g_n, norm, scope, _ptr(w), _ptr(p), float(lam), float(eps),
        float(tau), float(step), _ptr(norms), _ptr(pen_next),
        ctypes.cast(ctypes.addressof(reg), ctypes.POINTER(ctypes.c_double)), mask.ctypes.data,
        _ptr(grad), _ptr(w_prox))
    if rc:
        raise ValueError("oracle_group_reweight rejected its arguments")
    return {"norms": norms, "pen_next": pen_next, "reg": reg.value, "mask": mask,
            "w_prox": w_prox}
