"""ctypes binding of librt3d (include/rt3d.h), argument marshalling only.

Every computation runs in the HIP library; this module converts Python
arguments (torch tensors, numpy arrays) to the C ABI's pointers and sizes
and turns error codes into exceptions.  If the library has not been built it
raises: there is no CPU fallback.

Device tensors are channels-last and contiguous: x is [n, t, h, w, c_in],
y and residual are [n, to, ho, wo, c_out] (torch dtypes float32, bfloat16,
float16); bias is a float32 [c_out] device tensor; blobs are uint8 tensors.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librt3d.so")

RT3D_OK = 0
RT3D_ERR_INVALID_ARG = 1
RT3D_ERR_UNSUPPORTED = 2
RT3D_ERR_BUFFER_TOO_SMALL = 3
RT3D_ERR_BLOB_MISMATCH = 4
RT3D_ERR_HIP = 5

RT3D_F32 = 0
RT3D_BF16 = 1
RT3D_F16 = 2
RT3D_RELU = 1
RT3D_RESIDUAL = 2

DTYPE_CODES = {"f32": RT3D_F32, "bf16": RT3D_BF16, "f16": RT3D_F16}

EXPORTED = (
    "rt3d_status_string", "rt3d_last_error_detail", "rt3d_conv3d_out_shape",
    "rt3d_kgs_pack_size", "rt3d_kgs_pack", "rt3d_kgs_unpack", "rt3d_conv3d_workspace_size",
    "rt3d_kgs_conv3d_fwd", "rt3d_kgs_conv3d_fwd_noalloc", "rt3d_dense_pack_size", "rt3d_dense_pack", "rt3d_conv3d_dense_fwd",
    "rt3d_maxpool3d_fwd", "rt3d_group_units", "rt3d_group_workspace_size", "rt3d_group_reweight",
)

RT3D_SCOPE_KGS = 0
RT3D_SCOPE_VANILLA = 1


class Rt3dError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.detail = detail
        super().__init__("rt3d status %d (%s): %s" % (status, _status_name(status), detail))


class Conv3dDesc(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n", "c_in", "c_out", "t", "h", "w", "kt", "kh", "kw", "st", "sh", "sw",
        "pt", "ph", "pw", "g_m", "g_n", "dtype")] + [("flags", ctypes.c_uint32)] + [
        (name, ctypes.c_int32) for name in ("qt", "qh", "qw", "y_c_total", "y_c_off",
                                            "x_c_total", "x_c_off")]


class PackInfo(ctypes.Structure):
    _fields_ = [
        ("magic", ctypes.c_uint64), ("desc_hash", ctypes.c_uint64),
        ("version", ctypes.c_uint32), ("variant", ctypes.c_uint32),
        ("tile_groups", ctypes.c_uint32), ("vanilla", ctypes.c_uint32),
        ("packed_bytes", ctypes.c_uint64),
        ("canon_off", ctypes.c_uint64 * 4), ("canon_bytes", ctypes.c_uint64 * 4),
        ("derived_off", ctypes.c_uint64), ("derived_bytes", ctypes.c_uint64),
        ("kept_positions", ctypes.c_uint64), ("kept_weights", ctypes.c_uint64),
        ("plan", ctypes.c_uint64 * 16),
    ]


class GroupDesc(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "c_out", "c_in", "kt", "kh", "kw", "g_m", "g_n", "dtype", "norm", "scope")]


_lib = None


def load():
    """Load librt3d.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("librt3d.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    u64 = ctypes.c_uint64
    i32 = ctypes.c_int32
    D = P(Conv3dDesc)
    I = P(PackInfo)
    sig = {
        "rt3d_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "rt3d_last_error_detail": ([], ctypes.c_char_p),
        "rt3d_conv3d_out_shape": ([D, P(i32), P(i32), P(i32)], ctypes.c_int),
        "rt3d_kgs_pack_size": ([D, vp, P(u64)], ctypes.c_int),
        "rt3d_kgs_pack": ([D, vp, vp, vp, u64, I], ctypes.c_int),
        "rt3d_kgs_unpack": ([D, I, vp, vp], ctypes.c_int),
        "rt3d_conv3d_workspace_size": ([D, I, P(u64)], ctypes.c_int),
        "rt3d_kgs_conv3d_fwd": ([D, I, vp, vp, vp, vp, vp, vp, u64, vp], ctypes.c_int),
        "rt3d_kgs_conv3d_fwd_noalloc": ([D, I, vp, vp, vp, vp, vp, vp], ctypes.c_int),
        "rt3d_dense_pack_size": ([D, P(u64)], ctypes.c_int),
        "rt3d_dense_pack": ([D, vp, vp, u64, I], ctypes.c_int),
        "rt3d_conv3d_dense_fwd": ([D, I, vp, vp, vp, vp, vp, vp, u64, vp], ctypes.c_int),
        "rt3d_maxpool3d_fwd": ([i32] * 15 + [vp, vp, vp], ctypes.c_int),
        "rt3d_group_units": ([P(GroupDesc), P(ctypes.c_int64)], ctypes.c_int),
        "rt3d_group_workspace_size": ([P(GroupDesc), P(u64)], ctypes.c_int),
        "rt3d_group_reweight": ([P(GroupDesc), vp, vp] + [ctypes.c_float] * 4 + [vp] * 7 +
                                [u64, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _status_name(status: int) -> str:
    try:
        return load().rt3d_status_string(status).decode()
    except Exception:  # pragma: no cover - library missing while formatting an error
        return "?"


def _check(status: int):
    if status != RT3D_OK:
        raise Rt3dError(status, load().rt3d_last_error_detail().decode())


def make_desc(n, c_in, c_out, thw, k=(3, 3, 3), stride=(1, 1, 1), pad=(1, 1, 1), g=(4, 4),
              dtype="f32", relu=True, residual=False, pool=(1, 1, 1), y_c_total=0,
              y_c_off=0, x_c_total=0, x_c_off=0) -> Conv3dDesc:
    """Fill an rt3d_conv3d_desc (``pool``: fused max-pool window = stride;
    ``y_c_total`` / ``y_c_off``: write into a channel slice of a wider y;
    ``x_c_total`` / ``x_c_off``: read a channel slice of a wider x)."""
    flags = (RT3D_RELU if relu else 0) | (RT3D_RESIDUAL if residual else 0)
    code = DTYPE_CODES[dtype] if isinstance(dtype, str) else int(dtype)
    return Conv3dDesc(n, c_in, c_out, *thw, *k, *stride, *pad, g[0], g[1], code, flags, *pool,
                      y_c_total, y_c_off, x_c_total, x_c_off)


def _host_ptr(a: np.ndarray) -> int:
    if not a.flags["C_CONTIGUOUS"]:
        raise ValueError("host arrays must be C-contiguous")
    return a.ctypes.data


def _host_bytes(w) -> np.ndarray:
    """Raw element bytes of a host weight tensor (numpy array or CPU torch
    tensor, any of the three dtypes), C order."""
    try:
        import torch
        if isinstance(w, torch.Tensor):
            if w.is_cuda:
                raise ValueError("weights must be on the host")
            w = w.contiguous()
            return w.view(torch.uint8).numpy() if w.dtype != torch.uint8 else w.numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(w).view(np.uint8)


def _dev_ptr(t, name: str) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous (channels-last layout)" % name)
    return t.data_ptr()


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def rt3d_conv3d_out_shape(desc: Conv3dDesc) -> Tuple[int, int, int]:
    to, ho, wo = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(load().rt3d_conv3d_out_shape(ctypes.byref(desc), ctypes.byref(to), ctypes.byref(ho),
                                        ctypes.byref(wo)))
    return to.value, ho.value, wo.value


def rt3d_kgs_pack_size(desc: Conv3dDesc, mask: np.ndarray) -> int:
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    out = ctypes.c_uint64()
    _check(load().rt3d_kgs_pack_size(ctypes.byref(desc), _host_ptr(m), ctypes.byref(out)))
    return out.value


def rt3d_kgs_pack(desc: Conv3dDesc, w, mask: np.ndarray) -> Tuple[np.ndarray, PackInfo]:
    """Pack host weights [M][N][kt][kh][kw] + mask [P][Q][K_s]; returns the
    host blob (uint8 array) and its info."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    wb = _host_bytes(w)
    size = rt3d_kgs_pack_size(desc, m)
    blob = np.zeros(size, dtype=np.uint8)
    info = PackInfo()
    _check(load().rt3d_kgs_pack(ctypes.byref(desc), _host_ptr(wb), _host_ptr(m), _host_ptr(blob),
                                size, ctypes.byref(info)))
    return blob, info


def rt3d_kgs_unpack(desc: Conv3dDesc, info: PackInfo, blob: np.ndarray, out: np.ndarray) -> None:
    """Write W * expand(mask) into the host array ``out`` (dense layout)."""
    _check(load().rt3d_kgs_unpack(ctypes.byref(desc), ctypes.byref(info), _host_ptr(blob),
                                  _host_ptr(out)))


def rt3d_conv3d_workspace_size(desc: Conv3dDesc, info: PackInfo) -> int:
    out = ctypes.c_uint64()
    _check(load().rt3d_conv3d_workspace_size(ctypes.byref(desc), ctypes.byref(info),
                                             ctypes.byref(out)))
    return out.value


def rt3d_kgs_conv3d_fwd(desc: Conv3dDesc, info: PackInfo, blob_dev, x, bias, residual, y,
                        workspace=None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().rt3d_kgs_conv3d_fwd(
        ctypes.byref(desc), ctypes.byref(info), _dev_ptr(blob_dev, "blob"), _dev_ptr(x, "x"),
        _dev_ptr(bias, "bias"), _dev_ptr(residual, "residual"), _dev_ptr(y, "y"),
        _dev_ptr(workspace, "workspace"), ws_bytes, _stream_ptr(stream)))


def rt3d_kgs_conv3d_fwd_noalloc(desc: Conv3dDesc, info: PackInfo, blob_dev, x, bias, residual, y,
                                stream=None) -> None:
    """KGS forward whose split-K scratch is the library's own device array."""
    _check(load().rt3d_kgs_conv3d_fwd_noalloc(
        ctypes.byref(desc), ctypes.byref(info), _dev_ptr(blob_dev, "blob"), _dev_ptr(x, "x"),
        _dev_ptr(bias, "bias"), _dev_ptr(residual, "residual"), _dev_ptr(y, "y"),
        _stream_ptr(stream)))


def rt3d_dense_pack_size(desc: Conv3dDesc) -> int:
    out = ctypes.c_uint64()
    _check(load().rt3d_dense_pack_size(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def rt3d_dense_pack(desc: Conv3dDesc, w) -> Tuple[np.ndarray, PackInfo]:
    wb = _host_bytes(w)
    size = rt3d_dense_pack_size(desc)
    blob = np.zeros(size, dtype=np.uint8)
    info = PackInfo()
    _check(load().rt3d_dense_pack(ctypes.byref(desc), _host_ptr(wb), _host_ptr(blob), size,
                                  ctypes.byref(info)))
    return blob, info


def rt3d_conv3d_dense_fwd(desc: Conv3dDesc, info: PackInfo, blob_dev, x, bias, residual, y,
                          workspace=None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().rt3d_conv3d_dense_fwd(
        ctypes.byref(desc), ctypes.byref(info), _dev_ptr(blob_dev, "blob"), _dev_ptr(x, "x"),
        _dev_ptr(bias, "bias"), _dev_ptr(residual, "residual"), _dev_ptr(y, "y"),
        _dev_ptr(workspace, "workspace"), ws_bytes, _stream_ptr(stream)))


def rt3d_maxpool3d_fwd(x, y, k, stride, dtype: str, stream=None, pad=(0, 0, 0)) -> None:
    """x [n, t, h, w, c] -> y [n, to, ho, wo, c] (device, channels-last)."""
    n, t, h, w, c = x.shape
    _check(load().rt3d_maxpool3d_fwd(n, c, t, h, w, *k, *stride, *pad, DTYPE_CODES[dtype],
                                     _dev_ptr(x, "x"), _dev_ptr(y, "y"), _stream_ptr(stream)))


def canonical_sections(info: PackInfo, blob: np.ndarray, np_dtype) -> Tuple[np.ndarray, ...]:
    """Views of the four canonical sections of a host KGS blob."""
    def sec(i, dt):
        off, nb = info.canon_off[i], info.canon_bytes[i]
        return blob[off:off + nb].view(dt)
    return sec(0, np.uint32), sec(1, np.uint16), sec(2, np.uint64), sec(3, np_dtype)


def make_group_desc(c_out, c_in, k=(3, 3, 3), g=(4, 4), dtype="f32", norm=2,
                    scope=RT3D_SCOPE_KGS) -> GroupDesc:
    """Fill an rt3d_group_desc."""
    code = DTYPE_CODES[dtype] if isinstance(dtype, str) else int(dtype)
    return GroupDesc(c_out, c_in, *k, g[0], g[1], code, norm, scope)


def rt3d_group_units(desc: GroupDesc) -> int:
    out = ctypes.c_int64()
    _check(load().rt3d_group_units(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def rt3d_group_workspace_size(desc: GroupDesc) -> int:
    out = ctypes.c_uint64()
    _check(load().rt3d_group_workspace_size(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def rt3d_group_reweight(desc: GroupDesc, w, pen=None, lam=1.0, eps=1e-6, tau=0.0, step=1.0,
                        norms=None, pen_next=None, reg=None, mask=None, grad=None, w_prox=None,
                        workspace=None, stream=None) -> None:
    """Group norms / reweighted penalty over device weights ``w``
    [c_out, c_in, kt, kh, kw]; every output is an optional device tensor
    (float32 per unit, a float32 scalar ``reg``, uint8 mask [P, Q, K_s],
    float32 ``grad`` and ``w_prox`` of w's shape and dtype)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().rt3d_group_reweight(
        ctypes.byref(desc), _dev_ptr(w, "w"), _dev_ptr(pen, "pen"), float(lam), float(eps),
        float(tau), float(step), _dev_ptr(norms, "norms"), _dev_ptr(pen_next, "pen_next"),
        _dev_ptr(reg, "reg"), _dev_ptr(mask, "mask"), _dev_ptr(grad, "grad"),
        _dev_ptr(w_prox, "w_prox"), _dev_ptr(workspace, "workspace"), ws_bytes,
        _stream_ptr(stream)))
