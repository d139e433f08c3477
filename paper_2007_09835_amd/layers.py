"""Layer objects over the C ABI: pack once on the host, keep the blob and
bias on the device, launch the HIP kernels per call.

Memory management and argument marshalling only; every arithmetic step of a
forward pass runs in librt3d's kernels.  Activations are channels-last
contiguous device tensors [n, t, h, w, c].
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np
import torch

from . import rt3d

TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


class Conv3d:
    """One packed 3-D convolution (dense when ``mask`` is None, else KGS).

    ``w`` is a host tensor [M][N][kt][kh][kw] already in the layer dtype;
    ``bias`` a host float array [M] (or None); ``mask`` uint8 [P][Q][K_s].
    """

    def __init__(self, c_in: int, c_out: int, thw: Sequence[int], k, stride, pad, w,
                 bias=None, mask: Optional[np.ndarray] = None, dtype: str = "bf16",
                 relu: bool = True, residual: bool = False, g=(4, 4), device="cuda",
                 batch: int = 1, pool=(1, 1, 1)):
        """``batch`` is the batch size the layer is planned for (the blob
        works for any batch; the tile shapes are chosen for this one).
        ``pool`` fuses a max-pool (window = stride) after the activation."""
        self.dtype = dtype
        self.sparse = mask is not None
        self.desc = rt3d.make_desc(batch, c_in, c_out, tuple(thw), tuple(k), tuple(stride),
                                   tuple(pad), tuple(g), dtype, relu=relu, residual=residual,
                                   pool=tuple(pool))
        if self.sparse:
            blob, self.info = rt3d.rt3d_kgs_pack(self.desc, w, mask)
        else:
            blob, self.info = rt3d.rt3d_dense_pack(self.desc, w)
        self.blob = torch.from_numpy(blob).to(device)
        self.bias = None if bias is None else torch.as_tensor(
            np.asarray(bias, dtype=np.float32)).to(device)
        self.out_thw = rt3d.rt3d_conv3d_out_shape(self.desc)
        self.c_out = c_out
        self.device = device
        self._ws = {}

    def desc_for(self, n: int) -> rt3d.Conv3dDesc:
        d = rt3d.Conv3dDesc.from_buffer_copy(self.desc)
        d.n = n
        return d

    def out_shape(self, n: int):
        return (n, *self.out_thw, self.c_out)

    def workspace(self, n: int) -> Optional[torch.Tensor]:
        """Split-K workspace for batch n (allocated once per batch size)."""
        if n not in self._ws:
            nbytes = rt3d.rt3d_conv3d_workspace_size(self.desc_for(n), self.info)
            self._ws[n] = (None if nbytes == 0 else
                           torch.empty(nbytes // 4, dtype=torch.float32, device=self.device))
        return self._ws[n]

    def __call__(self, x: torch.Tensor, residual: Optional[torch.Tensor] = None,
                 out: Optional[torch.Tensor] = None, stream=None,
                 use_workspace: bool = True, c_off: int = 0, x_off: int = 0) -> torch.Tensor:
        """``out`` may hold more channels than c_out: the layer then writes
        channels [c_off, c_off + c_out) of it (fused concatenation); ``x``
        may hold more channels than c_in: the layer reads [x_off, x_off +
        c_in) of it."""
        n = x.shape[0]
        if out is None:
            out = torch.empty(self.out_shape(n), dtype=TORCH_DTYPES[self.dtype], device=x.device)
        ws = self.workspace(n) if use_workspace and n > 0 else None
        d = self.desc_for(n)
        if out.shape[-1] != self.c_out or c_off:
            d.y_c_total, d.y_c_off = out.shape[-1], c_off
        if x.shape[-1] != d.c_in or x_off:
            d.x_c_total, d.x_c_off = x.shape[-1], x_off
        fwd = rt3d.rt3d_kgs_conv3d_fwd if self.sparse else rt3d.rt3d_conv3d_dense_fwd
        fwd(d, self.info, self.blob, x, self.bias, residual, out, ws, stream)
        return out


def maxpool3d(x: torch.Tensor, k, stride, dtype: str, out: Optional[torch.Tensor] = None,
              stream=None, pad=(0, 0, 0)) -> torch.Tensor:
    n, t, h, w, c = x.shape
    to, ho, wo = ((t + 2 * pad[0] - k[0]) // stride[0] + 1, (h + 2 * pad[1] - k[1]) // stride[1] + 1,
                  (w + 2 * pad[2] - k[2]) // stride[2] + 1)
    if out is None:
        out = torch.empty((n, to, ho, wo, c), dtype=x.dtype, device=x.device)
    rt3d.rt3d_maxpool3d_fwd(x, out, k, stride, dtype, stream, pad)
    return out
