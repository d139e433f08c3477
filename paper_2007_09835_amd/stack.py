"""Whole-network forward passes built from librt3d calls: the C3D conv stack
(eight 3x3x3 convs with max-pools) and the R(2+1)D-18-shaped stack
(factorised (2+1)-D convs with residual adds fused into the epilogue).

Only orchestration lives here: packing at construction, preallocated
activation buffers, and the sequence of C-ABI launches on one stream (so the
whole pass can also be captured in a HIP graph).  Weights are seeded and
synthetic (no trained models are available).
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import layers, synth


class Stack:
    """A stack of packed layers.  ``mode`` is "kgs" (KGS masks on the
    non-dense layers), "vanilla" (whole-group masks at ``rate``) or "dense"
    (every layer on the dense kernel)."""

    def __init__(self, net: str, batch: int = 1, dtype: str = "bf16", mode: str = "kgs",
                 rate: float = 3.0, tag: Optional[str] = None, device: str = "cuda",
                 fuse_pool: bool = True, group=(4, 4)):
        """``fuse_pool`` folds each max-pool into the preceding conv's
        epilogue; otherwise the pools run as separate kernels.  ``group`` is
        the kernel group size (g_M, g_N) of the KGS masks."""
        self.net, self.batch, self.dtype, self.mode, self.rate = net, batch, dtype, mode, rate
        self.fuse_pool = fuse_pool
        self.group = tuple(group)
        tag = tag or net
        if net == "c3d":
            self.layers = synth.c3d_stack(rate if mode == "kgs" else 3.0, tag=tag, g=self.group)
        elif net == "r2plus1d":
            self.layers = synth.r2plus1d_stack(tag=tag, g=self.group)
        else:
            raise ValueError(net)
        tdt = layers.TORCH_DTYPES[dtype]
        self.convs: List[layers.Conv3d] = []
        self.masks: List[Optional[np.ndarray]] = []
        for l in self.layers:
            d = synth.layer_params(tag, l, mask_kind=("dense" if mode == "dense" else mode),
                                   rate=rate)
            if l.dense or mode == "dense":
                mask = None
            else:
                mask = d.mask
            self.masks.append(None if l.dense else d.mask)
            w = synth.to_dtype(d.w, dtype)
            pool = l.pool_after[0] if (fuse_pool and l.pool_after) else (1, 1, 1)
            self.convs.append(layers.Conv3d(l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad,
                                            w, d.bias.astype(np.float32), mask, dtype,
                                            relu=l.relu, residual=l.residual_from is not None,
                                            g=l.g, device=device, batch=batch, pool=pool))
        # activation buffers (channels-last), allocated once
        self.x = torch.zeros((batch, self.layers[0].t, self.layers[0].h, self.layers[0].w,
                              self.layers[0].c_in), dtype=tdt, device=device)
        self.bufs: Dict[str, torch.Tensor] = {}
        self.pool_bufs: Dict[str, torch.Tensor] = {}
        for l, c in zip(self.layers, self.convs):
            self.bufs[l.name] = torch.empty(c.out_shape(batch), dtype=tdt, device=device)
            if l.pool_after and not fuse_pool:
                k, s = l.pool_after
                n, t, h, w, ch = c.out_shape(batch)
                self.pool_bufs[l.name] = torch.empty(
                    (n, (t - k[0]) // s[0] + 1, (h - k[1]) // s[1] + 1, (w - k[2]) // s[2] + 1, ch),
                    dtype=tdt, device=device)

    def kept_rate(self) -> float:
        """Whole-stack MAC pruning rate of the masks in use (1 when dense)."""
        if self.mode == "dense":
            return 1.0
        return synth.stack_rate(self.layers, self.masks)

    def dense_macs(self) -> int:
        return sum(l.dense_macs(self.batch) for l in self.layers)

    def executed_macs(self) -> int:
        """MACs of the kept weights (border positions counted nominally)."""
        if self.mode == "dense":
            return self.dense_macs()
        return int(round(self.dense_macs() / self.kept_rate()))

    def forward(self, x: Optional[torch.Tensor] = None, timers=None) -> torch.Tensor:
        """Run the stack on ``x`` (default: the internal input buffer).
        ``timers`` maps a layer index to a (start, end) event pair recorded
        around that layer's conv."""
        cur = self.x if x is None else x
        outs: Dict[str, torch.Tensor] = {}
        for i, (l, conv) in enumerate(zip(self.layers, self.convs)):
            inp = outs[l.input_from] if l.input_from else cur
            res = outs[l.residual_from] if l.residual_from else None
            ev = timers.get(i) if timers else None
            if ev:
                ev[0].record()
            y = conv(inp, res, out=self.bufs[l.name])
            if ev:
                ev[1].record()
            outs[l.name] = y
            if l.pool_after and not self.fuse_pool:
                k, s = l.pool_after
                y = layers.maxpool3d(y, k, s, self.dtype, out=self.pool_bufs[l.name])
                outs[l.name] = y
            cur = y
        return cur
