"""Whole-network forward passes built from librt3d calls: the C3D conv stack
(eight 3x3x3 convs with max-pools), the R(2+1)D-18-shaped stack
(factorised (2+1)-D convs with residual adds fused into the epilogue) and
the S3D-shaped stack (Inception blocks whose branches write channel slices
of one output, separable convs, padded max-pools).

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
        # A layer output whose channel count is not a multiple of 8 (the
        # R(2+1)D mid widths) gets a channel pitch rounded up to 8, so the
        # next layer stages its halo with whole 16-byte loads; the pad
        # channels stay zero.  Residual sources keep their exact width.
        self.bufs: Dict[str, torch.Tensor] = {}
        self.pool_bufs: Dict[str, torch.Tensor] = {}
        residual_sources = {l.residual_from for l in self.layers if l.residual_from}
        for l, c in zip(self.layers, self.convs):
            shape = list(c.out_shape(batch))
            if shape[-1] % 8 and l.name not in residual_sources:
                shape[-1] = (shape[-1] + 7) // 8 * 8
            self.bufs[l.name] = torch.zeros(shape, dtype=tdt, device=device)
            if l.pool_after and not fuse_pool:
                k, s = l.pool_after
                n, t, h, w, ch = self.bufs[l.name].shape
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

    def layer_calls(self):
        """(layer, fn) for every conv: fn launches that conv alone on the
        buffers a forward pass gives it (for per-layer timing)."""
        calls = []
        cur = self.x
        for l, conv in zip(self.layers, self.convs):
            inp = self.bufs[l.input_from] if l.input_from else cur
            res = self.bufs[l.residual_from] if l.residual_from else None
            calls.append((l, lambda conv=conv, inp=inp, res=res, o=self.bufs[l.name]:
                          conv(inp, res, out=o)))
            cur = self.pool_bufs.get(l.name, self.bufs[l.name])
        return calls

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


class S3DStack:
    """The S3D-shaped stack (synth.s3d_layers): convs and padded max-pools
    over named buffers; the four branches of an Inception block write their
    channel slices of the block output directly (fused concatenation)."""

    net = "s3d"

    def __init__(self, batch: int = 1, dtype: str = "bf16", mode: str = "kgs",
                 rate: float = 2.1, tag: str = "s3d", device: str = "cuda", group=(4, 4),
                 clip=(16, 224), n_streams: int = 2):
        """``clip`` = (frames, height = width) of the input; ``n_streams``
        streams run independent ops concurrently (1 = strictly in order)."""
        self.batch, self.dtype, self.mode, self.rate = batch, dtype, mode, rate
        self.group = tuple(group)
        self.layers, self.ops = synth.s3d_stack(rate if mode == "kgs" else 2.1, tag=tag,
                                                g=self.group, clip=tuple(clip))
        tdt = layers.TORCH_DTYPES[dtype]
        self.convs, self.masks = [], []
        by_name = {}
        for l in self.layers:
            d = synth.layer_params(tag, l, mask_kind=("dense" if mode == "dense" else mode),
                                   rate=rate)
            mask = None if (l.dense or mode == "dense") else d.mask
            self.masks.append(None if l.dense else d.mask)
            conv = layers.Conv3d(l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad,
                                 synth.to_dtype(d.w, dtype), d.bias.astype(np.float32), mask,
                                 dtype, relu=l.relu, g=l.g, device=device, batch=batch)
            self.convs.append(conv)
            by_name[l.name] = (l, conv)
        self._by_name = by_name
        # buffer shapes from the op list
        l0 = self.layers[0]
        shapes = {"x": (l0.t, l0.h, l0.w, l0.c_in)}
        for op in self.ops:
            if op[0] == "conv":
                _, name, src, dst, c_off, _ = op
                l, conv = by_name[name]
                c_prev = shapes.get(dst, (0, 0, 0, 0))[3]
                shapes[dst] = (*conv.out_thw, max(c_prev, c_off + l.c_out))
            else:
                _, src, dst, k, st, pd = op
                t, h, w, c = shapes[src]
                shapes[dst] = (*((i + 2 * p - kk) // s + 1
                                 for i, kk, s, p in zip((t, h, w), k, st, pd)), c)
        self.x = torch.zeros((batch, *shapes["x"]), dtype=tdt, device=device)
        self.bufs: Dict[str, torch.Tensor] = {"x": self.x}
        for name, shp in shapes.items():
            if name != "x":
                self.bufs[name] = torch.empty((batch, *shp), dtype=tdt, device=device)
        self.pool_bufs: Dict[str, torch.Tensor] = {}
        self.out_name = self.ops[-1][3]
        self._schedule(n_streams)

    def _schedule(self, n_streams: int):
        """Dependencies between ops by the channel ranges they read and
        write (branches of a block write disjoint slices of one buffer), and a
        stream per op: an op continues the stream of a dependency that stream
        ended with, else takes the least recently used stream.  The branches
        of a block then run concurrently."""
        def ranges(op):
            if op[0] == "conv":
                _, name, src, dst, c_off, x_off = op
                l, _ = self._by_name[name]
                return [(src, x_off, x_off + l.c_in)], [(dst, c_off, c_off + l.c_out)]
            _, src, dst, *_ = op
            c = self.bufs[src].shape[-1]
            return [(src, 0, c)], [(dst, 0, c)]
        writers: Dict[str, list] = {}   # buffer -> [(c0, c1, op index)]
        self.deps: List[List[int]] = []
        for i, op in enumerate(self.ops):
            reads, writes = ranges(op)
            d = set()
            for buf, c0, c1 in reads:
                for w0, w1, j in writers.get(buf, []):
                    if w0 < c1 and c0 < w1:
                        d.add(j)
            for buf, c0, c1 in writes:
                writers.setdefault(buf, []).append((c0, c1, i))
            self.deps.append(sorted(d))
        self.stream_of: List[int] = []
        last = [-1] * max(1, n_streams)      # last op issued on each stream
        used = [0] * len(last)
        for i, d in enumerate(self.deps):
            pick = next((s for s in range(len(last)) if last[s] in d), None)
            if pick is None:
                pick = min(range(len(last)), key=lambda s: used[s])
            self.stream_of.append(pick)
            last[pick] = i
            used[pick] = i + 1
        self.streams = [None] + [torch.cuda.Stream() for _ in range(len(last) - 1)]
        self.events = [torch.cuda.Event() for _ in self.ops]

    def kept_rate(self) -> float:
        if self.mode == "dense":
            return 1.0
        return synth.stack_rate(self.layers, self.masks)

    def dense_macs(self) -> int:
        return sum(l.dense_macs(self.batch) for l in self.layers)

    def layer_calls(self):
        calls = []
        for op in self.ops:
            if op[0] == "conv":
                _, name, src, dst, c_off, x_off = op
                l, conv = self._by_name[name]
                calls.append((l, lambda conv=conv, i=self.bufs[src], o=self.bufs[dst], c=c_off,
                              xo=x_off: conv(i, None, out=o, c_off=c, x_off=xo)))
        return calls

    def forward(self, x: Optional[torch.Tensor] = None) -> torch.Tensor:
        """One pass.  Ops run on the current stream and up to n_streams - 1
        side streams, forked from it and joined back at the end (so the pass
        can be captured in one HIP graph)."""
        if x is not None:
            self.x.copy_(x)
        main = torch.cuda.current_stream()
        streams = [main] + self.streams[1:]
        for st in streams[1:]:
            st.wait_stream(main)
        for i, op in enumerate(self.ops):
            st = streams[self.stream_of[i]]
            for j in self.deps[i]:
                if self.stream_of[j] != self.stream_of[i]:
                    st.wait_event(self.events[j])
            if op[0] == "conv":
                _, name, src, dst, c_off, x_off = op
                _, conv = self._by_name[name]
                conv(self.bufs[src], None, out=self.bufs[dst], c_off=c_off, x_off=x_off, stream=st)
            else:
                _, src, dst, k, stv, pd = op
                layers.maxpool3d(self.bufs[src], k, stv, self.dtype, out=self.bufs[dst], pad=pd,
                                 stream=st)
            self.events[i].record(st)
        for st in streams[1:]:
            main.wait_stream(st)
        return self.bufs[self.out_name]


def make_stack(net: str, batch: int = 1, dtype: str = "bf16", mode: str = "kgs",
               rate: float = 3.0, fuse_pool: bool = True, group=(4, 4), streams: int = 2):
    """The named stack (c3d, r2plus1d or s3d; ``streams`` applies to s3d)."""
    if net == "s3d":
        return S3DStack(batch, dtype, mode, rate, group=group, n_streams=streams)
    return Stack(net, batch, dtype, mode, rate, fuse_pool=fuse_pool, group=group)
