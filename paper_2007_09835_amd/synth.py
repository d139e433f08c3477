"""Seeded synthetic workloads: layer shape tables, masks, weights, inputs.

This module holds no convolution arithmetic; it only decides shapes and draws
random numbers, so that the GPU path and the CPU oracle see identical bytes.

The paper evaluates on UCF101 clips with pretrained C3D / R(2+1)D weights
(Section 5, experimental setup), none of which exist here.  The stand-ins keep
the paper's shapes: 16-frame 112x112 RGB clips, the C3D conv stack and an
R(2+1)D-18-shaped stack, kernel groups of g_M = g_N = 4 (Section 3: g_N = 4,
g_M = 4 or 8), and masks drawn uniformly per group.

RNG: numpy ``Generator(PCG64(SeedSequence([2007_09835, *keys])))`` where the
keys name the workload, the layer and the role of the tensor, so every tensor
is reproducible on its own.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import List, Optional, Sequence, Tuple

import numpy as np

SEED = 2007_09835
GROUP = 4  # g_M = g_N = 4 in every workload


def _key(k) -> int:
    if isinstance(k, (int, np.integer)):
        return int(k) & 0xFFFFFFFF
    return zlib.crc32(str(k).encode())


def rng_for(*keys) -> np.random.Generator:
    """Independent generator for one (workload, layer, role) tuple."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, *map(_key, keys)])))


@dataclasses.dataclass
class ConvLayer:
    """One 3-D CONV layer of a workload (shapes only)."""
    name: str
    c_in: int
    c_out: int
    t: int
    h: int
    w: int
    k: Tuple[int, int, int]            # (kt, kh, kw); kt is the kernel depth K_d
    stride: Tuple[int, int, int] = (1, 1, 1)
    pad: Tuple[int, int, int] = (0, 0, 0)
    dense: bool = False                # kept dense in the workload (no KGS mask)
    relu: bool = True
    residual_from: Optional[str] = None  # name of the tensor added before ReLU
    input_from: Optional[str] = None     # name of the tensor this layer reads (None: previous)
    pool_after: Optional[Tuple[Tuple[int, int, int], Tuple[int, int, int]]] = None
    keep: Optional[int] = None         # kept positions per group (KGS layers)
    g: Tuple[int, int] = (GROUP, GROUP)  # kernel group size (g_M filters, g_N channels)
    group_rate: Optional[float] = None   # 1x1x1 KGS layers: whole-group pruning rate

    @property
    def ks(self) -> int:
        return self.k[0] * self.k[1] * self.k[2]

    @property
    def out_thw(self) -> Tuple[int, int, int]:
        return tuple((i + 2 * p - k) // s + 1
                     for i, k, s, p in zip((self.t, self.h, self.w), self.k, self.stride, self.pad))

    @property
    def voxels_out(self) -> int:
        to, ho, wo = self.out_thw
        return to * ho * wo

    @property
    def groups(self) -> Tuple[int, int]:
        return -(-self.c_out // self.g[0]), -(-self.c_in // self.g[1])

    def dense_macs(self, batch: int = 1) -> int:
        """Multiply-accumulates of the dense layer (the paper's "FLOPs")."""
        return batch * self.voxels_out * self.c_out * self.c_in * self.ks


# --------------------------------------------------------------------------
# Shape tables
# --------------------------------------------------------------------------

def c3d_layers() -> List[ConvLayer]:
    """C3D convolution stack on one 16x112x112 clip: eight 3x3x3 pad-1 convs
    with ReLU, max-pool 1x2x2 after conv1 and 2x2x2 after conv2/3b/4b."""
    p1 = ((1, 2, 2), (1, 2, 2))
    p2 = ((2, 2, 2), (2, 2, 2))
    spec = [("conv1", 3, 64, 16, 112, p1, True),
            ("conv2", 64, 128, 16, 56, p2, False),
            ("conv3a", 128, 256, 8, 28, None, False),
            ("conv3b", 256, 256, 8, 28, p2, False),
            ("conv4a", 256, 512, 4, 14, None, False),
            ("conv4b", 512, 512, 4, 14, p2, False),
            ("conv5a", 512, 512, 2, 7, None, False),
            ("conv5b", 512, 512, 2, 7, None, False)]
    return [ConvLayer(n, ci, co, t, hw, hw, (3, 3, 3), (1, 1, 1), (1, 1, 1), dense=d, relu=True,
                      pool_after=pool)
            for n, ci, co, t, hw, pool, d in spec]


def r2plus1d_mid(n_in: int, n_out: int) -> int:
    """Mid-width of a (2+1)-D factorised conv with the parameter count of the
    full 3x3x3 conv it replaces: floor(27 N_i N_o / (9 N_i + 3 N_o))."""
    return (27 * n_in * n_out) // (9 * n_in + 3 * n_out)


def r2plus1d_layers() -> List[ConvLayer]:
    """R(2+1)D-18-shaped stack on one 16x112x112 clip.

    Stem: 1x7x7 stride (1,2,2) 3->45 then 3x1x1 45->64 (both dense).  Four
    stages of two residual blocks at widths 64/128/256/512; a block is two
    (2+1)-D convs, each a 1x3x3 spatial conv to the mid-width followed by a
    3x1x1 temporal conv; the first block of stages 3-5 is strided by 2 in
    T, H and W and has a dense 1x1x1 stride-2 shortcut.  The residual add and
    the final ReLU of a block are fused into its last temporal conv.
    """
    layers: List[ConvLayer] = []
    t, hw = 16, 112
    layers.append(ConvLayer("stem_s", 3, 45, t, hw, hw, (1, 7, 7), (1, 2, 2), (0, 3, 3), dense=True))
    hw = 56
    layers.append(ConvLayer("stem_t", 45, 64, t, hw, hw, (3, 1, 1), (1, 1, 1), (1, 0, 0), dense=True))
    prev = "stem_t"
    c = 64
    for stage, width in enumerate((64, 128, 256, 512), start=2):
        for blk in range(2):
            s = 2 if (blk == 0 and stage > 2) else 1
            block_in = prev
            shortcut = block_in
            if s == 2:
                sc = ConvLayer(f"l{stage}b{blk}_down", c, width, t, hw, hw, (1, 1, 1), (2, 2, 2),
                               (0, 0, 0), dense=True, relu=False, input_from=block_in)
                layers.append(sc)
                shortcut = sc.name
            cin = c
            for conv in range(2):
                st = s if conv == 0 else 1
                mid = r2plus1d_mid(cin, width)
                sp = ConvLayer(f"l{stage}b{blk}c{conv}_s", cin, mid, t, hw, hw, (1, 3, 3),
                               (1, st, st), (0, 1, 1), input_from=(block_in if conv == 0 else None))
                layers.append(sp)
                t2, hw2 = t, (hw + 2 - 3) // st + 1
                last = conv == 1
                tp = ConvLayer(f"l{stage}b{blk}c{conv}_t", mid, width, t2, hw2, hw2, (3, 1, 1),
                               (st, 1, 1), (1, 0, 0), relu=True,
                               residual_from=(shortcut if last else None))
                layers.append(tp)
                t, hw = (t2 + 2 - 3) // st + 1, hw2
                cin = width
            c = width
            prev = layers[-1].name
    return layers


# S3D (Inception-style blocks with separable convs).  Each entry of the op
# list is ("conv", layer name, input buffer, output buffer, channel offset)
# or ("pool", input buffer, output buffer, window, stride, padding).
S3D_MIXED = [  # name, in, b0, b1 reduce, b1, b2 reduce, b2, b3
    ("m3b", 192, 64, 96, 128, 16, 32, 32),
    ("m3c", 256, 128, 128, 192, 32, 96, 64),
    ("m4b", 480, 192, 96, 208, 16, 48, 64),
    ("m4c", 512, 160, 112, 224, 24, 64, 64),
    ("m4d", 512, 128, 128, 256, 24, 64, 64),
    ("m4e", 512, 112, 144, 288, 32, 64, 64),
    ("m4f", 528, 256, 160, 320, 32, 128, 128),
    ("m5b", 832, 256, 160, 320, 32, 128, 128),
    ("m5c", 832, 384, 192, 384, 48, 128, 128),
]


def s3d_layers(t: int = 16, hw: int = 224) -> Tuple[List[ConvLayer], list]:
    """S3D-shaped conv stack on one t x hw x hw RGB clip: a separable 7x7x7
    stem (1x7x7 stride (1,2,2), then 7x1x1 stride (2,1,1)), max-pool 1x3x3
    stride (1,2,2), 1x1x1 and separable 3x3x3 convs, max-pool, then nine
    Inception blocks (mixed 3b-3c, 4b-4f, 5b-5c) separated by 3x3x3 / 2x2x2
    stride-2 pools.  A block's branches are 1x1x1; 1x1x1 then separable 3x3x3
    (1x3x3 then 3x1x1); the same with other widths; 3x3x3 stride-1 max-pool
    then 1x1x1.  Every conv has a ReLU (batch-norm folded into weights and
    bias).

    The three 1x1x1 convs that read the block input are one conv (their
    filters concatenated, written [b1 reduce | b2 reduce | b0] into the block
    buffer), and every branch writes its slice of that buffer, so a block
    buffer holds [b1 reduce | b2 reduce | b0 | b1 | b2 | b3] and the next
    block reads its channels from b0 on.  Returns (layers, ops): an op is
    ("conv", layer, input buffer, output buffer, output channel offset,
    input channel offset) or ("pool", input, output, window, stride, pad)."""
    layers: List[ConvLayer] = []
    ops: list = []
    shapes = {"x": (3, t, hw, hw)}   # buffer -> (channels per voxel, t, h, w)

    def conv(name, src, dst, c_out, k, stride=(1, 1, 1), pad=(0, 0, 0), c_off=0, dense=False,
             x_off=0, c_in=None):
        c_buf, ti, hi, wi = shapes[src]
        c_in = c_buf - x_off if c_in is None else c_in
        l = ConvLayer(name, c_in, c_out, ti, hi, wi, k, stride, pad, dense=dense)
        layers.append(l)
        ops.append(("conv", name, src, dst, c_off, x_off))
        c_prev = shapes.get(dst, (0,))[0]
        shapes[dst] = (max(c_prev, c_off + c_out), *l.out_thw)
        return l.out_thw

    def pool(src, dst, k, stride, pad):
        c, ti, hi, wi = shapes[src]
        out = tuple((i + 2 * p - kk) // s + 1 for i, kk, s, p in zip((ti, hi, wi), k, stride, pad))
        ops.append(("pool", src, dst, k, stride, pad))
        shapes[dst] = (c, *out)

    def sep(name, src, dst, c_out, c_off=0, k=3, stride=(1, 1, 1), dense=False, x_off=0,
            c_in=None):
        pk = k // 2
        conv(name + "_s", src, name + "_s", c_out, (1, k, k), (1, stride[1], stride[2]),
             (0, pk, pk), dense=dense, x_off=x_off, c_in=c_in)
        conv(name + "_t", name + "_s", dst, c_out, (k, 1, 1), (stride[0], 1, 1), (pk, 0, 0),
             c_off=c_off)

    sep("c1a", "x", "c1a", 64, k=7, stride=(2, 2, 2), dense=True)
    layers[-1].dense = False  # only the spatial stem conv (3 input channels) stays dense
    pool("c1a", "p2a", (1, 3, 3), (1, 2, 2), (0, 1, 1))
    conv("c2b", "p2a", "c2b", 64, (1, 1, 1))
    sep("c2c", "c2b", "c2c", 192)
    pool("c2c", "p3a", (1, 3, 3), (1, 2, 2), (0, 1, 1))
    cur, cur_off = "p3a", 0
    for name, c_in, b0, b1r, b1, b2r, b2, b3 in S3D_MIXED:
        if name == "m4b":
            pool(cur, "p4a", (3, 3, 3), (2, 2, 2), (1, 1, 1))
            cur = "p4a"
        if name == "m5b":
            pool(cur, "p5a", (2, 2, 2), (2, 2, 2), (0, 0, 0))
            cur = "p5a"
        e = b1r + b2r + b0
        conv(name + "_e", cur, name, e, (1, 1, 1), x_off=cur_off, c_in=c_in)
        sep(name + "_b1", name, name, b1, c_off=e, x_off=0, c_in=b1r)
        sep(name + "_b2", name, name, b2, c_off=e + b1, x_off=b1r, c_in=b2r)
        pool(cur, name + "_p", (3, 3, 3), (1, 1, 1), (1, 1, 1))
        conv(name + "_b3", name + "_p", name, b3, (1, 1, 1), c_off=e + b1 + b2, x_off=cur_off,
             c_in=c_in)
        cur, cur_off = name, b1r + b2r
    return layers, ops


def s3d_stack(rate: float = 2.1, tag: str = "s3d", g: Tuple[int, int] = (GROUP, GROUP),
              clip: Tuple[int, int] = (16, 224)) -> Tuple[List[ConvLayer], list]:
    """S3D stack with KGS masks for a whole-stack MAC pruning rate of about
    ``rate`` (the 3-channel stem conv stays dense, so the other layers are
    pruned at r = (D - D_dense) / (D / rate - D_dense)): kernels of K_s
    positions keep K_s / r of them per group (randomised rounding per
    layer), 1x1x1 layers keep round(P*Q/r) whole groups."""
    layers, ops = s3d_layers(*clip)
    r = rng_for(tag, "keep", int(rate * 1000))
    d_total = sum(l.dense_macs() for l in layers)
    d_dense = sum(l.dense_macs() for l in layers if l.dense)
    layer_rate = (d_total - d_dense) / (d_total / rate - d_dense) if rate > 1.0 else 1.0
    for l in layers:
        l.g = tuple(g)
        if l.dense or rate <= 1.0:
            continue
        if l.ks == 1:
            l.group_rate = layer_rate
        else:
            kstar = l.ks / layer_rate
            lo = int(np.floor(kstar))
            l.keep = min(l.ks, max(1, lo + int(r.random() < kstar - lo)))
    return layers, ops


# --------------------------------------------------------------------------
# Masks
# --------------------------------------------------------------------------

def kgs_mask(rng: np.random.Generator, p_groups: int, q_groups: int, ks: int,
             keep) -> np.ndarray:
    """KGS mask [P][Q][K_s]: for every group (p-major, q-minor) keep ``keep``
    kernel positions drawn uniformly without replacement.  ``keep`` may be an
    int or a [P][Q] array of per-group counts."""
    keep_arr = np.broadcast_to(np.asarray(keep, dtype=np.int64), (p_groups, q_groups))
    mask = np.zeros((p_groups, q_groups, ks), dtype=np.uint8)
    for p in range(p_groups):
        for q in range(q_groups):
            k = int(keep_arr[p, q])
            if k:
                mask[p, q, rng.choice(ks, size=k, replace=False)] = 1
    return mask


def vanilla_mask(rng: np.random.Generator, p_groups: int, q_groups: int, ks: int,
                 rate: float) -> np.ndarray:
    """Vanilla structured mask: round(P*Q/rate) whole groups kept, chosen
    uniformly without replacement; every other group is pruned entirely."""
    n_keep = int(round(p_groups * q_groups / rate))
    mask = np.zeros((p_groups * q_groups, ks), dtype=np.uint8)
    mask[rng.choice(p_groups * q_groups, size=n_keep, replace=False)] = 1
    return mask.reshape(p_groups, q_groups, ks)


def stack_keep_counts(layers: Sequence[ConvLayer], rate: float, tag: str,
                      band: float = 0.05) -> List[Optional[int]]:
    """Per-layer kept positions for a whole-stack MAC pruning rate ``rate``.

    Uniform solution k* = K_s (D/R - D_dense) / (D - D_dense), randomised
    rounding to floor/ceil with probability frac(k*), then a greedy repair
    (one position at a time on the layer that brings the rate closest to the
    target) until the rate lies within ``rate +- band``.
    """
    rng = rng_for(tag, "keep", int(rate * 1000))
    d_total = sum(l.dense_macs() for l in layers)
    d_dense = sum(l.dense_macs() for l in layers if l.dense)
    if rate <= 1.0:
        return [None if l.dense else l.ks for l in layers]
    ks = [l.ks for l in layers if not l.dense]
    if len(set(ks)) != 1:
        raise ValueError("uniform k* needs one kernel volume")
    kstar = ks[0] * (d_total / rate - d_dense) / (d_total - d_dense)
    keep: List[Optional[int]] = []
    for l in layers:
        if l.dense:
            keep.append(None)
        else:
            lo = int(np.floor(kstar))
            keep.append(min(l.ks, max(1, lo + int(rng.random() < kstar - lo))))

    def achieved(kp):
        kept = sum(l.dense_macs() * (1.0 if k is None else k / l.ks) for l, k in zip(layers, kp))
        return d_total / kept

    for _ in range(1000):
        r = achieved(keep)
        if abs(r - rate) <= band:
            return keep
        step = 1 if r > rate else -1
        best, best_err = None, None
        for i, (l, k) in enumerate(zip(layers, keep)):
            if k is None or not (1 <= k + step <= l.ks):
                continue
            trial = list(keep)
            trial[i] = k + step
            err = abs(achieved(trial) - rate)
            if best_err is None or err < best_err:
                best, best_err = i, err
        if best is None:
            break
        keep[best] += step
    raise ValueError("could not reach the requested pruning rate")


def stack_rate(layers: Sequence[ConvLayer], masks: Sequence[Optional[np.ndarray]]) -> float:
    """Whole-stack pruning rate: dense MACs over kept MACs, where a KGS layer
    keeps V * sum over groups of g_m_eff * g_n_eff * k (border positions are
    counted nominally, as the paper's FLOP counts do)."""
    dense = 0
    kept = 0
    for l, m in zip(layers, masks):
        d = l.dense_macs()
        dense += d
        if m is None:
            kept += d
        else:
            kept += l.voxels_out * kept_weights(l, m)
    return dense / kept


def kept_weights(l: ConvLayer, mask: np.ndarray) -> int:
    """Number of weights kept by a mask: sum over groups of g_m_eff*g_n_eff*k."""
    p_groups, q_groups = l.groups
    gm = np.full(p_groups, l.g[0])
    gm[-1] = l.c_out - l.g[0] * (p_groups - 1)
    gn = np.full(q_groups, l.g[1])
    gn[-1] = l.c_in - l.g[1] * (q_groups - 1)
    k = mask.sum(axis=2, dtype=np.int64)
    return int((gm[:, None] * gn[None, :] * k).sum())


# --------------------------------------------------------------------------
# Tensors
# --------------------------------------------------------------------------

def to_dtype(a: np.ndarray, dtype: str):
    """Round a float64 array to the workload dtype (round-to-nearest-even)
    and return it as a CPU torch tensor of that dtype."""
    import torch
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).to(tdt)


def kaiming(rng: np.random.Generator, c_out: int, c_in: int, k: Tuple[int, int, int]) -> np.ndarray:
    """Kaiming-normal weights N(0, 2 / (c_in * kt * kh * kw))."""
    fan_in = c_in * k[0] * k[1] * k[2]
    return rng.normal(0.0, np.sqrt(2.0 / fan_in), size=(c_out, c_in, *k))


def unit_scaled_weights(rng: np.random.Generator, c_out: int, c_in: int, k: Tuple[int, int, int],
                        g: Tuple[int, int], lo: float = 0.02) -> np.ndarray:
    """Kaiming-normal weights with one log-uniform scale in [lo, 1] per kernel
    group and kernel position, standing in for trained weights whose group
    norms spread over orders of magnitude (the input of the group-lasso
    penalty; no trained weights are available)."""
    w = kaiming(rng, c_out, c_in, k)
    p_groups, q_groups = -(-c_out // g[0]), -(-c_in // g[1])
    ks = k[0] * k[1] * k[2]
    scale = np.exp(rng.uniform(np.log(lo), 0.0, size=(p_groups, q_groups, ks)))
    full = np.repeat(np.repeat(scale, g[0], axis=0)[:c_out], g[1], axis=1)[:, :c_in]
    return w * full.reshape(c_out, c_in, *k)


@dataclasses.dataclass
class LayerData:
    layer: ConvLayer
    w: np.ndarray                  # float64 [M][N][kt][kh][kw] (round with to_dtype)
    bias: np.ndarray               # float64 [M] (bias stays fp32 on the GPU)
    mask: Optional[np.ndarray]     # uint8 [P][Q][K_s] or None (dense layer)


def layer_params(tag: str, layer: ConvLayer, mask_kind: str = "kgs", rate: float = 3.0,
                 w_std: Optional[float] = None, b_std: float = 0.01) -> LayerData:
    """Weights, bias and mask of one layer.  ``mask_kind`` is "kgs" (uses
    layer.keep per group), "vanilla" (whole groups at ``rate``) or "dense"."""
    wr = rng_for(tag, layer.name, "w")
    if w_std is None:
        w = kaiming(wr, layer.c_out, layer.c_in, layer.k)
    else:
        w = wr.normal(0.0, w_std, size=(layer.c_out, layer.c_in, *layer.k))
    b = rng_for(tag, layer.name, "b").normal(0.0, b_std, size=layer.c_out)
    p_groups, q_groups = layer.groups
    if layer.dense or mask_kind == "dense":
        mask = None
    elif mask_kind == "vanilla":
        mask = vanilla_mask(rng_for(tag, layer.name, "mask"), p_groups, q_groups, layer.ks, rate)
    elif layer.group_rate is not None:
        # one kernel position: keeping or pruning it is keeping or pruning the group
        mask = vanilla_mask(rng_for(tag, layer.name, "mask"), p_groups, q_groups, layer.ks,
                            layer.group_rate)
    else:
        mask = kgs_mask(rng_for(tag, layer.name, "mask"), p_groups, q_groups, layer.ks, layer.keep)
    return LayerData(layer, w, b, mask)


def clip_input(tag: str, batch: int = 1, kind: str = "uniform01",
               c: int = 3, t: int = 16, h: int = 112, w: int = 112) -> np.ndarray:
    """Input volume [n][c][t][h][w], float64: U(0,1) RGB-like clips
    ("uniform01"), U(-1,1) ("uniform11") or |N(0,1)| post-ReLU-like
    activations ("halfnormal")."""
    r = rng_for(tag, "x", batch, c, t, h, w)
    shape = (batch, c, t, h, w)
    if kind == "uniform01":
        return r.random(shape)
    if kind == "uniform11":
        return r.uniform(-1.0, 1.0, shape)
    if kind == "halfnormal":
        return np.abs(r.standard_normal(shape))
    raise ValueError(kind)


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------

def single_layer_small() -> Tuple[ConvLayer, dict]:
    """KGS layer 16->32 on 8x28x28, 3x3x3 s1 p1, 9 of 27 positions kept per
    group, W ~ N(0, 0.05^2), b ~ N(0, 0.01^2), x ~ U(-1, 1), ReLU, fp32."""
    l = ConvLayer("small", 16, 32, 8, 28, 28, (3, 3, 3), (1, 1, 1), (1, 1, 1), keep=9)
    return l, dict(tag="small16x32", w_std=0.05, x_kind="uniform11", dtype="f32")


def single_layer_conv3b() -> Tuple[ConvLayer, dict]:
    """C3D conv3b-shaped KGS layer 256->256 on 8x28x28, 10 of 27 kept
    (about 2.7x), Kaiming-normal weights, |N(0,1)| inputs, ReLU."""
    l = ConvLayer("conv3b", 256, 256, 8, 28, 28, (3, 3, 3), (1, 1, 1), (1, 1, 1), keep=10)
    return l, dict(tag="conv3b256", w_std=None, x_kind="halfnormal")


def c3d_stack(rate: float = 3.0, tag: str = "c3d", g: Tuple[int, int] = (GROUP, GROUP)
              ) -> List[ConvLayer]:
    """C3D stack with per-layer keep counts for a whole-stack rate (conv1
    dense), kernel groups of g = (g_M, g_N)."""
    layers = c3d_layers()
    for l, k in zip(layers, stack_keep_counts(layers, rate, tag)):
        l.keep = k
        l.g = tuple(g)
    return layers


def r2plus1d_stack(tag: str = "r2plus1d", g: Tuple[int, int] = (GROUP, GROUP)) -> List[ConvLayer]:
    """R(2+1)D-18 stack: spatial KGS convs keep 3 or 4 of 9 positions,
    temporal ones 1 or 2 of 3, drawn per layer; stem and shortcuts dense."""
    layers = r2plus1d_layers()
    r = rng_for(tag, "keep")
    for l in layers:
        l.g = tuple(g)
        if l.dense:
            continue
        l.keep = int(r.integers(3, 5)) if l.ks == 9 else int(r.integers(1, 3))
    return layers
