"""Shared helpers for the GPU parity tests: seeded inputs in the layer dtype,
the same values as float64 for the oracle, and relative-L2 comparison."""
import numpy as np
import torch

import oracle
from paper_2007_09835_amd import layers, synth

TOL = {"f32": 1e-4, "bf16": 1e-2, "f16": 1e-2}


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


def rounded(a64, dtype):
    """(tensor in dtype, float64 numpy of exactly those values)."""
    t = synth.to_dtype(a64, dtype)
    return t, t.to(torch.float64).numpy()


def to_device_ndhwc(t_ncdhw, device="cuda"):
    return t_ncdhw.permute(0, 2, 3, 4, 1).contiguous().to(device)


def from_device_ndhwc(y):
    return y.permute(0, 4, 1, 2, 3).to(torch.float64).cpu().numpy()


class LayerCase:
    """A conv layer with seeded tensors, ready to run on the GPU and in the
    oracle.  x64 / w64 / res64 are the float64 images of the dtype values."""

    def __init__(self, tag, n, c_in, c_out, thw, k, stride, pad, dtype, mask=None, relu=True,
                 residual=False, w_std=None, x_kind="halfnormal", g=(4, 4), bias=True,
                 pool=(1, 1, 1)):
        self.dtype, self.mask, self.g, self.pool = dtype, mask, g, tuple(pool)
        self.k, self.stride, self.pad, self.relu = k, stride, pad, relu
        r = synth.rng_for(tag, "w")
        if w_std is None:
            w = synth.kaiming(r, c_out, c_in, k)
        else:
            w = r.normal(0.0, w_std, size=(c_out, c_in, *k))
        self.w_t, self.w64 = rounded(w, dtype)
        self.b64 = synth.rng_for(tag, "b").normal(0, 0.01, c_out) if bias else None
        x = synth.clip_input(tag, n, x_kind, c_in, *thw)
        self.x_t, self.x64 = rounded(x, dtype)
        to, ho, wo = oracle.out_shape(*thw, k, stride, pad)
        self.res_t = self.res64 = None
        if residual:
            res = synth.rng_for(tag, "res").standard_normal((n, c_out, to, ho, wo))
            self.res_t, self.res64 = rounded(res, dtype)
        self.conv = layers.Conv3d(c_in, c_out, thw, k, stride, pad, self.w_t,
                                  None if self.b64 is None else self.b64.astype(np.float32),
                                  mask, dtype, relu=relu, residual=residual, g=g, batch=n,
                                  pool=pool)
        # The kernel adds a float32 bias: the oracle sees the same float32 values.
        self.b_oracle = None if self.b64 is None else self.b64.astype(np.float32).astype(np.float64)

    def run_gpu(self):
        x = to_device_ndhwc(self.x_t)
        res = None if self.res_t is None else to_device_ndhwc(self.res_t)
        y = self.conv(x, res)
        torch.cuda.synchronize()
        return from_device_ndhwc(y)

    def oracle_full(self):
        if self.mask is None:
            y = oracle.conv3d_dense(self.x64, self.w64, self.b_oracle, self.res64, self.stride,
                                    self.pad, self.relu)
        else:
            y = oracle.conv3d_kgs(self.x64, self.w64, self.mask, *self.g, self.b_oracle,
                                  self.res64, self.stride, self.pad, self.relu)
        if self.pool != (1, 1, 1):
            y = oracle.maxpool3d(y, self.pool, self.pool)
        return y

    def oracle_points(self, idx):
        return oracle.conv3d_points(self.x64, self.w64, idx, self.mask, *self.g, self.b_oracle,
                                    self.res64, self.stride, self.pad, self.relu)


def sample_indices(shape, count, seed=0):
    """Random flat output indices plus every corner voxel of every 37th filter
    (borders exercise padding and ragged bricks)."""
    n, c, to, ho, wo = shape
    rng = np.random.default_rng(seed)
    total = n * c * to * ho * wo
    idx = set(rng.choice(total, size=min(count, total), replace=False).tolist())
    for b in range(n):
        for m in range(0, c, 37):
            for t in (0, to - 1):
                for h in (0, ho - 1):
                    for w in (0, wo - 1):
                        idx.add((((b * c + m) * to + t) * ho + h) * wo + w)
    return np.array(sorted(idx), dtype=np.int64)
