"""Shared helpers for the GPU parity tests: seeded inputs in the layer dtype,
the same values as float64 for the oracle, and relative-L2 comparison."""
import numpy as np
import torch

import oracle
from paper_2007_09835_amd import layers, synth

TOL = {"f32": 1e-4, "bf16": 1e-2, "f16": 1e-2}

# Spacing of the dtype's numbers in [1, 2) and below its smallest normal.
_EPS = {"f32": 2.0 ** -23, "bf16": 2.0 ** -7, "f16": 2.0 ** -10}
_MIN_ULP = {"f32": 2.0 ** -149, "bf16": 2.0 ** -133, "f16": 2.0 ** -24}


def ulp(x, dtype):
    """Spacing of the dtype's representable numbers at |x|."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, np.finfo(np.float64).tiny)))
    return np.maximum(np.exp2(e) * _EPS[dtype], _MIN_ULP[dtype])


def error_bound(ref, absref, kept_terms, dtype):
    """Per-output bound on |y_gpu - y_ref|: one unit in the last place of the
    output dtype at ref (the final round to nearest, also across a binade)
    plus K * 2^-23 * sum |w x| (float32 accumulation of K products in any
    order: |error| <= K u sum |terms| with u = 2^-24, taken twice).  absref
    is sum |w||x| + |bias| (+ |residual|) at that output; ReLU and max-pool
    are 1-Lipschitz, so the bound carries through them."""
    return ulp(ref, dtype) + np.asarray(kept_terms, dtype=np.float64) * 2.0 ** -23 * absref


def assert_within_bound(got, ref, bound, label):
    err = np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))
    ratio = err / bound
    worst = int(np.argmax(ratio))
    print(f"{label}: worst |err|/bound = {ratio.flat[worst]:.3f} (err {err.flat[worst]:.3e}, "
          f"bound {np.asarray(bound).flat[worst]:.3e}, ref {np.asarray(ref).flat[worst]:.4e})",
          flush=True)
    assert np.all(err <= bound), (label, float(ratio.flat[worst]), worst)


def kept_terms_per_filter(mask, g, c_in, ks, c_out):
    """Products summed into each filter's outputs: c_in * K_s when dense,
    else the kept (channel, position) pairs of its kernel groups."""
    if mask is None:
        return np.full(c_out, c_in * ks, dtype=np.int64)
    gm, gn = g
    widths = np.array([min(gn, c_in - q * gn) for q in range(mask.shape[1])], dtype=np.int64)
    per_group_row = (mask.astype(np.int64).sum(axis=2) * widths[None, :]).sum(axis=1)   # [P]
    return per_group_row[np.arange(c_out) // gm]


def window_indices(idx, pooled_shape, pool, full_shape):
    """Flat indices (into the unpooled [n][c][to][ho][wo] output) of the
    max-pool window of every flat pooled index: [len(idx), window]."""
    n, c, pt, ph, pw = pooled_shape
    _, _, to, ho, wo = full_shape
    qt, qh, qw = pool
    i = np.asarray(idx, dtype=np.int64)
    w_ = i % pw
    h_ = (i // pw) % ph
    t_ = (i // (pw * ph)) % pt
    nc = i // (pw * ph * pt)
    cols = []
    for dt in range(qt):
        for dh in range(qh):
            for dw in range(qw):
                cols.append(((nc * to + t_ * qt + dt) * ho + h_ * qh + dh) * wo + w_ * qw + dw)
    return np.stack(cols, axis=1)


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

    def _abs_terms(self):
        b = None if self.b_oracle is None else np.abs(self.b_oracle)
        r = None if self.res64 is None else np.abs(self.res64)
        return np.abs(self.x64), np.abs(self.w64), b, r

    def bound_full(self, ref):
        """Per-output error bound of the full (pooled) output."""
        ax, aw, ab, ar = self._abs_terms()
        if self.mask is None:
            s = oracle.conv3d_dense(ax, aw, ab, ar, self.stride, self.pad, False)
        else:
            s = oracle.conv3d_kgs(ax, aw, self.mask, *self.g, ab, ar, self.stride, self.pad, False)
        c_out, c_in = self.w64.shape[:2]
        ks = int(np.prod(self.k))
        kt = kept_terms_per_filter(self.mask, self.g, c_in, ks, c_out)[None, :, None, None, None]
        if self.pool != (1, 1, 1):
            # bound of the max = max of the window's bounds (ulp taken at the
            # unpooled reference values)
            ref_full = self.oracle_full_unpooled()
            per = error_bound(ref_full, s, kt, self.dtype)
            return oracle.maxpool3d(per, self.pool, self.pool)
        return error_bound(ref, s, kt, self.dtype)

    def bound_points(self, idx, ref):
        ax, aw, ab, ar = self._abs_terms()
        s = oracle.conv3d_points(ax, aw, idx, self.mask, *self.g, ab, ar, self.stride, self.pad,
                                 False)
        n, c_out = self.x64.shape[0], self.w64.shape[0]
        to, ho, wo = oracle.out_shape(*self.x64.shape[2:], self.k, self.stride, self.pad)
        m = (np.asarray(idx) // (to * ho * wo)) % c_out
        ks = int(np.prod(self.k))
        kt = kept_terms_per_filter(self.mask, self.g, self.w64.shape[1], ks, c_out)[m]
        return error_bound(ref, s, kt, self.dtype)

    def oracle_full_unpooled(self):
        if self.mask is None:
            return oracle.conv3d_dense(self.x64, self.w64, self.b_oracle, self.res64, self.stride,
                                       self.pad, self.relu)
        return oracle.conv3d_kgs(self.x64, self.w64, self.mask, *self.g, self.b_oracle,
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
