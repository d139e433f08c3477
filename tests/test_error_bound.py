"""The per-output error bound the GPU parity tests apply (harness.error_bound),
checked on the CPU against what it must accept and what it must reject.

* Accept: the layer computed the way the kernels compute it -- float32
  products and sums (torch conv3d on the CPU in float32 over the masked
  weights), then rounded to the 16-bit output dtype -- stays within the
  bound at every output, in bf16 and fp16, with and without a fused pool.
* Reject: the same computation with one (4-channel block, kernel position)
  item of one kernel group dropped, the mistake a wrong item list or pair
  plan would make, breaks the bound somewhere; so does a sign flip of one
  output (the relative-L2 bar alone lets both pass on large layers).
"""
import numpy as np
import pytest
import torch

import oracle
from harness import error_bound, kept_terms_per_filter, rel_l2, ulp
from paper_2007_09835_amd import synth

TORCH = {"bf16": torch.bfloat16, "f16": torch.float16}


def _case(dt, seed=3, c_in=64, c_out=32, thw=(4, 9, 9), keep=9):
    rng = np.random.default_rng(seed)
    w = synth.kaiming(rng, c_out, c_in, (3, 3, 3))
    w = torch.from_numpy(w).to(TORCH[dt]).double().numpy()
    x = np.abs(rng.standard_normal((1, c_in, *thw)))
    x = torch.from_numpy(x).to(TORCH[dt]).double().numpy()
    b = rng.normal(0, 0.01, c_out).astype(np.float32).astype(np.float64)
    mask = synth.kgs_mask(rng, c_out // 4, c_in // 4, 27, keep)
    return w, x, b, mask


def _float32_layer(x, w, b, mask, dt, pool=None):
    """The layer as the kernels compute it: float32 arithmetic, one rounding
    to the output dtype at the end (after ReLU and the max)."""
    full = np.repeat(np.repeat(mask, 4, 0), 4, 1).reshape(w.shape)
    wm = torch.from_numpy(np.where(full == 1, w, 0.0)).float()
    y = torch.nn.functional.conv3d(torch.from_numpy(x).float(), wm, torch.from_numpy(b).float(),
                                   padding=1)
    y = torch.relu(y)
    if pool:
        y = torch.nn.functional.max_pool3d(y, pool, pool)
    return y.to(TORCH[dt]).double().numpy()


def _bound(x, w, b, mask, dt, ref_unpooled, pool=None):
    s = oracle.conv3d_kgs(np.abs(x), np.abs(w), mask, 4, 4, np.abs(b), None, (1, 1, 1),
                          (1, 1, 1), False)
    kt = kept_terms_per_filter(mask, (4, 4), x.shape[1], 27, w.shape[0])[None, :, None, None, None]
    per = error_bound(ref_unpooled, s, kt, dt)
    return oracle.maxpool3d(per, pool, pool) if pool else per


@pytest.mark.parametrize("pool", [None, (2, 2, 2)])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_bound_accepts_float32_accumulation(dt, pool):
    w, x, b, mask = _case(dt)
    ref_full = oracle.conv3d_kgs(x, w, mask, 4, 4, b, None, (1, 1, 1), (1, 1, 1), True)
    ref = oracle.maxpool3d(ref_full, pool, pool) if pool else ref_full
    got = _float32_layer(x, w, b, mask, dt, pool)
    bound = _bound(x, w, b, mask, dt, ref_full, pool)
    assert np.all(np.abs(got - ref) <= bound)
    # and the bound is not vacuous: a few units in the last place where the
    # output is nonzero
    nz = ref != 0
    assert np.median(bound[nz] / ulp(ref[nz], dt)) < 4.0


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_bound_rejects_a_dropped_item(dt):
    # conv3b-like reduction depth (256 channels x 27 positions) and width,
    # small volume
    w, x, b, mask = _case(dt, seed=5, c_in=256, c_out=256, thw=(2, 5, 5))
    ref = oracle.conv3d_kgs(x, w, mask, 4, 4, b, None, (1, 1, 1), (1, 1, 1), True)
    bound = _bound(x, w, b, mask, dt, ref)
    caught = 0
    rng = np.random.default_rng(11)
    for _ in range(6):
        p, q = rng.integers(mask.shape[0]), rng.integers(mask.shape[1])
        pos = int(rng.choice(np.flatnonzero(mask[p, q])))
        bad = mask.copy()
        bad[p, q, pos] = 0
        got = _float32_layer(x, w, b, bad, dt)
        # the relative-L2 bar of the parity tests would let this through
        assert rel_l2(got, ref) < 1e-2
        caught += int(np.any(np.abs(got - ref) > bound))
    assert caught == 6


def test_bound_rejects_a_sign_flip():
    w, x, b, mask = _case("bf16", seed=8, c_in=128, c_out=64, thw=(4, 12, 12))
    ref = oracle.conv3d_kgs(x, w, mask, 4, 4, b, None, (1, 1, 1), (1, 1, 1), False)
    got = _float32_layer(x, w, b, mask, "bf16")
    got_lin = torch.from_numpy(ref).to(torch.bfloat16).double().numpy()
    bound = _bound(x, w, b, mask, "bf16", ref)
    assert np.all(np.abs(got_lin - ref) <= bound)
    mag = np.abs(ref).ravel()
    i = int(np.argsort(mag)[len(mag) // 2])   # an output of median magnitude
    got_lin.flat[i] = -got_lin.flat[i]
    assert rel_l2(got_lin, ref) < 1e-2
    assert np.any(np.abs(got_lin - ref) > bound)
    del got
