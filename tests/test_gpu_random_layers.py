"""GPU parity on layers drawn at random (fixed seed, so the list is the same
on every run): channel counts that are not multiples of the group or tile
sizes, group sizes 4x4 to 16x8, kernel extents, strides, batch 1-2, fused
pools and residuals, bf16 / fp16 / fp32, and every 16-bit KGS mapping.  Each
layer is compared in full with the oracle: relative L2 within the bar and
every output within its own bound."""
import numpy as np
import pytest

from harness import LayerCase
from paper_2007_09835_amd import build, synth
from test_gpu_parity import check_full

pytestmark = pytest.mark.gpu

TUNES16 = ["", "kgs_map=0,kgs_mfw=2", "kgs_map=0,kgs_mfw=4", "kgs_map=1", "kgs_map=1,pair_mfw=2",
           "kgs_map=1,pair_mfw=4", "kgs_map=2", "slots=128"]


def _cases(count=24, seed=20070983):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        dtype = ["bf16", "f16", "f32"][i % 3]
        g = [(4, 4), (8, 4), (16, 4), (4, 8), (16, 8)][rng.integers(5)]
        c_in = int(rng.integers(5, 97))
        c_out = int(rng.integers(1, 97))
        k = [(3, 3, 3), (1, 3, 3), (3, 1, 1), (1, 1, 1)][rng.integers(4)]
        stride = (1, 1, 1) if rng.random() < 0.6 else [(2, 2, 2), (1, 2, 2)][rng.integers(2)]
        pad = tuple(kk // 2 for kk in k)
        thw = (int(rng.integers(max(k[0], 2), 7)), int(rng.integers(4, 13)), int(rng.integers(4, 13)))
        keep = int(rng.integers(0, k[0] * k[1] * k[2] + 1))
        n = int(rng.integers(1, 3))
        pool = (1, 1, 1)
        if stride == (1, 1, 1) and rng.random() < 0.4:
            pool = [(1, 2, 2), (2, 2, 2)][rng.integers(2)]
        residual = pool == (1, 1, 1) and rng.random() < 0.3
        tune = "" if dtype == "f32" else TUNES16[rng.integers(len(TUNES16))]
        out.append((f"r{i}", n, c_in, c_out, thw, k, stride, pad, g, keep, dtype, pool, residual, tune))
    return out


CASES = _cases()


@pytest.fixture(scope="module", autouse=True)
def built():
    build.build(force=False)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_random_layer(ci, monkeypatch):
    tag, n, c_in, c_out, thw, k, stride, pad, g, keep, dtype, pool, residual, tune = CASES[ci]
    if tune:
        monkeypatch.setenv("RT3D_TUNE", tune)
    P, Q = -(-c_out // g[0]), -(-c_in // g[1])
    mask = synth.kgs_mask(synth.rng_for(tag, "mask"), P, Q, k[0] * k[1] * k[2], keep)
    case = LayerCase(tag, n, c_in, c_out, thw, k, stride, pad, dtype, mask, g=g, residual=residual,
                     pool=pool)
    check_full(case, f"random {CASES[ci]}")
