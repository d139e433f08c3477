"""GPU parity: the HIP kernels through the C ABI against the CPU oracle.

Bars: fp32 relative L2 <= 1e-4, bf16 / fp16 <= 1e-2 (float32 accumulation
in the kernels, float64 in the oracle, outputs rounded to the layer dtype).
Small layers are compared element by element in full; full-size workload
layers are compared on sampled outputs that the oracle computes one by one.
Invariants that need no oracle (all-zero mask, vanilla-pruned groups,
determinism) are checked bit-exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from harness import (TOL, LayerCase, assert_within_bound, error_bound, from_device_ndhwc,
                     kept_terms_per_filter, rel_l2, rounded, sample_indices, to_device_ndhwc)
from paper_2007_09835_amd import build, layers, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def built():
    build.build(force=False)


def masked(tag, c_out, c_in, k, keep, g=(4, 4)):
    P, Q = -(-c_out // g[0]), -(-c_in // g[1])
    return synth.kgs_mask(synth.rng_for(tag, "mask"), P, Q, k[0] * k[1] * k[2], keep)


def check_full(case, label):
    """relL2 against the bar, and every output within its own bound
    (harness.error_bound: rounding + float32 accumulation)."""
    got = case.run_gpu()
    ref = case.oracle_full()
    err = rel_l2(got, ref)
    print(f"{label}: relL2={err:.3e} maxabs={np.abs(got - ref).max():.3e}", flush=True)
    assert got.shape == ref.shape
    assert err <= TOL[case.dtype], (label, err)
    assert_within_bound(got, ref, case.bound_full(ref), label)
    return got, ref


def check_sampled(case, label, count=3000):
    got = case.run_gpu()
    assert case.pool == (1, 1, 1)
    idx = sample_indices(got.shape, count)
    ref = case.oracle_points(idx)
    err = rel_l2(got.ravel()[idx], ref)
    print(f"{label}: sampled relL2={err:.3e} ({len(idx)} outputs)", flush=True)
    assert err <= TOL[case.dtype], (label, err)
    assert_within_bound(got.ravel()[idx], ref, case.bound_points(idx, ref), label)
    return got


# ---------------------------------------------------------------------------
# Small layers, full comparison
# ---------------------------------------------------------------------------

def test_small_config_fp32():
    """16->32 on 8x28x28, 3x3x3 s1 p1, 9 of 27 positions per 4x4 group, fp32."""
    layer, cfg = synth.single_layer_small()
    mask = masked(cfg["tag"], 32, 16, (3, 3, 3), 9)
    case = LayerCase(cfg["tag"], 1, 16, 32, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1), "f32",
                     mask, w_std=0.05, x_kind="uniform11")
    check_full(case, "small16x32 f32")


SHAPES = [
    # tag, n, c_in, c_out, thw, k, stride, pad, keep
    ("s1", 1, 16, 32, (4, 6, 9), (3, 3, 3), (1, 1, 1), (1, 1, 1), 9),
    ("s2", 2, 24, 20, (5, 7, 6), (3, 3, 3), (2, 2, 2), (1, 1, 1), 12),
    ("s3", 1, 10, 13, (3, 9, 11), (3, 3, 3), (1, 1, 1), (1, 1, 1), 7),     # partial groups
    ("s4", 1, 32, 48, (4, 10, 10), (1, 3, 3), (1, 2, 2), (0, 1, 1), 4),
    ("s5", 1, 40, 36, (6, 5, 5), (3, 1, 1), (2, 1, 1), (1, 0, 0), 2),
    ("s6", 1, 3, 16, (2, 20, 20), (1, 7, 7), (1, 2, 2), (0, 3, 3), 20),
    ("s7", 1, 64, 64, (2, 9, 9), (1, 1, 1), (2, 2, 2), (0, 0, 0), 1),
    ("s8", 1, 45, 23, (3, 6, 7), (3, 3, 3), (1, 1, 1), (1, 1, 1), 27),     # c_in, c_out % 4 != 0
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_kgs_small_shapes(si, dtype):
    tag, n, c_in, c_out, thw, k, stride, pad, keep = SHAPES[si]
    mask = masked(tag, c_out, c_in, k, min(keep, k[0] * k[1] * k[2]))
    case = LayerCase(tag, n, c_in, c_out, thw, k, stride, pad, dtype, mask)
    check_full(case, f"kgs {tag} {dtype}")


@pytest.mark.parametrize("tune", ["kgs_f32=0", "kgs_f32=1"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_f32_kgs_both_mappings(si, tune, monkeypatch):
    """fp32 KGS on the exact 4x4x1 kernel (kgs_f32=0) and on the 16x16x4
    kernel over the tile's union of kept items (kgs_f32=1), forced; the
    planner picks the union only for layers too small to be MFMA-bound."""
    monkeypatch.setenv("RT3D_TUNE", tune)
    tag, n, c_in, c_out, thw, k, stride, pad, keep = SHAPES[si]
    mask = masked(tag, c_out, c_in, k, min(keep, k[0] * k[1] * k[2]))
    case = LayerCase(tag + "f" + tune[-1], n, c_in, c_out, thw, k, stride, pad, "f32", mask)
    assert case.conv.info.variant == (9 if tune.endswith("1") else 4)
    check_full(case, f"kgs f32 {tag} {tune}")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_dense_small_shapes(si, dtype):
    tag, n, c_in, c_out, thw, k, stride, pad, _ = SHAPES[si]
    case = LayerCase(tag + "d", n, c_in, c_out, thw, k, stride, pad, dtype, None)
    check_full(case, f"dense {tag} {dtype}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("slots", ["64", "128"])
@pytest.mark.parametrize("sparse", [True, False])
@pytest.mark.parametrize("si", [0, 1, 2, 7])
def test_both_brick_widths(si, sparse, slots, dtype, monkeypatch):
    """The item kernels with 64- and 128-slot bricks (16-bit: 4 or 8 voxel
    fragments per wave; exact fp32 KGS: one or two slots per lane) on the
    same layers."""
    monkeypatch.setenv("RT3D_TUNE", "slots=" + slots)
    tag, n, c_in, c_out, thw, k, stride, pad, keep = SHAPES[si]
    mask = masked(tag, c_out, c_in, k, min(keep, k[0] * k[1] * k[2])) if sparse else None
    case = LayerCase(tag + "w" + slots, n, c_in, c_out, thw, k, stride, pad, dtype, mask)
    check_full(case, f"{'kgs' if sparse else 'dense'} {tag} {dtype} slots={slots}")


# First-layer shapes (c_in <= 4, w * c_in % 4 == 0) run on the
# small-input-channel kernel: wave-private bricks of 1x2x32 voxels, weights in
# registers, halo lines staged by one 8-byte buffer load per lane (words
# before the input's first byte read as zero), optional 1x2x2 pooling in
# registers.  Widths leave a ragged last brick.
SMALL_CIN = [
    # tag, n, c_in, c_out, thw, k, pad, pool, dtype, sparse, residual
    ("c1", 1, 3, 64, (4, 10, 72), (3, 3, 3), (1, 1, 1), (1, 2, 2), "bf16", False, False),
    ("c2", 2, 3, 40, (3, 7, 44), (3, 3, 3), (1, 1, 1), (1, 1, 1), "f16", True, False),
    ("c3", 1, 4, 20, (2, 6, 33), (1, 3, 3), (0, 1, 1), (1, 1, 1), "bf16", False, True),
    ("c4", 1, 1, 16, (5, 5, 12), (3, 3, 3), (0, 1, 1), (1, 2, 2), "bf16", True, False),
    ("c5", 3, 2, 64, (3, 9, 40), (3, 1, 3), (1, 0, 1), (1, 2, 2), "f16", False, True),
    # 1x7x7 stride (1,2,2) stems (S3D 3->64, R(2+1)D 3->45: 8 K-steps) and a 5x5 tap window
    ("c6", 1, 3, 64, (3, 13, 76), (1, 7, 7), (0, 3, 3), (1, 1, 1), "bf16", False, False),
    ("c7", 2, 3, 45, (2, 9, 68), (1, 7, 7), (0, 3, 3), (1, 1, 1), "f16", True, False),
    ("c8", 1, 2, 20, (2, 8, 40), (1, 5, 5), (0, 2, 2), (1, 2, 2), "bf16", False, True),
    # w * c_in % 4 != 0: halo lines would start at different offsets within
    # their 8-byte words, so these run on the item kernel
    ("c9", 1, 3, 32, (3, 6, 45), (3, 3, 3), (1, 1, 1), (1, 2, 2), "bf16", True, False),
    ("c10", 2, 1, 16, (2, 5, 9), (1, 3, 3), (0, 1, 1), (1, 1, 1), "f16", False, False),
]
SMALL_CIN_STRIDE = {"c6": (1, 2, 2), "c7": (1, 2, 2)}


@pytest.mark.parametrize("ci", range(len(SMALL_CIN)))
def test_small_input_channel_layers(ci):
    tag, n, c_in, c_out, thw, k, pad, pool, dtype, sparse, residual = SMALL_CIN[ci]
    mask = masked(tag, c_out, c_in, k, max(1, (k[0] * k[1] * k[2]) // 3)) if sparse else None
    case = LayerCase(tag, n, c_in, c_out, thw, k, SMALL_CIN_STRIDE.get(tag, (1, 1, 1)), pad, dtype,
                     mask, residual=residual, pool=pool)
    small = thw[2] * c_in % 4 == 0
    assert (case.conv.info.variant in (5, 6)) == small, case.conv.info.variant
    check_full(case, f"small c_in {tag} {dtype} {'kgs' if sparse else 'dense'}")


# Kernel groups wider than 4x4 (g_M, g_N in {4, 8, 16}): the planner expands
# each group mask to its 4x4 blocks, so a 16-filter tile of a g_M = 16 layer
# walks exactly its group's kept items.
GROUPED = [
    # tag, n, c_in, c_out, thw, k, stride, pad, g, keep
    ("g1", 1, 32, 48, (4, 7, 9), (3, 3, 3), (1, 1, 1), (1, 1, 1), (16, 4), 9),
    ("g2", 2, 24, 40, (3, 8, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), (8, 4), 10),
    ("g3", 1, 36, 33, (4, 6, 6), (1, 3, 3), (1, 2, 2), (0, 1, 1), (16, 8), 4),   # partial groups
    ("g4", 1, 20, 16, (5, 5, 5), (3, 1, 1), (1, 1, 1), (1, 0, 0), (4, 8), 2),
    ("g5", 1, 64, 64, (3, 6, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), (16, 16), 8),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("gi", range(len(GROUPED)))
def test_kgs_group_sizes(gi, dtype):
    tag, n, c_in, c_out, thw, k, stride, pad, g, keep = GROUPED[gi]
    mask = masked(tag, c_out, c_in, k, keep, g)
    case = LayerCase(tag, n, c_in, c_out, thw, k, stride, pad, dtype, mask, g=g)
    check_full(case, f"kgs {tag} g={g} {dtype}")


def test_conv3b_shape_with_16x4_groups():
    """C3D conv3b-shaped layer with g = 16x4 (MFMA-width groups) at full size,
    sampled outputs."""
    mask = masked("g16conv3b", 256, 256, (3, 3, 3), 9, (16, 4))
    case = LayerCase("g16conv3b", 1, 256, 256, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1),
                     "bf16", mask, x_kind="halfnormal", g=(16, 4))
    check_sampled(case, "conv3b g=16x4 bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_residual_epilogue(dtype):
    mask = masked("res", 24, 16, (3, 1, 1), 2)
    case = LayerCase("res", 2, 16, 24, (6, 7, 7), (3, 1, 1), (1, 1, 1), (1, 0, 0), dtype, mask,
                     residual=True)
    check_full(case, f"kgs residual {dtype}")
    dcase = LayerCase("resd", 2, 16, 24, (6, 7, 7), (3, 1, 1), (1, 1, 1), (1, 0, 0), dtype, None,
                      residual=True)
    check_full(dcase, f"dense residual {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_all_zero_mask_gives_relu_bias_exactly(dtype):
    mask = np.zeros((8, 4, 27), dtype=np.uint8)
    case = LayerCase("zero", 1, 16, 32, (4, 6, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype, mask)
    got = case.run_gpu()
    b = np.maximum(case.b_oracle, 0.0)
    expect = torch.from_numpy(b).to(layers.TORCH_DTYPES[dtype]).to(torch.float64).numpy()
    assert np.array_equal(got, np.broadcast_to(expect[None, :, None, None, None], got.shape))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_one_mask_matches_dense_kernel(dtype):
    mask = np.ones((8, 8, 27), dtype=np.uint8)
    case = LayerCase("ones", 1, 32, 32, (4, 8, 8), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype, mask)
    got, ref = check_full(case, f"all-ones {dtype}")
    dense = layers.Conv3d(32, 32, (4, 8, 8), (3, 3, 3), (1, 1, 1), (1, 1, 1), case.w_t,
                          case.b64.astype(np.float32), None, dtype)
    yd = from_device_ndhwc(dense(to_device_ndhwc(case.x_t)))
    assert rel_l2(got, yd) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_vanilla_pruned_group_ignores_its_channels(dtype):
    """Section 3: a vanilla-pruned group (p, q) removes every link from
    channel block q to filter block p: perturbing those channels leaves the
    block's outputs bit-identical."""
    c_in, c_out = 32, 32
    rng = synth.rng_for("vanilla-test", "mask")
    mask = synth.vanilla_mask(rng, 8, 8, 27, 3.0)
    p, q = [(p, q) for p in range(8) for q in range(8) if mask[p, q, 0] == 0][0]
    case = LayerCase("vanilla", 1, c_in, c_out, (4, 8, 8), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype,
                     mask)
    y1 = case.run_gpu()
    x2 = case.x_t.clone()
    x2[:, 4 * q:4 * q + 4] += 1.0
    y2 = from_device_ndhwc(case.conv(to_device_ndhwc(x2)))
    assert np.array_equal(y1[:, 4 * p:4 * p + 4], y2[:, 4 * p:4 * p + 4])
    assert not np.array_equal(y1, y2)
    check_full(case, f"vanilla {dtype}")


@pytest.mark.parametrize("x_off", [0, 2])
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("sparse", [True, False])
def test_odd_channel_slice_of_a_wider_input(dtype, sparse, x_off):
    """A layer of 13 input channels reads channels x_off..x_off+12 of a
    16-channel input.  Offset 0: pitch and offset are multiples of 8, so the
    halo staging loads whole 16-byte pieces and cuts each row's last piece
    to the layer's channels; offset 2: it reads two channels per 4-byte load
    and masks the one past the slice.  The channels outside the slice hold
    NaN, so any of them reaching a product shows in the output."""
    mask = masked("oddslice", 24, 13, (3, 3, 3), 11) if sparse else None
    case = LayerCase("oddslice", 2, 13, 24, (4, 7, 9), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype, mask)
    x = to_device_ndhwc(case.x_t)
    wide = torch.full((*x.shape[:-1], 16), float("nan"), dtype=x.dtype, device=x.device)
    wide[..., x_off:x_off + 13] = x
    got = from_device_ndhwc(case.conv(wide, None, x_off=x_off))
    ref = case.oracle_full()
    assert np.isfinite(got).all()
    err = rel_l2(got, ref)
    print(f"odd slice {dtype} sparse={sparse}: relL2={err:.3e}", flush=True)
    assert err <= TOL[dtype], err
    assert_within_bound(got, ref, case.bound_full(ref), "odd slice")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("sparse", [True, False])
def test_split_k_matches_unsplit(dtype, sparse):
    """A small-voxel layer splits its channels across workgroups (fp32
    partials + ordered reduction); with no workspace it runs unsplit.  Both
    match the oracle, and the split result is reproducible bit for bit."""
    mask = masked("split", 128, 256, (3, 3, 3), 9) if sparse else None
    case = LayerCase("split", 1, 256, 128, (2, 7, 7), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype, mask,
                     residual=True)
    assert case.conv.workspace(1) is not None
    got, ref = check_full(case, f"split {'kgs' if sparse else 'dense'} {dtype}")
    x = to_device_ndhwc(case.x_t)
    r = to_device_ndhwc(case.res_t)
    again = from_device_ndhwc(case.conv(x, r))
    assert np.array_equal(got, again)
    unsplit = from_device_ndhwc(case.conv(x, r, use_workspace=False))
    assert rel_l2(unsplit, ref) <= TOL[dtype]


POOLED = [
    # tag, n, c_in, c_out, thw, pool, dtype, sparse, residual
    ("pa", 1, 16, 32, (4, 8, 12), (1, 2, 2), "bf16", True, False),
    ("pb", 2, 32, 48, (6, 9, 11), (2, 2, 2), "bf16", True, False),    # floor: odd extents
    ("pc", 1, 24, 16, (5, 7, 9), (2, 2, 2), "f32", True, True),
    ("pd", 1, 64, 64, (4, 8, 8), (2, 2, 2), "f16", False, False),
    ("pe", 1, 256, 128, (4, 6, 6), (2, 2, 2), "bf16", True, False),   # split-K + pooled reduce
    ("pf", 1, 256, 128, (4, 6, 6), (2, 2, 2), "f32", False, True),
    ("pg", 1, 3, 64, (2, 16, 16), (1, 2, 2), "bf16", False, False),   # conv1-like
    ("ph", 1, 128, 64, (3, 9, 9), (1, 3, 3), "bf16", True, False),    # 9-voxel window, split-K
    ("pi", 1, 96, 40, (6, 5, 5), (3, 1, 1), "f16", True, True),       # 3-voxel window, residual
]


@pytest.mark.parametrize("pi", range(len(POOLED)))
def test_fused_pool_epilogue(pi):
    """conv -> act -> max-pool fused in the epilogue equals the oracle's
    max-pool of its conv output (window = stride, floor extents)."""
    tag, n, c_in, c_out, thw, pool, dtype, sparse, residual = POOLED[pi]
    mask = masked(tag, c_out, c_in, (3, 3, 3), 9) if sparse else None
    case = LayerCase(tag, n, c_in, c_out, thw, (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype, mask,
                     residual=residual, pool=pool)
    check_full(case, f"pooled {tag} {dtype} {'kgs' if sparse else 'dense'}")


def test_blob_packed_for_another_batch_size():
    """The tile shapes are chosen for the batch size given at pack time (64-
    or 128-slot bricks, 16- or 64-filter KGS tiles); a blob packed for one
    batch size gives the same results at another."""
    def repack(case, c_in, c_out, thw, k, stride, pad, batch):
        case.conv = layers.Conv3d(c_in, c_out, thw, k, stride, pad, case.w_t,
                                  case.b64.astype(np.float32), case.mask, case.dtype,
                                  batch=batch)

    # packed for batch 1 (64-slot bricks), run at batch 3
    mask = masked("rb1", 48, 32, (3, 3, 3), 9)
    case = LayerCase("rb1", 3, 32, 48, (4, 10, 12), (3, 3, 3), (1, 1, 1), (1, 1, 1), "bf16", mask)
    repack(case, 32, 48, (4, 10, 12), (3, 3, 3), (1, 1, 1), (1, 1, 1), 1)
    check_full(case, "batch-1 blob at batch 3")
    # packed for batch 32 (64-filter KGS tiles on a wide layer), run at batch 1
    mask = masked("rb32", 256, 256, (3, 3, 3), 13)
    case = LayerCase("rb32", 1, 256, 256, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1), "bf16",
                     mask)
    repack(case, 256, 256, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1), 32)
    check_sampled(case, "batch-32 blob at batch 1", count=1500)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("sparse", [True, False])
@pytest.mark.parametrize("shape", [((4, 4, 32), 32, 48), ((4, 6, 34), 40, 36)])
def test_pooled_register_epilogue(shape, sparse, dtype):
    """2x2x2 pooling done on the accumulator registers (2x2x16 bricks of 64
    slots: the four w-rows of a brick and adjacent lanes form the windows),
    including a ragged second brick along w (34 = 16 + 16 + 2)."""
    thw, c_in, c_out = shape
    mask = masked("prp", c_out, c_in, (3, 3, 3), 9) if sparse else None
    case = LayerCase("prp%d" % c_in, 1, c_in, c_out, thw, (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype,
                     mask, pool=(2, 2, 2))
    plan = np.frombuffer(bytes(case.conv.info.plan), dtype=np.int32)
    assert tuple(plan[:3]) == (2, 2, 16) and plan[8] == 64, plan[:9]
    check_full(case, f"pooled registers {thw} {'kgs' if sparse else 'dense'} {dtype}")


def test_runs_are_deterministic():
    mask = masked("det", 64, 64, (3, 3, 3), 9)
    case = LayerCase("det", 1, 64, 64, (4, 14, 14), (3, 3, 3), (1, 1, 1), (1, 1, 1), "bf16", mask)
    assert np.array_equal(case.run_gpu(), case.run_gpu())


def test_empty_batch_is_a_no_op():
    mask = masked("empty", 16, 16, (3, 3, 3), 9)
    case = LayerCase("empty", 1, 16, 16, (4, 6, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), "bf16", mask)
    x = torch.empty((0, 4, 6, 6, 16), dtype=torch.bfloat16, device="cuda")
    y = case.conv(x)
    torch.cuda.synchronize()
    assert y.shape == (0, 4, 6, 6, 16)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("k,stride,pad", [((1, 2, 2), (1, 2, 2), (0, 0, 0)),
                                          ((2, 2, 2), (2, 2, 2), (0, 0, 0)),
                                          ((3, 3, 3), (2, 1, 2), (0, 0, 0)),
                                          ((3, 3, 3), (1, 1, 1), (1, 1, 1)),
                                          ((1, 3, 3), (1, 2, 2), (0, 1, 1)),
                                          ((3, 3, 3), (2, 2, 2), (1, 1, 1))])
def test_maxpool_exact(dtype, k, stride, pad):
    # shifted negative so that a padded zero would win if padding took part
    x64 = synth.clip_input("pool", 2, "halfnormal", 24, 6, 9, 10) - 3.0
    x_t, x_ref = rounded(x64, dtype)
    y = layers.maxpool3d(to_device_ndhwc(x_t), k, stride, dtype, pad=pad)
    ref = oracle.maxpool3d(x_ref, k, stride, pad)
    assert np.array_equal(from_device_ndhwc(y), ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_concatenation_writes_only_its_slice(dtype):
    """Three layers (dense 1x1x1, KGS 3x3x3, KGS 1x3x3) write channel slices
    of one wider output, as the branches of an Inception block do; each
    slice matches its oracle and the channels no layer owns keep their
    sentinel."""
    n, thw = 1, (4, 10, 12)
    specs = [("cat_a", 16, 12, (1, 1, 1), (0, 0, 0), None, 0),
             ("cat_b", 16, 20, (3, 3, 3), (1, 1, 1), 9, 16),
             ("cat_c", 16, 8, (1, 3, 3), (0, 1, 1), 4, 40)]
    c_total = 52  # channels 12..15 and 36..39 and 48..51 belong to nobody
    x64 = synth.clip_input("cat", n, "halfnormal", 16, *thw)
    x_t, x_ref = rounded(x64, dtype)
    x = to_device_ndhwc(x_t)
    y = torch.full((n, *thw, c_total), -7.0, dtype=layers.TORCH_DTYPES[dtype], device="cuda")
    refs = []
    for tag, c_in, c_out, k, pad, keep, off in specs:
        mask = None if keep is None else masked(tag, c_out, c_in, k, keep)
        case = LayerCase(tag, n, c_in, c_out, thw, k, (1, 1, 1), pad, dtype, mask)
        case.x_t, case.x64 = x_t, x_ref
        case.conv(x, out=y, c_off=off)
        ref = case.oracle_full()
        refs.append((off, c_out, ref, case.bound_full(ref)))
    torch.cuda.synchronize()
    got = from_device_ndhwc(y)
    owned = np.zeros(c_total, bool)
    for off, c_out, ref, bound in refs:
        assert rel_l2(got[:, off:off + c_out], ref) <= TOL[dtype]
        assert_within_bound(got[:, off:off + c_out], ref, bound, f"slice {off}")
        owned[off:off + c_out] = True
    assert np.all(got[:, ~owned] == -7.0)


# ---------------------------------------------------------------------------
# Full-size workload layers, sampled comparison
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_conv3b_config(dtype):
    """256->256 on 8x28x28, 10 of 27 kept per group, Kaiming weights,
    |N(0,1)| inputs."""
    layer, cfg = synth.single_layer_conv3b()
    mask = masked(cfg["tag"], 256, 256, (3, 3, 3), 10)
    case = LayerCase(cfg["tag"], 1, 256, 256, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype,
                     mask)
    check_sampled(case, f"conv3b {dtype}")
    dense = LayerCase(cfg["tag"] + "d", 1, 256, 256, (8, 28, 28), (3, 3, 3), (1, 1, 1), (1, 1, 1),
                      dtype, None)
    check_sampled(dense, f"conv3b dense {dtype}")


@pytest.mark.parametrize("li", range(8))
def test_c3d_stack_layers(li):
    """Each C3D layer at batch 1 with its own seeded input of the layer's
    shape (U(0,1) clip for conv1, |N(0,1)| activations after), whole-stack
    pruning rate 3x, bf16."""
    stack = synth.c3d_stack(3.0)
    l = stack[li]
    mask = None if l.dense else synth.kgs_mask(synth.rng_for("c3d", l.name, "mask"), *l.groups,
                                               l.ks, l.keep)
    case = LayerCase("c3d-" + l.name, 1, l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad,
                     "bf16", mask, x_kind="uniform01" if li == 0 else "halfnormal")
    check_sampled(case, f"c3d {l.name}")


R21 = synth.r2plus1d_stack()


@pytest.mark.parametrize("li", range(len(R21)))
def test_r2plus1d_layers(li):
    l = R21[li]
    mask = None if l.dense else synth.kgs_mask(synth.rng_for("r21d", l.name, "mask"), *l.groups,
                                               l.ks, l.keep)
    case = LayerCase("r21d-" + l.name, 1, l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad,
                     "bf16", mask, relu=l.relu, residual=l.residual_from is not None,
                     x_kind="uniform01" if li == 0 else "halfnormal")
    check_sampled(case, f"r21d {l.name}", count=1500)


@pytest.mark.parametrize("variant", ["kgs2", "kgs5", "vanilla3"])
@pytest.mark.parametrize("li", [1, 3, 7])
def test_c3d_batch32_layers(variant, li):
    """Batch-32 layers of the throughput sweep (KGS at 2x and 5x, vanilla at
    3x)."""
    rate = {"kgs2": 2.0, "kgs5": 5.0, "vanilla3": 3.0}[variant]
    stack = synth.c3d_stack(rate, tag="c3d-b32")
    l = stack[li]
    r = synth.rng_for("c3d-b32", variant, l.name, "mask")
    if variant.startswith("vanilla"):
        mask = synth.vanilla_mask(r, *l.groups, l.ks, rate)
    else:
        mask = synth.kgs_mask(r, *l.groups, l.ks, l.keep)
    case = LayerCase(f"b32-{variant}-{l.name}", 32, l.c_in, l.c_out, (l.t, l.h, l.w), l.k,
                     l.stride, l.pad, "bf16", mask)
    check_sampled(case, f"b32 {variant} {l.name}", count=2000)



# ---------------------------------------------------------------------------
# S3D-shaped stack: Inception blocks (fused concatenation), padded pools
# ---------------------------------------------------------------------------

def _s3d_oracle_op(op, stack, src64, layer_by_name, absolute=False):
    """float64 result of one op of the S3D stack on the float64 input src64
    ([n][c][t][h][w]); a conv returns its c_out channels.  absolute: the
    conv of |x|, |w| plus |bias| without activation (the error bound's sum)."""
    if op[0] == "pool":
        _, _, _, k, st, pd = op
        return oracle.maxpool3d(src64, k, st, pd)
    _, name, _, _, _, x_off = op
    i, l = layer_by_name[name]
    src64 = src64[:, x_off:x_off + l.c_in]
    d = synth.layer_params("s3d", l)
    w64 = synth.to_dtype(d.w, stack.dtype).double().numpy()
    b64 = d.bias.astype(np.float32).astype(np.float64)
    relu = l.relu
    if absolute:
        src64, w64, b64, relu = np.abs(src64), np.abs(w64), np.abs(b64), False
    mask = stack.masks[i]
    if mask is None:
        return oracle.conv3d_dense(src64, w64, b64, None, l.stride, l.pad, relu)
    return oracle.conv3d_kgs(src64, w64, mask, *l.g, b64, None, l.stride, l.pad, relu)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_s3d_small_clip_every_op(dtype):
    """The whole S3D-shaped stack at a small clip (8x32x32, KGS at 2.1x):
    every conv and pool checked against the oracle applied to the GPU's own
    input buffer of that op (pools bit-exact), and for fp32 the whole chain
    against the oracle run end to end."""
    from paper_2007_09835_amd.stack import S3DStack
    st = S3DStack(1, dtype, "kgs", 2.1, clip=(8, 32))
    x64 = synth.clip_input("s3d-small", 1, "uniform01", 3, 8, 32, 32)
    x_t, x_ref = rounded(x64, dtype)
    st.x.copy_(to_device_ndhwc(x_t))
    st.forward()
    torch.cuda.synchronize()
    layer_by_name = {l.name: (i, l) for i, l in enumerate(st.layers)}
    host = {name: from_device_ndhwc(buf) for name, buf in st.bufs.items()}
    chain = {"x": x_ref}
    for op in st.ops:
        src, dst = (op[2], op[3]) if op[0] == "conv" else (op[1], op[2])
        ref = _s3d_oracle_op(op, st, host[src], layer_by_name)
        if op[0] == "pool":
            assert np.array_equal(host[dst], ref), op
        else:
            i, l = layer_by_name[op[1]]
            off, c_out = op[4], l.c_out
            err = rel_l2(host[dst][:, off:off + c_out], ref)
            assert err <= TOL[dtype], (op, err)
            s_abs = _s3d_oracle_op(op, st, host[src], layer_by_name, absolute=True)
            kt = kept_terms_per_filter(st.masks[i], l.g, l.c_in, l.ks, l.c_out)[None, :, None, None, None]
            assert_within_bound(host[dst][:, off:off + c_out], ref,
                                error_bound(ref, s_abs, kt, dtype), f"s3d small {op[1]}")
        if dtype == "f32":
            full = _s3d_oracle_op(op, st, chain[src], layer_by_name)
            if op[0] == "pool":
                chain[dst] = full
            else:
                if dst not in chain:
                    chain[dst] = np.zeros_like(host[dst])
                chain[dst][:, op[4]:op[4] + full.shape[1]] = full
    if dtype == "f32":
        assert rel_l2(host[st.out_name], chain[st.out_name]) <= 1e-4
    print("s3d small", dtype, "ops", len(st.ops), "rate %.2f" % st.kept_rate(), flush=True)


S3D_LAYERS = synth.s3d_stack()[0]


@pytest.mark.parametrize("li", range(0, len(S3D_LAYERS), 3))
def test_s3d_layers_full_size(li):
    """Every third layer of the S3D-shaped stack at its full 16x224x224-clip
    size, bf16, KGS at 2.1x (1x1x1 layers: whole groups), sampled outputs."""
    l = S3D_LAYERS[li]
    d = synth.layer_params("s3d", l)
    mask = None if l.dense else d.mask
    case = LayerCase("s3d-" + l.name, 1, l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad,
                     "bf16", mask, x_kind="uniform01" if li == 0 else "halfnormal")
    check_sampled(case, f"s3d {l.name}")


# ---------------------------------------------------------------------------
# Pair mapping (2:4 sparse MFMA over pairs of items that no kernel group of a
# 16-filter tile keeps both of; compact weight stream).  Not the planner's
# default, so it is forced through the tuning switch.
# ---------------------------------------------------------------------------

PAIR_TUNES = ["kgs_map=2", "kgs_map=1", "kgs_map=1,pair_mfw=2", "kgs_map=1,pair_mfw=4"]


@pytest.mark.parametrize("tune", PAIR_TUNES)
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_pair_mapping_small_shapes(si, dtype, tune, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", tune)
    tag, n, c_in, c_out, thw, k, stride, pad, keep = SHAPES[si]
    mask = masked(tag, c_out, c_in, k, min(keep, k[0] * k[1] * k[2]))
    case = LayerCase(tag + "p", n, c_in, c_out, thw, k, stride, pad, dtype, mask)
    if c_in > 4:
        assert case.conv.info.variant == (8 if tune == "kgs_map=2" else 7)
    check_full(case, f"pairs {tag} {dtype} {tune}")


@pytest.mark.parametrize("tune", PAIR_TUNES)
@pytest.mark.parametrize("pi", [0, 1, 4, 7, 8])
def test_pair_mapping_pooled_and_split(pi, tune, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", tune)
    tag, n, c_in, c_out, thw, pool, dtype, sparse, residual = POOLED[pi]
    mask = masked(tag, c_out, c_in, (3, 3, 3), 9)
    case = LayerCase(tag + "p", n, c_in, c_out, thw, (3, 3, 3), (1, 1, 1), (1, 1, 1),
                     "bf16" if dtype == "f32" else dtype, mask, residual=residual, pool=pool)
    assert case.conv.info.variant == (8 if tune == "kgs_map=2" else 7)
    check_full(case, f"pairs pooled {tag} {tune}")


@pytest.mark.parametrize("tune", PAIR_TUNES)
@pytest.mark.parametrize("gi", [1, 3, 4])
def test_pair_mapping_group_sizes(gi, tune, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", tune)
    tag, n, c_in, c_out, thw, k, stride, pad, g, keep = GROUPED[gi]
    mask = masked(tag, c_out, c_in, k, keep, g)
    case = LayerCase(tag + "p", n, c_in, c_out, thw, k, stride, pad, "bf16", mask, g=g)
    check_full(case, f"pairs {tag} g={g}")


@pytest.mark.parametrize("tune", PAIR_TUNES)
@pytest.mark.parametrize("variant", ["kgs3", "vanilla3"])
@pytest.mark.parametrize("li", [1, 3, 6])
def test_pair_mapping_c3d_layers(li, variant, tune, monkeypatch):
    """Full-size C3D layers at batch 1 on the pair mapping, sampled outputs."""
    monkeypatch.setenv("RT3D_TUNE", tune)
    stack = synth.c3d_stack(3.0)
    l = stack[li]
    r = synth.rng_for("c3d-pair", variant, l.name, "mask")
    mask = (synth.vanilla_mask(r, *l.groups, l.ks, 3.0) if variant == "vanilla3"
            else synth.kgs_mask(r, *l.groups, l.ks, l.keep))
    case = LayerCase(f"pair-{variant}-{l.name}", 1, l.c_in, l.c_out, (l.t, l.h, l.w), l.k,
                     l.stride, l.pad, "bf16", mask)
    assert case.conv.info.variant == (8 if tune == "kgs_map=2" else 7)
    check_sampled(case, f"pairs c3d {variant} {l.name} {tune}", count=2000)


# ---------------------------------------------------------------------------
# Step counts of every residue: a chunk of the 16-bit union kernel runs
# eight-step passes, at most one four-step pass and a three-step tail whose
# loads are unconditional; each 16-filter tile below keeps exactly 8 n - r
# items (all four groups keep the same ones), so its chunks take n steps for
# n = 1..16, 20 and 27 and every n mod 8.
# ---------------------------------------------------------------------------

STEP_COUNTS = [1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15, 16, 20, 27]


def step_count_mask(c_in, chunk_q, seed):
    """KGS mask [P][Q][27] where tile t keeps, in every chunk of chunk_q
    channel groups, exactly 8 n_t - (t % 8) items (n_t = STEP_COUNTS[t],
    at least one item); the four groups of a tile share their items."""
    rng = np.random.default_rng(seed)
    P, Q = 4 * len(STEP_COUNTS), c_in // 4
    mask = np.zeros((P, Q, 27), dtype=np.uint8)
    for t, n in enumerate(STEP_COUNTS):
        for q0 in range(0, Q, chunk_q):
            slots = chunk_q * 27
            k = max(1, min(slots, 8 * n - (t % 8)))
            pick = rng.choice(slots, size=k, replace=False)
            for s in pick:
                mask[4 * t:4 * t + 4, q0 + s // 27, s % 27] = 1
    return mask


@pytest.mark.parametrize("tune", ["kgs_mfw=1", "kgs_mfw=2", "kgs_mfw=4"])
@pytest.mark.parametrize("c_in", [32, 64])
def test_union_every_step_count(c_in, tune, monkeypatch):
    """Union tiles whose chunks take 1..16, 20 and 27 K-steps (every
    residue mod 8, below and above the eight-step pass), one or two channel
    chunks, 16/32/64-filter tiles, in full against the oracle; with a
    workspace the two-chunk layer also runs split (the second split starts
    mid-stream)."""
    monkeypatch.setenv("RT3D_TUNE", tune + ",cc=32")
    mask = step_count_mask(c_in, 8, 1000 + c_in)
    c_out = 4 * mask.shape[0]
    case = LayerCase(f"steps{c_in}{tune[-1]}", 1, c_in, c_out, (3, 5, 6), (3, 3, 3), (1, 1, 1),
                     (1, 1, 1), "bf16", mask)
    assert case.conv.info.variant == 3
    got, ref = check_full(case, f"union step counts c_in={c_in} {tune}")
    x = to_device_ndhwc(case.x_t)
    unsplit = from_device_ndhwc(case.conv(x, None, use_workspace=False))
    assert_within_bound(unsplit, ref, case.bound_full(ref), f"unsplit {c_in} {tune}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_union_block_order(si, dtype, monkeypatch):
    """The 16-bit union with its 4-filter blocks reordered (kgs_order=1, so
    that tile-mates keep similar items; the epilogue writes every filter to
    its layer position) on the small shapes, both brick widths' plans, in
    full against the oracle."""
    monkeypatch.setenv("RT3D_TUNE", "kgs_order=1,kgs_mfw=1")
    tag, n, c_in, c_out, thw, k, stride, pad, keep = SHAPES[si]
    mask = masked(tag, c_out, c_in, k, min(keep, k[0] * k[1] * k[2]))
    case = LayerCase(tag + "o", n, c_in, c_out, thw, k, stride, pad, dtype, mask)
    check_full(case, f"kgs block order {tag} {dtype}")


@pytest.mark.parametrize("tune", ["kgs_mfw=1", "kgs_mfw=4,slots=128"])
def test_union_block_order_alike_pairs(tune, monkeypatch):
    """Alternate blocks keep two disjoint item sets, so reordering halves the
    K-steps (the planner's CPU test pins that); pooled and split variants of
    the same layer run through the register, LDS-tile and split-reduction
    epilogues with the block map, in full against the oracle."""
    monkeypatch.setenv("RT3D_TUNE", tune + ",kgs_order=1")
    c_in, c_out = 64, 96
    P, Q = c_out // 4, c_in // 4
    mask = np.zeros((P, Q, 27), np.uint8)
    mask[0::2, :, 0:9] = 1
    mask[1::2, :, 9:18] = 1
    for pool, thw in (((1, 1, 1), (3, 6, 7)), ((2, 2, 2), (4, 6, 8))):
        case = LayerCase("alike" + tune[-1] + str(pool[0]), 1, c_in, c_out, thw, (3, 3, 3),
                         (1, 1, 1), (1, 1, 1), "bf16", mask, pool=pool, residual=pool == (1, 1, 1))
        check_full(case, f"alike blocks {tune} pool={pool}")
        x = to_device_ndhwc(case.x_t)
        res = None if case.res_t is None else to_device_ndhwc(case.res_t)
        unsplit = from_device_ndhwc(case.conv(x, res, use_workspace=False))
        ref = case.oracle_full()
        assert_within_bound(unsplit, ref, case.bound_full(ref), f"alike unsplit {tune} {pool}")
