"""Host-side tests of the C ABI (no GPU needed).

* the library loads and exports every function include/rt3d.h declares;
* the canonical KGS sections written by rt3d_kgs_pack are bit-identical to
  the oracle's pack (Section 3 compact format) for every dtype, group size
  and partial-group shape;
* unpack(pack(W, mask)) == W * expand(mask) bit-exactly;
* bookkeeping (kept positions / weights, vanilla detection, sizes);
* every documented error path returns its status code.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
from paper_2007_09835_amd import rt3d

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def built():
    from paper_2007_09835_amd import build
    build.build(force=False)


def header_functions():
    text = open(os.path.join(ROOT, "include", "rt3d.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rt3d_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(rt3d.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(rt3d.EXPORTED) == names


def _np_dtype(dt):
    return {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[dt]


def _weights(rng, shape, dt):
    w = rng.standard_normal(shape).astype(np.float32)
    if dt == "f32":
        return w
    if dt == "f16":
        return w.astype(np.float16)
    return torch.from_numpy(w).to(torch.bfloat16).view(torch.uint16).numpy()


PACK_CASES = [
    # c_out, c_in, k, g_m, g_n, keep_frac
    (32, 16, (3, 3, 3), 4, 4, 0.33),
    (13, 10, (3, 3, 3), 4, 4, 0.4),
    (9, 7, (1, 3, 3), 4, 4, 0.5),
    (6, 11, (3, 1, 1), 4, 4, 0.6),
    (24, 20, (3, 3, 3), 8, 4, 0.3),
    (40, 36, (1, 1, 1), 16, 8, 0.5),
    (5, 6, (1, 1, 3), 4, 4, 0.5),
    (8, 8, (3, 3, 3), 4, 4, 0.0),
    (8, 8, (3, 3, 3), 4, 4, 1.0),
]


@pytest.mark.parametrize("ci", range(len(PACK_CASES)))
@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_canonical_pack_matches_oracle_bitwise(ci, dt):
    c_out, c_in, k, g_m, g_n, frac = PACK_CASES[ci]
    rng = np.random.default_rng(1000 + ci)
    w = _weights(rng, (c_out, c_in, *k), dt)
    P, Q, ks = -(-c_out // g_m), -(-c_in // g_n), k[0] * k[1] * k[2]
    mask = (rng.random((P, Q, ks)) < frac).astype(np.uint8)
    desc = rt3d.make_desc(1, c_in, c_out, (4, 5, 6), k, (1, 1, 1), tuple(x // 2 for x in k),
                          (g_m, g_n), dt)
    blob, info = rt3d.rt3d_kgs_pack(desc, w, mask)
    gp, pos, vp, vals = rt3d.canonical_sections(info, blob, _np_dtype(dt))
    ogp, opos, ovp, ovals = oracle.kgs_pack(w, mask, g_m, g_n)
    assert np.array_equal(gp, ogp)
    assert np.array_equal(pos, opos)
    assert np.array_equal(vp, ovp)
    assert vals.tobytes() == ovals.tobytes()
    assert info.kept_positions == mask.sum()
    assert info.kept_weights == len(ovals)
    assert info.packed_bytes == len(blob) == rt3d.rt3d_kgs_pack_size(desc, mask)
    # round trip
    out = np.zeros_like(w)
    rt3d.rt3d_kgs_unpack(desc, info, blob, out)
    full = np.repeat(np.repeat(mask, g_m, 0), g_n, 1)[:c_out, :c_in].reshape(c_out, c_in, *k)
    expect = np.where(full == 1, w, np.zeros_like(w))
    assert out.tobytes() == expect.tobytes()


@pytest.mark.parametrize("tune", ["kgs_f32=0", "kgs_f32=1"])
def test_pack_never_reads_pruned_weights(tune, monkeypatch):
    """Pruned positions hold NaN; the blob must be identical to packing the
    zero-filled weights (except nothing reads them at all), for the exact
    fp32 layout and the fp32 union layout."""
    monkeypatch.setenv("RT3D_TUNE", tune)
    rng = np.random.default_rng(5)
    w = rng.standard_normal((16, 8, 3, 3, 3)).astype(np.float32)
    mask = (rng.random((4, 2, 27)) < 0.3).astype(np.uint8)
    full = np.repeat(np.repeat(mask, 4, 0), 4, 1).reshape(w.shape)
    w_nan = np.where(full == 1, w, np.float32(np.nan))
    w_zero = np.where(full == 1, w, np.float32(0))
    for dt_w in (w_nan, w_zero):
        desc = rt3d.make_desc(1, 8, 16, (4, 4, 4), dtype="f32")
        blob, info = rt3d.rt3d_kgs_pack(desc, dt_w, mask)
        assert info.variant == (9 if tune.endswith("1") else 4)
        if dt_w is w_nan:
            b_nan = blob
        else:
            b_zero = blob
    assert b_nan.tobytes() == b_zero.tobytes()


def test_vanilla_mask_is_detected():
    rng = np.random.default_rng(2)
    w = rng.standard_normal((16, 16, 3, 3, 3)).astype(np.float32)
    mask = np.zeros((4, 4, 27), dtype=np.uint8)
    mask[rng.random((4, 4)) < 0.4] = 1
    desc = rt3d.make_desc(1, 16, 16, (4, 4, 4), dtype="bf16")
    wb = _weights(rng, w.shape, "bf16")
    _, info = rt3d.rt3d_kgs_pack(desc, wb, mask)
    assert info.vanilla == 1
    mask[0, 0, 0] ^= 1
    _, info = rt3d.rt3d_kgs_pack(desc, wb, mask)
    assert info.vanilla == 0


def test_dense_pack_sizes_and_info():
    desc = rt3d.make_desc(2, 64, 128, (16, 56, 56), dtype="bf16")
    w = _weights(np.random.default_rng(0), (128, 64, 3, 3, 3), "bf16")
    blob, info = rt3d.rt3d_dense_pack(desc, w)
    assert info.packed_bytes == len(blob) == rt3d.rt3d_dense_pack_size(desc)
    assert info.kept_weights == 128 * 64 * 27
    assert rt3d.rt3d_conv3d_out_shape(desc) == (16, 56, 56)
    assert rt3d.rt3d_conv3d_workspace_size(desc, info) == 0


def _brick_slots(desc):
    """Voxel slots per workgroup of the layer's plan (Tiling.slots: the
    ninth int32 of the plan)."""
    w = _weights(np.random.default_rng(1), (desc.c_out, desc.c_in, desc.kt, desc.kh, desc.kw),
                 {0: "f32", 1: "bf16", 2: "f16"}[desc.dtype])
    _, info = rt3d.rt3d_dense_pack(desc, w)
    return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[8])


def _plan_mfw(desc):
    w = _weights(np.random.default_rng(1), (desc.c_out, desc.c_in, desc.kt, desc.kh, desc.kw),
                 {0: "f32", 1: "bf16", 2: "f16"}[desc.dtype])
    _, info = rt3d.rt3d_dense_pack(desc, w)
    return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[10])


def test_brick_width_follows_the_layer_size(monkeypatch):
    """Brick rule (dense packs): 64-slot bricks when 128-slot bricks times
    16-filter tiles give fewer than 1024 waves (one per SIMD of the GPU) for
    pooled 16-bit layers, 8192 for unpooled 16-bit layers (their narrow-tile
    epilogue runs in registers) and 256 for fp32, and for every 16-bit layer
    whose wave tile has four 16-filter rows (on 128-slot bricks those tiles
    leave one wave per SIMD); larger one- and two-row layers keep 128;
    RT3D_TUNE=slots=N overrides the choice at pack time."""
    monkeypatch.delenv("RT3D_TUNE", raising=False)
    pooled_big = rt3d.make_desc(1, 32, 64, (16, 56, 56), dtype="bf16", pool=(2, 2, 2))   # 1568
    pooled_small = rt3d.make_desc(1, 256, 256, (8, 28, 28), dtype="bf16", pool=(2, 2, 2))  # 784
    unpooled = rt3d.make_desc(1, 32, 64, (16, 56, 56), dtype="bf16")       # 1568 waves
    unpooled_big = rt3d.make_desc(4, 32, 64, (16, 56, 56), dtype="f16")    # 6272 waves
    unpooled_huge = rt3d.make_desc(8, 32, 64, (16, 56, 56), dtype="f16")   # 12544 waves
    conv2 = rt3d.make_desc(1, 64, 128, (16, 56, 56), dtype="bf16", pool=(2, 2, 2))   # 32-filter tiles
    wide32 = rt3d.make_desc(32, 256, 256, (8, 28, 28), dtype="bf16")       # 64-filter tiles
    f32 = rt3d.make_desc(1, 256, 256, (8, 28, 28), dtype="f32")             # 784 waves
    f32_small = rt3d.make_desc(1, 16, 32, (8, 28, 28), dtype="f32")         # 49 x 2 = 98 waves
    assert _brick_slots(pooled_big) == 128
    assert _brick_slots(pooled_small) == 64
    assert _brick_slots(unpooled) == 64
    assert _brick_slots(unpooled_big) == 64
    assert _brick_slots(unpooled_huge) == 128
    assert (_plan_mfw(conv2), _brick_slots(conv2)) == (2, 128)
    assert (_plan_mfw(wide32), _brick_slots(wide32)) == (4, 64)
    assert _brick_slots(f32) == 128
    assert _brick_slots(f32_small) == 64
    monkeypatch.setenv("RT3D_TUNE", "slots=128")
    assert _brick_slots(pooled_small) == 128
    assert _brick_slots(f32_small) == 128
    assert _brick_slots(conv2) == 128
    monkeypatch.setenv("RT3D_TUNE", "slots=64")
    assert _brick_slots(pooled_big) == 64
    assert _brick_slots(f32) == 64


def test_dense_tile_width_rules(monkeypatch):
    """Dense 16-bit tile widths for layers of 256+ filters: 64 filters with
    2000+ output voxels, 32 below; 16 for fewer than 256 output voxels, and
    for a shallow reduction (c_in taps < 4096) that the launch model would
    split on wider tiles but not on 16-filter ones (C3D conv3a at batch 1,
    not conv3b, whose reduction is twice as deep; at batch 32 the wide tiles
    fill the GPU unsplit).  fp32 keeps the voxel rule."""
    monkeypatch.delenv("RT3D_TUNE", raising=False)
    k3 = dict(k=(3, 3, 3), pad=(1, 1, 1))
    conv3a = rt3d.make_desc(1, 128, 256, (8, 28, 28), dtype="bf16", **k3)
    conv3b = rt3d.make_desc(1, 256, 256, (8, 28, 28), dtype="bf16", **k3)
    conv3a_b32 = rt3d.make_desc(32, 128, 256, (8, 28, 28), dtype="bf16", **k3)
    conv4b = rt3d.make_desc(1, 512, 512, (4, 14, 14), dtype="bf16", **k3)
    conv5a = rt3d.make_desc(1, 512, 512, (2, 7, 7), dtype="bf16", **k3)
    conv5a_b32 = rt3d.make_desc(32, 512, 512, (2, 7, 7), dtype="bf16", **k3)
    conv5a_f32 = rt3d.make_desc(1, 512, 512, (2, 7, 7), dtype="f32", **k3)
    assert _plan_mfw(conv3a) == 1
    assert _plan_mfw(conv3b) == 4
    assert _plan_mfw(conv3a_b32) == 4
    assert _plan_mfw(conv4b) == 2
    assert _plan_mfw(conv5a) == 1
    assert _plan_mfw(conv5a_b32) == 4
    assert _plan_mfw(conv5a_f32) == 2
    monkeypatch.setenv("RT3D_TUNE", "dense_mfw=4")
    assert _plan_mfw(conv3a) == 4


def test_kgs_tile_width_follows_union_size(monkeypatch):
    """KGS layers with 256+ filters and a 64-filter wave per SIMD walk the
    union of 16 kernel groups (64-filter tiles) when the 16-filter union
    already covers most items; sparser masks and batch-1 layers keep
    16-filter tiles.  Plan fields: mfw is the eleventh int32.  (Checked with
    the union mapping forced: the planner prefers the pair mapping wherever
    it saves K-steps and the union would use narrow tiles.)"""
    monkeypatch.setenv("RT3D_TUNE", "kgs_map=0")
    rng = np.random.default_rng(3)
    w = _weights(rng, (256, 256, 3, 3, 3), "bf16")

    def mfw(n, keep):
        desc = rt3d.make_desc(n, 256, 256, (8, 28, 28), dtype="bf16")
        mask = np.zeros((64, 64, 27), np.uint8)
        for p in range(64):
            for q in range(64):
                mask[p, q, rng.choice(27, keep, replace=False)] = 1
        _, info = rt3d.rt3d_kgs_pack(desc, w, mask)
        return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[10])

    assert mfw(32, 13) == 4   # 16-filter union ~93% of items: the wide union is cheaper
    assert mfw(32, 5) == 1    # ~56%: the narrow union is cheaper
    assert mfw(1, 13) == 1    # batch 1: too few 64-filter waves

    # Deep reductions (512 input channels x 27 taps) take the wide union with
    # fewer voxels, from 512 narrow (16-filter) waves: C3D conv5a at batch 32
    # (2x7x7 outputs, 25 bricks x 32 tiles), not at batch 8 (7 x 32).
    w5 = _weights(rng, (512, 512, 3, 3, 3), "bf16")

    def mfw5(n, keep):
        desc = rt3d.make_desc(n, 512, 512, (2, 7, 7), dtype="bf16")
        mask = np.zeros((128, 128, 27), np.uint8)
        for p in range(128):
            for q in range(128):
                mask[p, q, rng.choice(27, keep, replace=False)] = 1
        _, info = rt3d.rt3d_kgs_pack(desc, w5, mask)
        return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[10])

    assert mfw5(32, 9) == 4
    assert mfw5(8, 9) == 1
    assert mfw5(32, 5) == 1   # the narrow union is still cheaper when sparse

    # Spatial-only 1x3x3 layers with 1.25M+ outputs on 64-slot bricks: the
    # union of eight blocks (R(2+1)D layer 2: 64 -> 144 at 16x56x56)
    w2 = _weights(rng, (144, 64, 1, 3, 3), "bf16")

    def mfw2(n, c_out, thw):
        desc = rt3d.make_desc(n, 64, c_out, thw, (1, 3, 3), (1, 1, 1), (0, 1, 1), dtype="bf16")
        mask = np.zeros(((c_out + 3) // 4, 16, 9), np.uint8)
        for p in range(mask.shape[0]):
            for q in range(16):
                mask[p, q, rng.choice(9, 4, replace=False)] = 1
        _, info = rt3d.rt3d_kgs_pack(desc, w2[:c_out], mask)
        return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[10])

    assert mfw2(1, 144, (16, 56, 56)) == 2
    assert mfw2(1, 144, (8, 28, 28)) == 1    # 0.9M outputs


def _expect_status(status, fn, *args):
    with pytest.raises(rt3d.Rt3dError) as ei:
        fn(*args)
    assert ei.value.status == status, ei.value.detail
    assert ei.value.detail


def test_error_paths():
    rng = np.random.default_rng(3)
    w = rng.standard_normal((8, 8, 3, 3, 3)).astype(np.float32)
    mask = np.ones((2, 2, 27), dtype=np.uint8)
    good = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32")
    blob, info = rt3d.rt3d_kgs_pack(good, w, mask)

    bad_mask = mask.copy()
    bad_mask[1, 1, 5] = 2
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_kgs_pack, good, w, bad_mask)
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_kgs_pack_size,
                   rt3d.make_desc(1, 0, 8, (4, 4, 4)), mask)
    _expect_status(rt3d.RT3D_ERR_UNSUPPORTED, rt3d.rt3d_kgs_pack_size,
                   rt3d.make_desc(1, 8, 8, (4, 4, 4), stride=(3, 1, 1)), mask)
    _expect_status(rt3d.RT3D_ERR_UNSUPPORTED, rt3d.rt3d_kgs_pack_size,
                   rt3d.make_desc(1, 8, 8, (4, 4, 4), g=(2, 4)), mask)
    big = rt3d.make_desc(1, 8, 8, (9, 9, 9), k=(9, 1, 1), pad=(0, 0, 0))
    _expect_status(rt3d.RT3D_ERR_UNSUPPORTED, rt3d.rt3d_kgs_pack_size, big,
                   np.ones((2, 2, 9), np.uint8))
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_kgs_pack_size,
                   rt3d.make_desc(1, 8, 8, (1, 1, 1), k=(3, 3, 3), pad=(0, 0, 0)), mask)
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_conv3d_out_shape,
                   rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype=7))

    # too-small buffer, straight through the C ABI
    lib = rt3d.load()
    small = np.zeros(16, np.uint8)
    inf = rt3d.PackInfo()
    st = lib.rt3d_kgs_pack(ctypes.byref(good), w.ctypes.data, mask.ctypes.data, small.ctypes.data,
                           16, ctypes.byref(inf))
    assert st == rt3d.RT3D_ERR_BUFFER_TOO_SMALL
    st = lib.rt3d_kgs_pack(ctypes.byref(good), None, mask.ctypes.data, small.ctypes.data, 16,
                           ctypes.byref(inf))
    assert st == rt3d.RT3D_ERR_INVALID_ARG

    # blob/desc mismatch and the dense/KGS confusion are caught before any launch
    other = rt3d.make_desc(1, 8, 8, (4, 4, 5), dtype="f32")
    out = np.zeros_like(w)
    _expect_status(rt3d.RT3D_ERR_BLOB_MISMATCH, rt3d.rt3d_kgs_unpack, other, info, blob, out)
    st = lib.rt3d_conv3d_dense_fwd(ctypes.byref(good), ctypes.byref(info), 16, 16, None, None, 16,
                                   None, 0, None)
    assert st == rt3d.RT3D_ERR_BLOB_MISMATCH
    tampered = rt3d.PackInfo.from_buffer_copy(info)
    tampered.magic = 0
    st = lib.rt3d_kgs_conv3d_fwd(ctypes.byref(good), ctypes.byref(tampered), 16, 16, None, None, 16,
                                 None, 0, None)
    assert st == rt3d.RT3D_ERR_BLOB_MISMATCH
    # residual flag without a residual pointer, misaligned pointers
    res_desc = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", residual=True)
    _, rinfo = rt3d.rt3d_kgs_pack(res_desc, w, mask)
    st = lib.rt3d_kgs_conv3d_fwd(ctypes.byref(res_desc), ctypes.byref(rinfo), 256, 256, None, None,
                                 256, None, 0, None)
    assert st == rt3d.RT3D_ERR_INVALID_ARG
    st = lib.rt3d_kgs_conv3d_fwd(ctypes.byref(good), ctypes.byref(info), 256, 258, None, None, 256,
                                 None, 0, None)
    assert st == rt3d.RT3D_ERR_INVALID_ARG
    st = lib.rt3d_maxpool3d_fwd(1, 8, 4, 4, 4, 5, 2, 2, 1, 2, 2, 0, 0, 0, 0, 256, 256, None)
    assert st == rt3d.RT3D_ERR_INVALID_ARG
    # padding above half the window
    st = lib.rt3d_maxpool3d_fwd(1, 8, 4, 4, 4, 3, 3, 3, 1, 1, 1, 2, 1, 1, 0, 256, 256, None)
    assert st == rt3d.RT3D_ERR_INVALID_ARG
    # fused concatenation: the slice must fit and keep 4-channel alignment
    cat = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", y_c_total=12, y_c_off=6)
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_conv3d_out_shape, cat)
    cat = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", y_c_total=18, y_c_off=2)
    _expect_status(rt3d.RT3D_ERR_UNSUPPORTED, rt3d.rt3d_conv3d_out_shape, cat)
    cat = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", y_c_total=16, y_c_off=8)
    assert rt3d.rt3d_conv3d_out_shape(cat) == (4, 4, 4)
    # input channel slice: must fit; network-input layers (c_in <= 4) read whole voxels
    sl = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", x_c_total=12, x_c_off=6)
    _expect_status(rt3d.RT3D_ERR_INVALID_ARG, rt3d.rt3d_conv3d_out_shape, sl)
    sl = rt3d.make_desc(1, 3, 8, (4, 4, 4), dtype="bf16", x_c_total=8, x_c_off=0)
    _expect_status(rt3d.RT3D_ERR_UNSUPPORTED, rt3d.rt3d_conv3d_out_shape, sl)
    sl = rt3d.make_desc(1, 8, 8, (4, 4, 4), dtype="f32", x_c_total=20, x_c_off=12)
    assert rt3d.rt3d_conv3d_out_shape(sl) == (4, 4, 4)
    assert lib.rt3d_status_string(99)
    assert lib.rt3d_status_string(rt3d.RT3D_ERR_HIP) == b"HIP runtime error"


def test_group_units_and_workspace():
    d = rt3d.make_group_desc(9, 6, k=(1, 3, 3), g=(4, 4))
    assert rt3d.rt3d_group_units(d) == 3 * 2 * 9
    d.scope = rt3d.RT3D_SCOPE_VANILLA
    assert rt3d.rt3d_group_units(d) == 3 * 2
    # one workgroup per filter group and block of channel groups, a float each
    c5 = rt3d.make_group_desc(512, 512, g=(4, 4), dtype="bf16")
    ws = rt3d.rt3d_group_workspace_size(c5)
    assert ws % 256 == 0 and 4 * 2048 <= ws <= 4 * 4096


def test_group_reweight_error_paths():
    lib = rt3d.load()
    good = rt3d.make_group_desc(8, 8, g=(4, 4), dtype="f32")

    def call(desc, w=256, eps=1e-6, lam=1.0, step=1.0, tau=0.0, reg=None, ws=None, ws_bytes=0,
             norms=None, wp=None):
        return lib.rt3d_group_reweight(ctypes.byref(desc), w, None, lam, eps, tau, step, norms,
                                       None, reg, None, None, wp, ws, ws_bytes, None)

    def desc(**kw):
        d = rt3d.GroupDesc.from_buffer_copy(good)
        for k, v in kw.items():
            setattr(d, k, v)
        return d

    assert call(desc(norm=3)) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(desc(scope=2)) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(desc(dtype=9)) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(desc(c_out=0)) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(desc(g_m=0)) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(desc(g_n=17)) == rt3d.RT3D_ERR_UNSUPPORTED
    assert call(desc(kt=8)) == rt3d.RT3D_ERR_UNSUPPORTED
    # one unit's weights must fit the staging buffer: 16 * 16 * 49 > 12288
    assert call(desc(g_m=16, g_n=16, kt=1, kh=7, kw=7)) == rt3d.RT3D_ERR_UNSUPPORTED
    assert call(good, w=None) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, eps=0.0) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, eps=float("nan")) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, lam=-1.0) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, step=-1.0) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, tau=float("inf")) == rt3d.RT3D_ERR_INVALID_ARG
    assert call(good, norms=258) == rt3d.RT3D_ERR_INVALID_ARG          # misaligned float*
    assert call(desc(dtype=rt3d.RT3D_BF16), wp=257) == rt3d.RT3D_ERR_INVALID_ARG
    # the penalty value needs the per-workgroup workspace
    assert call(good, reg=256) == rt3d.RT3D_ERR_BUFFER_TOO_SMALL
    assert call(good, reg=256, ws=512, ws_bytes=2) == rt3d.RT3D_ERR_BUFFER_TOO_SMALL
    # nothing requested: nothing launched
    assert call(good) == rt3d.RT3D_OK


def test_small_channel_kernel_choice():
    """The small-input-channel kernel takes layers with c_in <= 4 whose halo
    lines fit one word per lane (at most 253 elements) and whose rows hold a
    multiple of 4 elements (w * c_in % 4 == 0: every line of a brick starts at
    the same offset within its word); the rest run on the item kernel.  Pack
    is host-only, so the choice is visible without a GPU."""
    rng = np.random.default_rng(7)

    def variant(c_in, w, k=(3, 3, 3), stride=(1, 1, 1), pad=(1, 1, 1)):
        desc = rt3d.make_desc(1, c_in, 32, (4, 6, w), k, stride, pad, dtype="bf16")
        _, info = rt3d.rt3d_dense_pack(desc, _weights(rng, (32, c_in) + tuple(k), "bf16"))
        return info.variant

    assert variant(3, 44) == 5          # 132 elements per row
    assert variant(3, 45) == 1          # 135: lines start at different word offsets
    assert variant(1, 12) == 5
    assert variant(1, 9) == 1
    # line elements (31 sw + kw) c_in: 252 fits, 256 does not
    assert variant(4, 40, (1, 1, 1), (1, 2, 2), (0, 0, 0)) == 5
    assert variant(4, 40, (1, 2, 2), (1, 2, 2), (0, 0, 0)) == 1
    # stems: 1x7x7 stride (1, 2, 2) on RGB, 207 elements per line
    assert variant(3, 224, (1, 7, 7), (1, 2, 2), (0, 3, 3)) == 5


def test_stack_pads_ragged_channel_pitch():
    """The R(2+1)D stack gives layer outputs whose channel count is not a
    multiple of 8 a pitch rounded up to 8 (zero pad channels), so the next
    layer stages whole 16-byte pieces; residual sources keep their width.
    Built on the host (packing and buffers only, no launch)."""
    from paper_2007_09835_amd.stack import Stack
    st = Stack("r2plus1d", 1, "bf16", "kgs", 3.0, device="cpu")
    residual_sources = {l.residual_from for l in st.layers if l.residual_from}
    padded = {}
    for l in st.layers:
        b = st.bufs[l.name]
        if l.name in residual_sources:
            assert b.shape[-1] == l.c_out
        assert b.shape[-1] % 8 == 0 or l.name in residual_sources, l.name
        assert b.shape[-1] - l.c_out < 8
        if b.shape[-1] != l.c_out:
            padded[l.name] = (l.c_out, b.shape[-1])
            assert float(b[..., l.c_out:].abs().sum()) == 0.0
    assert padded == {"stem_s": (45, 48), "l3b0c0_s": (230, 232), "l4b0c0_s": (460, 464),
                      "l5b0c0_s": (921, 928)}


def test_channel_chunk_width_rule(monkeypatch):
    """16-bit chunks of 32 channels widen while the halo fits, except on
    layers of fewer than 256 output voxels whose 32-channel chunks carry 16
    or more K-steps (C3D conv5a at batch 1 keeps 32; conv4b and a 1x3x3
    layer of the same size widen)."""
    monkeypatch.delenv("RT3D_TUNE", raising=False)

    def cc(desc):
        w = _weights(np.random.default_rng(1), (desc.c_out, desc.c_in, desc.kt, desc.kh, desc.kw),
                     "bf16")
        _, info = rt3d.rt3d_dense_pack(desc, w)
        return int(np.frombuffer(bytes(info.plan), dtype=np.int32)[6])

    conv5a = rt3d.make_desc(1, 512, 512, (2, 7, 7), dtype="bf16")
    conv5a_b32 = rt3d.make_desc(32, 512, 512, (2, 7, 7), dtype="bf16")
    conv4b = rt3d.make_desc(1, 512, 512, (4, 14, 14), dtype="bf16")
    spatial = rt3d.make_desc(1, 512, 512, (2, 7, 7), k=(1, 3, 3), pad=(0, 1, 1), dtype="bf16")
    assert cc(conv5a) == 32
    assert cc(conv5a_b32) > 32
    assert cc(conv4b) > 32
    assert cc(spatial) > 32
