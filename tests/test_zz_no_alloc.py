"""The no-allocation KGS forward (rt3d_kgs_conv3d_fwd_noalloc): its split-K
partial sums live in the library's own device array instead of a caller
workspace.  Through the C ABI it must give exactly what rt3d_kgs_conv3d_fwd
gives with a full workspace (same launch, same kernels), on two calls in a
row with the second on a smaller input (the array keeps the first call's
contents), and it must refuse a layer whose split-K scratch exceeds the
array before launching anything.
"""
import numpy as np
import pytest
import torch

import oracle
from harness import TOL, LayerCase, from_device_ndhwc, rel_l2, to_device_ndhwc
from paper_2007_09835_amd import build, rt3d, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def built():
    build.build(force=False)


def _run_both(case, n):
    """(result of the workspace entry point, result of the no-allocation one,
    workspace bytes) for the first n clips of the case's input."""
    conv = case.conv
    d = conv.desc_for(n)
    x = to_device_ndhwc(case.x_t[:n])
    res = None if case.res_t is None else to_device_ndhwc(case.res_t[:n])
    need = rt3d.rt3d_conv3d_workspace_size(d, conv.info)
    ws = torch.empty(max(need, 4) // 4, dtype=torch.float32, device="cuda")
    y_ref = torch.full(conv.out_shape(n), 7.0, dtype=x.dtype, device="cuda")
    y = torch.full(conv.out_shape(n), -7.0, dtype=x.dtype, device="cuda")
    rt3d.rt3d_kgs_conv3d_fwd(d, conv.info, conv.blob, x, conv.bias, res, y_ref,
                             ws if need else None)
    rt3d.rt3d_kgs_conv3d_fwd_noalloc(d, conv.info, conv.blob, x, conv.bias, res, y)
    torch.cuda.synchronize()
    return from_device_ndhwc(y_ref), from_device_ndhwc(y), need


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(dtype):
    """A layer that splits its input channels (few voxels, 256 channels):
    batch 3, then batch 1 on the same scratch."""
    mask = synth.kgs_mask(synth.rng_for("noalloc", "mask"), 32, 64, 27, 9)
    case = LayerCase("noalloc", 3, 256, 128, (2, 7, 7), (3, 3, 3), (1, 1, 1), (1, 1, 1), dtype,
                     mask, residual=True)
    first_ref, first, need3 = _run_both(case, 3)
    print(f"noalloc {dtype}: split-K scratch {need3} bytes at batch 3", flush=True)
    assert need3 > 0, "the layer must use the scratch"
    assert np.array_equal(first, first_ref)
    assert rel_l2(first, case.oracle_full()) <= TOL[dtype]
    second_ref, second, need1 = _run_both(case, 1)
    print(f"noalloc {dtype}: split-K scratch {need1} bytes at batch 1", flush=True)
    assert np.array_equal(second, second_ref)
    assert rel_l2(second, case.oracle_full()[:1]) <= TOL[dtype]


def test_noalloc_unsplit_layer_and_empty_batch():
    """A layer that needs no scratch runs the same way; n = 0 is a no-op."""
    mask = synth.kgs_mask(synth.rng_for("noalloc2", "mask"), 8, 4, 27, 9)
    case = LayerCase("noalloc2", 1, 16, 32, (4, 10, 12), (3, 3, 3), (1, 1, 1), (1, 1, 1), "bf16",
                     mask)
    ref, got, need = _run_both(case, 1)
    assert need == 0
    assert np.array_equal(got, ref)
    d = case.conv.desc_for(0)
    rt3d.rt3d_kgs_conv3d_fwd_noalloc(d, case.conv.info, case.conv.blob, None, None, None, None)


def test_noalloc_refuses_a_layer_beyond_its_scratch():
    """1x1x1, 8192 -> 4096 channels on 12 clips of 8x8 voxels: the split-K
    workspace exceeds RT3D_NOALLOC_SCRATCH (32 MiB); the call fails before
    launching and leaves y untouched."""
    c_in, c_out, n = 8192, 4096, 12
    rng = synth.rng_for("noalloc3", "w")
    w = torch.from_numpy(rng.standard_normal((c_out, c_in, 1, 1, 1)).astype(np.float32) * 0.01)
    w = w.to(torch.bfloat16)
    mask = synth.kgs_mask(synth.rng_for("noalloc3", "mask"), c_out // 4, c_in // 4, 1, 1)
    mask[:, ::3] = 0
    desc = rt3d.make_desc(n, c_in, c_out, (1, 8, 8), (1, 1, 1), (1, 1, 1), (0, 0, 0), (4, 4),
                          "bf16")
    blob, info = rt3d.rt3d_kgs_pack(desc, w, mask)
    need = rt3d.rt3d_conv3d_workspace_size(desc, info)
    print(f"noalloc refusal: split-K workspace {need} bytes", flush=True)
    assert need > (32 << 20)
    blob_dev = torch.from_numpy(blob).cuda()
    x = torch.zeros((n, 1, 8, 8, c_in), dtype=torch.bfloat16, device="cuda")
    y = torch.full((n, 1, 8, 8, c_out), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rt3d.Rt3dError) as e:
        rt3d.rt3d_kgs_conv3d_fwd_noalloc(desc, info, blob_dev, x, None, None, y)
    assert e.value.status == 2, e.value          # RT3D_ERR_UNSUPPORTED
    assert "scratch" in e.value.detail
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())
