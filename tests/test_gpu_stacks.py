"""GPU parity of the network stacks exactly as bench.py builds and times them
(Section 5.2 / Table 2 report whole-model latency, so the timed pass is the
thing to check).

Each stack is built with ``stack.make_stack`` and the arguments bench.py
passes (fused pools, the benchmark clip, the planner's plans for that batch
size), run once eagerly, then captured in a HIP graph and replayed; every
activation buffer of the replay must equal the eager pass bit for bit, as
bench.py itself requires.  Then every layer's output buffer is checked
against the oracle applied to the GPU's own input buffer of that layer
(so an error does not hide behind the previous layer's rounding), on
sampled outputs plus border voxels, pooled layers through their windows:
relative L2 within the bar and every sampled output within its per-output
bound (harness.error_bound).  The plan each layer ran is printed, and the
plan of the headline's dominant layer is pinned.
"""
import numpy as np
import pytest
import torch

import oracle
from harness import (TOL, assert_within_bound, error_bound, from_device_ndhwc, kept_terms_per_filter,
                     rel_l2, sample_indices, window_indices)
from paper_2007_09835_amd import build, synth
from paper_2007_09835_amd.stack import make_stack

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def built():
    build.build(force=False)


def _plan(conv):
    i32 = np.frombuffer(bytes(conv.info.plan), dtype=np.int32)
    return {"variant": int(conv.info.variant), "brick": tuple(int(v) for v in i32[:3]),
            "slots": int(i32[8]), "cc": int(i32[6]), "mfw": int(i32[10]),
            "pool": (max(conv.desc.qt, 1), max(conv.desc.qh, 1), max(conv.desc.qw, 1))}


def _bench_stack(net, batch, mode, rate):
    """The stack and input exactly as bench.py sets them up."""
    st = make_stack(net, batch, "bf16", mode, rate, fuse_pool=True, group=(4, 4))
    l0 = st.layers[0]
    clip = synth.clip_input("bench-clip", batch, "uniform01", l0.c_in, l0.t, l0.h, l0.w)
    st.x.copy_(synth.to_dtype(clip, "bf16").permute(0, 2, 3, 4, 1).contiguous().cuda())
    return st


def _eager_then_graph(st):
    """Eager pass, then a captured graph replayed over zeroed buffers; the
    replay must reproduce the eager pass bit for bit."""
    st.forward()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in st.bufs.items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st.forward()
    for k, v in st.bufs.items():
        if k != "x":
            v.zero_()
    g.replay()
    torch.cuda.synchronize()
    for k, v in st.bufs.items():
        assert torch.equal(eager[k], v), ("graph replay differs", k)
    del g


def _layer_inputs(st, i):
    l = st.layers[i]
    if i == 0:
        src = st.x
    elif l.input_from:
        src = st.bufs[l.input_from]
    else:
        src = st.bufs[st.layers[i - 1].name]
    res = st.bufs[l.residual_from] if l.residual_from else None
    return src, res


def _check_layer(st, i, tag, mode, rate, clips, count, label):
    l, conv = st.layers[i], st.convs[i]
    d = synth.layer_params(tag, l, mask_kind=mode, rate=rate)
    mask = st.masks[i]
    src, res = _layer_inputs(st, i)
    x64 = from_device_ndhwc(src[clips])[:, :l.c_in]   # buffers may carry pad channels
    r64 = None if res is None else from_device_ndhwc(res[clips])[:, :l.c_out]
    w64 = synth.to_dtype(d.w, "bf16").double().numpy()
    b64 = d.bias.astype(np.float32).astype(np.float64)
    got = from_device_ndhwc(st.bufs[l.name][clips])[:, :l.c_out]
    to, ho, wo = l.out_thw
    full_shape = (len(clips), l.c_out, to, ho, wo)
    pool = _plan(conv)["pool"]
    idx = sample_indices(got.shape, count)
    win = window_indices(idx, got.shape, pool, full_shape)        # [points, window]
    flat = win.ravel()
    g = l.g
    ref_w = oracle.conv3d_points(x64, w64, flat, mask, *g, b64, r64, l.stride, l.pad, l.relu)
    abs_w = oracle.conv3d_points(np.abs(x64), np.abs(w64), flat, mask, *g, np.abs(b64),
                                 None if r64 is None else np.abs(r64), l.stride, l.pad, False)
    m = (flat // (to * ho * wo)) % l.c_out
    kt = kept_terms_per_filter(mask, g, l.c_in, l.ks, l.c_out)[m]
    bound_w = error_bound(ref_w, abs_w, kt, "bf16").reshape(win.shape)
    ref = ref_w.reshape(win.shape).max(axis=1)
    bound = bound_w.max(axis=1)
    err = rel_l2(got.ravel()[idx], ref)
    print(f"{label} {l.name}: plan {_plan(conv)} relL2={err:.3e} ({len(idx)} outputs)", flush=True)
    assert err <= TOL["bf16"], (l.name, err)
    assert_within_bound(got.ravel()[idx], ref, bound, f"{label} {l.name}")


@pytest.mark.parametrize("net,batch,mode,rate", [
    ("c3d", 1, "kgs", 3.0),          # the default bench.py line
    ("c3d", 32, "kgs", 3.0),         # throughput sweep, 3x
    ("c3d", 32, "vanilla", 3.0),     # throughput sweep, vanilla 3x
    ("r2plus1d", 1, "kgs", 3.0),     # bench.py --net r2plus1d
])
def test_stack_as_benchmarked(net, batch, mode, rate):
    st = _bench_stack(net, batch, mode, rate)
    _eager_then_graph(st)
    clips = [0] if batch == 1 else [0, batch - 1]
    for i in range(len(st.layers)):
        _check_layer(st, i, net, mode, rate, clips, 1500 if net == "r2plus1d" else 2500,
                     f"{net} b{batch} {mode}")
    if net == "c3d" and batch == 1 and mode == "kgs":
        # the plans of the default bench line's two largest layers: conv2
        # (32-filter union tiles on 128-slot bricks, pooled through the LDS
        # tile) and conv3b (its dominant layer by time)
        p = _plan(st.convs[1])
        assert p["pool"] == (2, 2, 2), p
        assert (p["variant"], p["slots"], p["brick"], p["mfw"]) == (3, 128, (4, 2, 16), 2), p
        p = _plan(st.convs[3])
        assert p["pool"] == (2, 2, 2), p
        assert (p["variant"], p["slots"], p["brick"], p["mfw"]) == (3, 64, (2, 2, 16), 1), p


def test_s3d_stack_as_benchmarked():
    """bench.py --net s3d: 59 conv launches over two streams in one graph,
    13 pools; every op's output against the oracle on its GPU input."""
    from paper_2007_09835_amd.stack import S3DStack
    st = S3DStack(1, "bf16", "kgs", 2.1)
    l0 = st.layers[0]
    clip = synth.clip_input("bench-clip", 1, "uniform01", l0.c_in, l0.t, l0.h, l0.w)
    st.x.copy_(synth.to_dtype(clip, "bf16").permute(0, 2, 3, 4, 1).contiguous().cuda())
    _eager_then_graph(st)
    by_name = {l.name: (i, l) for i, l in enumerate(st.layers)}
    for op in st.ops:
        if op[0] == "pool":
            _, src, dst, k, stv, pd = op
            got = from_device_ndhwc(st.bufs[dst])
            ref = oracle.maxpool3d(from_device_ndhwc(st.bufs[src]), k, stv, pd)
            assert np.array_equal(got, ref), op
            continue
        _, name, src, dst, c_off, x_off = op
        i, l = by_name[name]
        d = synth.layer_params("s3d", l, mask_kind="kgs", rate=2.1)
        mask = st.masks[i]
        x64 = from_device_ndhwc(st.bufs[src])[:, x_off:x_off + l.c_in]
        got = from_device_ndhwc(st.bufs[dst])[:, c_off:c_off + l.c_out]
        w64 = synth.to_dtype(d.w, "bf16").double().numpy()
        b64 = d.bias.astype(np.float32).astype(np.float64)
        idx = sample_indices(got.shape, 800)
        ref = oracle.conv3d_points(x64, w64, idx, mask, *l.g, b64, None, l.stride, l.pad, l.relu)
        s = oracle.conv3d_points(np.abs(x64), np.abs(w64), idx, mask, *l.g, np.abs(b64), None,
                                 l.stride, l.pad, False)
        to, ho, wo = l.out_thw
        kt = kept_terms_per_filter(mask, l.g, l.c_in, l.ks, l.c_out)[(idx // (to * ho * wo)) % l.c_out]
        err = rel_l2(got.ravel()[idx], ref)
        assert err <= TOL["bf16"], (name, err)
        assert_within_bound(got.ravel()[idx], ref, error_bound(ref, s, kt, "bf16"), f"s3d {name}")
