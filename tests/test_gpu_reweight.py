"""GPU parity of the group norms / reweighted group-lasso penalty kernel
(Section 4) against the float64 oracle, through the C ABI.

Tolerances: the kernel sums in float32, so norms, penalty factors, the
penalty value, gradients and float32 proximal outputs must agree with the
oracle to 1e-5 relative L2; proximal outputs rounded to bf16 / fp16 to 1e-2
/ 1e-3.  The mask is a float decision: it must equal (GPU norm > tau)
exactly, and the oracle's mask wherever the oracle's norm is not within
1e-5 (relative) of tau.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2007_09835_amd import rt3d, synth

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
PROX_TOL = {"f32": 1e-5, "bf16": 1e-2, "f16": 1e-3}


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


def weights(tag, c_out, c_in, k, g, dtype):
    w = synth.unit_scaled_weights(synth.rng_for("reweight", tag), c_out, c_in, k, g)
    t = synth.to_dtype(w, dtype)
    return t.cuda(), t.to(torch.float64).numpy()


def run_gpu(desc, w_dev, pen=None, lam=0.1, eps=1e-4, tau=0.0, step=1.0, grad0=None,
            in_place=False):
    units = rt3d.rt3d_group_units(desc)
    dev = w_dev.device
    out = {
        "norms": torch.full((units,), -1.0, device=dev),
        "pen_next": torch.full((units,), -1.0, device=dev),
        "reg": torch.full((1,), -1.0, device=dev),
        "mask": torch.full((-(-desc.c_out // desc.g_m), -(-desc.c_in // desc.g_n),
                            desc.kt * desc.kh * desc.kw), 7, dtype=torch.uint8, device=dev),
        "grad": (torch.zeros(w_dev.shape, device=dev) if grad0 is None
                 else torch.from_numpy(grad0).float().to(dev)),
    }
    if in_place:
        out["w_prox"] = w_dev.clone()
        src = out["w_prox"]
    else:
        out["w_prox"] = torch.zeros_like(w_dev)
        src = w_dev
    ws = torch.zeros(rt3d.rt3d_group_workspace_size(desc) // 4, device=dev)
    pen_t = None if pen is None else torch.from_numpy(np.ascontiguousarray(pen, np.float32)).to(dev)
    rt3d.rt3d_group_reweight(desc, src, pen_t, lam, eps, tau, step, norms=out["norms"],
                             pen_next=out["pen_next"], reg=out["reg"], mask=out["mask"],
                             grad=out["grad"], w_prox=out["w_prox"], workspace=ws)
    torch.cuda.synchronize()
    return {k: v.to(torch.float64).cpu().numpy() if k != "mask" else v.cpu().numpy()
            for k, v in out.items()}


def check(desc, w64, got, pen=None, lam=0.1, eps=1e-4, tau=0.0, step=1.0, grad0=None,
          dtype="f32"):
    grad = np.zeros(w64.shape) if grad0 is None else grad0.astype(np.float32).astype(np.float64)
    ref = oracle.group_reweight(w64, desc.g_m, desc.g_n, norm=desc.norm, scope=desc.scope,
                                pen=pen, lam=lam, eps=eps, tau=tau, step=step, grad=grad)
    n_ref = ref["norms"].ravel()
    assert rel_l2(got["norms"], n_ref) <= 1e-5
    assert rel_l2(got["pen_next"], ref["pen_next"].ravel()) <= 1e-5
    assert abs(got["reg"][0] - ref["reg"]) <= 1e-5 * max(abs(ref["reg"]), 1e-30)
    assert rel_l2(got["grad"], grad) <= 1e-5
    assert rel_l2(got["w_prox"], ref["w_prox"]) <= PROX_TOL[dtype]
    # mask: the GPU's own decision, and the oracle's away from the threshold
    per_pos = desc.scope == rt3d.RT3D_SCOPE_KGS
    ks = desc.kt * desc.kh * desc.kw
    gn = got["norms"].reshape(got["mask"].shape[:2] + ((ks,) if per_pos else (1,)))
    assert np.array_equal(got["mask"], np.broadcast_to(gn > np.float32(tau), got["mask"].shape))
    rn = ref["norms"].reshape(gn.shape)
    clear = np.broadcast_to(np.abs(rn - tau) > 1e-5 * np.maximum(rn, abs(tau)), got["mask"].shape)
    assert np.array_equal(got["mask"][clear], ref["mask"][clear])
    return ref


CASES = [
    # tag, c_out, c_in, k, g, dtype, norm, scope
    ("full44", 16, 16, (3, 3, 3), (4, 4), "f32", 2, 0),
    ("partial", 9, 6, (1, 3, 3), (4, 4), "f32", 2, 0),
    ("g24", 5, 7, (3, 1, 1), (2, 4), "f32", 1, 0),
    ("g164", 16, 12, (3, 3, 3), (16, 4), "bf16", 2, 0),
    ("vanilla", 24, 20, (3, 3, 3), (4, 4), "f32", 2, 1),
    ("vanilla_l1", 10, 13, (3, 3, 3), (4, 4), "bf16", 1, 1),
    ("big_kernel", 8, 8, (7, 7, 7), (4, 4), "f32", 2, 0),
    ("f16", 32, 24, (3, 3, 3), (4, 4), "f16", 2, 0),
    ("l1_f16", 12, 20, (1, 3, 3), (4, 4), "f16", 1, 0),
    # R(2+1)D partial mid widths (230 = 4*57 + 2) and a C3D-sized layer
    ("r21d_temporal", 64, 230, (3, 1, 1), (4, 4), "bf16", 2, 0),
    ("r21d_spatial", 230, 64, (1, 3, 3), (4, 4), "bf16", 2, 1),
    ("conv3b", 256, 256, (3, 3, 3), (4, 4), "bf16", 2, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_reweight_matches_oracle(case):
    tag, c_out, c_in, k, g, dtype, norm, scope = case
    print("reweight case", case, flush=True)
    desc = rt3d.make_group_desc(c_out, c_in, k, g, dtype, norm, scope)
    w_dev, w64 = weights(tag, c_out, c_in, k, g, dtype)
    units = rt3d.rt3d_group_units(desc)
    rng = synth.rng_for("reweight", tag, "pen")
    pen = rng.uniform(0.5, 20.0, units).astype(np.float32).astype(np.float64)
    grad0 = rng.standard_normal(w64.shape).astype(np.float32)
    ushape = ((-(-c_out // g[0]), -(-c_in // g[1])) + ((k[0] * k[1] * k[2],) if scope == 0 else ()))
    tau = float(np.median(oracle.group_reweight(w64, *g, norm=norm, scope=scope)["norms"]))
    got = run_gpu(desc, w_dev, pen, lam=0.05, eps=1e-4, tau=tau, step=0.5, grad0=grad0)
    check(desc, w64, got, pen.reshape(ushape), lam=0.05, eps=1e-4, tau=tau, step=0.5,
          grad0=grad0, dtype=dtype)


def test_default_penalty_in_place_and_repeatable():
    desc = rt3d.make_group_desc(20, 12, (3, 3, 3), (4, 4), "bf16", 2, 0)
    w_dev, w64 = weights("inplace", 20, 12, (3, 3, 3), (4, 4), "bf16")
    a = run_gpu(desc, w_dev, None, lam=0.2, tau=0.1)
    b = run_gpu(desc, w_dev, None, lam=0.2, tau=0.1, in_place=True)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
    check(desc, w64, a, None, lam=0.2, tau=0.1, dtype="bf16")


def test_pen_next_in_place_with_pen():
    desc = rt3d.make_group_desc(16, 16, (3, 3, 3), (4, 4), "f32", 2, 0)
    w_dev, w64 = weights("penplace", 16, 16, (3, 3, 3), (4, 4), "f32")
    pen = torch.linspace(0.5, 3.0, rt3d.rt3d_group_units(desc), device="cuda")
    pen_host = pen.cpu().double().numpy()
    rt3d.rt3d_group_reweight(desc, w_dev, pen, 0.1, 1e-3, 0.0, 1.0, pen_next=pen)
    torch.cuda.synchronize()
    ref = oracle.group_reweight(w64, 4, 4, norm=2, scope=0, pen=pen_host.reshape(4, 4, 27),
                                eps=1e-3)
    assert rel_l2(pen.cpu().numpy(), ref["pen_next"].ravel()) <= 1e-5


def test_zero_units_are_pruned_and_take_eps():
    desc = rt3d.make_group_desc(8, 8, (1, 1, 3), (4, 4), "f32", 2, 0)
    w = torch.randn(8, 8, 1, 1, 3, generator=torch.Generator().manual_seed(1))
    w[4:, :4, 0, 0, 1] = 0.0
    got = run_gpu(desc, w.cuda(), None, lam=0.1, eps=1e-3, tau=0.0)
    mask = got["mask"]
    assert mask[1, 0, 1] == 0 and mask.sum() == mask.size - 1
    # eps reaches the kernel as a float32
    assert got["pen_next"].reshape(2, 2, 3)[1, 0, 1] == np.float32(1.0) / np.float32(1e-3)
    assert np.all(got["w_prox"][4:, :4, 0, 0, 1] == 0.0)
    assert np.all(got["grad"][4:, :4, 0, 0, 1] == 0.0)


def test_reweighted_iterations_prune_small_units():
    """Four reweighting iterations on the quadratic stand-in objective
    1/2 |W - W0|^2 (each solved by the proximal map), GPU against oracle,
    then the mask that prunes the units driven (close) to zero."""
    desc = rt3d.make_group_desc(64, 64, (3, 3, 3), (4, 4), "f32", 2, 0)
    w_dev, w64 = weights("iterate", 64, 64, (3, 3, 3), (4, 4), "f32")
    lam, eps, tau = 5e-6, 1e-6, 1e-4
    units = rt3d.rt3d_group_units(desc)
    pen_g = torch.ones(units, device="cuda")
    wt_g = torch.empty_like(w_dev)
    mask_g = torch.empty((16, 16, 27), dtype=torch.uint8, device="cuda")
    pen_o = None
    for _ in range(4):
        rt3d.rt3d_group_reweight(desc, w_dev, pen_g, lam, eps, 0.0, 1.0, w_prox=wt_g)
        rt3d.rt3d_group_reweight(desc, wt_g, None, lam, eps, tau, 1.0, pen_next=pen_g,
                                 mask=mask_g)
        wt_o = oracle.group_reweight(w64, 4, 4, pen=pen_o, lam=lam, eps=eps)["w_prox"]
        r = oracle.group_reweight(wt_o, 4, 4, lam=lam, eps=eps, tau=tau)
        pen_o = r["pen_next"]
    torch.cuda.synchronize()
    assert rel_l2(wt_g.cpu().double().numpy(), wt_o) <= 1e-4
    kept = mask_g.cpu().numpy()
    assert 0.05 < kept.mean() < 0.95           # structure, not all-or-nothing
    agree = (kept == r["mask"]).mean()
    assert agree >= 0.999, agree


def test_c3d_stack_norms_bf16():
    """Every KGS layer of the C3D stack at its real size (bf16 weights)."""
    for layer in synth.c3d_layers():
        if layer.dense:
            continue
        desc = rt3d.make_group_desc(layer.c_out, layer.c_in, layer.k, (4, 4), "bf16", 2, 0)
        print("reweight c3d layer", layer.name, flush=True)
        w_dev, w64 = weights("c3d_" + layer.name, layer.c_out, layer.c_in, layer.k, (4, 4), "bf16")
        norms = torch.empty(rt3d.rt3d_group_units(desc), device="cuda")
        reg = torch.empty(1, device="cuda")
        ws = torch.zeros(rt3d.rt3d_group_workspace_size(desc) // 4, device="cuda")
        rt3d.rt3d_group_reweight(desc, w_dev, None, 1.0, 1e-6, 0.0, 1.0, norms=norms, reg=reg,
                                 workspace=ws)
        torch.cuda.synchronize()
        ref = oracle.group_reweight(w64, 4, 4, norm=2, scope=0)
        assert rel_l2(norms.cpu().numpy(), ref["norms"].ravel()) <= 1e-5
        assert abs(reg.item() - ref["reg"]) <= 1e-5 * ref["reg"]


def test_penalty_workspace_reuse_and_graph_replay():
    """One workspace serves layers of different sizes in turn, and a captured
    call gives the eager result on every replay."""
    descs = [rt3d.make_group_desc(64, 48, (3, 3, 3), (4, 4), "bf16", 2, 0),
             rt3d.make_group_desc(256, 256, (3, 3, 3), (4, 4), "bf16", 2, 0),
             rt3d.make_group_desc(40, 36, (1, 3, 3), (4, 4), "bf16", 1, 1)]
    ws = torch.zeros(max(rt3d.rt3d_group_workspace_size(d) for d in descs) // 4, device="cuda")
    reg = torch.empty(1, device="cuda")
    for rep in range(2):
        for i, d in enumerate(descs):
            w_dev, w64 = weights("reuse%d" % i, d.c_out, d.c_in, (d.kt, d.kh, d.kw), (4, 4), "bf16")
            rt3d.rt3d_group_reweight(d, w_dev, None, 0.5, 1e-6, 0.0, 1.0, reg=reg, workspace=ws)
            torch.cuda.synchronize()
            ref = oracle.group_reweight(w64, 4, 4, norm=d.norm, scope=d.scope, lam=0.5)["reg"]
            assert abs(reg.item() - ref) <= 1e-5 * ref, (rep, i)
    d = descs[1]
    w_dev, _ = weights("reuse1", d.c_out, d.c_in, (3, 3, 3), (4, 4), "bf16")
    rt3d.rt3d_group_reweight(d, w_dev, None, 0.5, 1e-6, 0.0, 1.0, reg=reg, workspace=ws)
    torch.cuda.synchronize()
    eager = reg.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rt3d.rt3d_group_reweight(d, w_dev, None, 0.5, 1e-6, 0.0, 1.0, reg=reg, workspace=ws)
    for _ in range(3):
        reg.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(reg, eager)
        _ = (w_dev.float() * 2).sum().item()  # unrelated eager work between replays
