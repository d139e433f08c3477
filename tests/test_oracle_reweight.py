"""Pins of the oracle's group norms and reweighted penalty (Section 4).

Each check fixes the oracle to something other than itself: a hand-worked
example (tests/golden/reweight_3x2x2.txt), numpy's norm routines, finite
differences of the penalty, the optimality conditions of the proximal map,
and the fixed point of the reweighting iteration on a quadratic objective.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            out[key.strip()] = np.array([float(v) for v in val.split()])
    return out


def _blocks(w, g_m, g_n):
    """Yield (p, q, block) with block = w[p*g_m:, q*g_n:, ...] of one group."""
    c_out, c_in = w.shape[:2]
    for p in range(-(-c_out // g_m)):
        for q in range(-(-c_in // g_n)):
            yield p, q, w[p * g_m:(p + 1) * g_m, q * g_n:(q + 1) * g_n]


def test_golden_hand_worked_example():
    g = _golden("reweight_3x2x2.txt")
    w = g["w"].reshape(3, 2, 1, 1, 2)
    pen = g["pen"].reshape(2, 1, 2)
    r2 = oracle.group_reweight(w, 2, 2, norm=2, scope=0, pen=pen, lam=0.1, eps=1.0, tau=2.0,
                               step=1.0)
    grad = np.zeros(w.shape)
    oracle.group_reweight(w, 2, 2, norm=2, scope=0, pen=pen, lam=0.1, eps=1.0, grad=grad)
    assert np.allclose(r2["norms"].ravel(), g["l2_norms"], rtol=0, atol=1e-15)
    assert r2["reg"] == pytest.approx(g["l2_reg"][0], rel=1e-15)
    assert np.allclose(1.0 / r2["pen_next"].ravel(), g["l2_pen_next_inv"], rtol=1e-15)
    assert np.array_equal(r2["mask"].ravel(), g["l2_mask_tau2"].astype(np.uint8))
    assert np.allclose(r2["w_prox"].ravel(), g["l2_prox"], rtol=0, atol=1e-14)
    assert np.allclose(grad.ravel(), g["l2_grad"], rtol=0, atol=1e-15)
    r1 = oracle.group_reweight(w, 2, 2, norm=1, scope=0, pen=pen, lam=0.1, eps=1.0)
    assert np.array_equal(r1["norms"].ravel(), g["l1_norms"])
    assert r1["reg"] == pytest.approx(g["l1_reg"][0], rel=1e-15)
    v2 = oracle.group_reweight(w, 2, 2, norm=2, scope=1)
    assert np.allclose(v2["norms"].ravel() ** 2, g["vanilla_l2_sq"], rtol=1e-15)
    v1 = oracle.group_reweight(w, 2, 2, norm=1, scope=1)
    assert np.array_equal(v1["norms"].ravel(), g["vanilla_l1"])


@pytest.mark.parametrize("shape,g", [((8, 8, 3, 3, 3), (4, 4)), ((9, 6, 1, 3, 3), (4, 4)),
                                     ((5, 7, 3, 1, 1), (2, 4)), ((16, 12, 3, 3, 3), (16, 4))])
def test_norms_match_numpy(shape, g):
    rng = np.random.default_rng(11)
    w = rng.standard_normal(shape)
    ks = int(np.prod(shape[2:]))
    for norm, ordv in ((2, None), (1, 1)):
        kgs = oracle.group_reweight(w, *g, norm=norm, scope=0)["norms"]
        van = oracle.group_reweight(w, *g, norm=norm, scope=1)["norms"]
        for p, q, blk in _blocks(w, *g):
            b = blk.reshape(blk.shape[0], blk.shape[1], ks)
            for s in range(ks):
                assert kgs[p, q, s] == pytest.approx(
                    np.linalg.norm(b[:, :, s].ravel(), ord=ordv), rel=1e-13)
            assert van[p, q] == pytest.approx(np.linalg.norm(b.ravel(), ord=ordv), rel=1e-13)


@pytest.mark.parametrize("norm,scope", [(2, 0), (1, 0), (2, 1), (1, 1)])
def test_gradient_matches_finite_differences(norm, scope):
    rng = np.random.default_rng(5)
    w = rng.standard_normal((6, 5, 1, 2, 2))
    # keep every weight away from 0 so the l1 norm is differentiable there
    w = np.sign(w) * (0.2 + np.abs(w))
    shape = (2, 2, 4) if scope == 0 else (2, 2)
    pen = rng.uniform(0.5, 2.0, shape)
    lam = 0.3
    grad = np.zeros(w.shape)
    oracle.group_reweight(w, 4, 4, norm=norm, scope=scope, pen=pen, lam=lam, grad=grad)
    h = 1e-6
    fd = np.zeros(w.shape)
    for e in np.ndindex(w.shape):
        wp, wm = w.copy(), w.copy()
        wp[e] += h
        wm[e] -= h
        fp = oracle.group_reweight(wp, 4, 4, norm=norm, scope=scope, pen=pen, lam=lam)["reg"]
        fm = oracle.group_reweight(wm, 4, 4, norm=norm, scope=scope, pen=pen, lam=lam)["reg"]
        fd[e] = (fp - fm) / (2 * h)
    assert np.allclose(grad, fd, rtol=1e-6, atol=1e-8)


def test_gradient_accumulates_and_zero_group_has_zero_gradient():
    w = np.zeros((4, 4, 1, 1, 2))
    w[:, :, 0, 0, 1] = 1.0
    grad = np.full(w.shape, 0.25)
    r = oracle.group_reweight(w, 4, 4, norm=2, scope=0, lam=2.0, grad=grad)
    # position 0: all-zero unit, subgradient 0; position 1: 16 ones, norm 4
    assert np.array_equal(r["norms"].ravel(), [0.0, 4.0])
    assert np.all(grad[..., 0] == 0.25)
    assert np.allclose(grad[..., 1], 0.25 + 2.0 * 1.0 / 4.0, rtol=0, atol=1e-15)


@pytest.mark.parametrize("norm", [1, 2])
def test_prox_satisfies_optimality_conditions(norm):
    """z = prox(w) minimises 1/2 |z - w|^2 + theta * sum_u P_u n_u(z): check the
    subgradient conditions unit by unit, independently of the closed form."""
    rng = np.random.default_rng(3)
    w = rng.standard_normal((8, 8, 1, 1, 3)) * rng.uniform(0.05, 2.0, (8, 8, 1, 1, 3))
    w[:4, 4:, 0, 0, 1] *= 0.02  # a unit small enough to be zeroed
    pen = rng.uniform(0.2, 3.0, (2, 2, 3))
    lam, step = 0.5, 0.7
    z = oracle.group_reweight(w, 4, 4, norm=norm, scope=0, pen=pen, lam=lam, step=step)["w_prox"]
    shrunk = zeroed = 0
    for p, q, blk in _blocks(w, 4, 4):
        zb = z[p * 4:(p + 1) * 4, q * 4:(q + 1) * 4]
        for s in range(3):
            wu, zu = blk[..., s].ravel(), zb[..., s].ravel()
            theta = step * lam * pen[p, q, s]
            if norm == 2:
                nz = np.linalg.norm(zu)
                if nz > 0:
                    shrunk += 1
                    assert np.allclose(zu - wu + theta * zu / nz, 0.0, atol=1e-12)
                else:
                    zeroed += 1
                    assert np.linalg.norm(wu) <= theta * (1 + 1e-12)
            else:
                for wi, zi in zip(wu, zu):
                    if zi != 0:
                        shrunk += 1
                        assert zi - wi + theta * np.sign(zi) == pytest.approx(0.0, abs=1e-12)
                    else:
                        zeroed += 1
                        assert abs(wi) <= theta * (1 + 1e-12)
    assert shrunk > 0 and zeroed > 0


def test_penalty_defaults_update_and_mask():
    rng = np.random.default_rng(8)
    w = rng.standard_normal((8, 4, 3, 3, 3))
    w[4:, :, 0, 0, 0] = 0.0  # one unit of group (1, 0) is exactly zero
    a = oracle.group_reweight(w, 4, 4, norm=2, scope=0, lam=0.7, eps=1e-3, tau=1.5)
    b = oracle.group_reweight(w, 4, 4, norm=2, scope=0, pen=np.ones((2, 1, 27)), lam=0.7,
                              eps=1e-3, tau=1.5)
    assert a["reg"] == b["reg"]
    # with unit penalty factors eq. (3) is the plain group lasso of eq. (2)
    assert a["reg"] == pytest.approx(0.7 * a["norms"].sum(), rel=1e-14)
    assert a["pen_next"][1, 0, 0] == 1.0 / 1e-3
    assert np.array_equal(a["mask"], (a["norms"] > 1.5).astype(np.uint8))
    # tau = 0 prunes exactly the units that are zero and keeps every other one
    z = oracle.group_reweight(w, 4, 4, norm=2, scope=0, tau=0.0)["mask"]
    assert z[1, 0, 0] == 0 and z.sum() == z.size - 1
    v = oracle.group_reweight(w, 4, 4, norm=2, scope=1, tau=5.0)
    assert np.array_equal(v["mask"], np.repeat((v["norms"] > 5.0)[..., None], 27, axis=2)
                          .astype(np.uint8))


def test_norms_scale_and_ignore_order_within_group():
    rng = np.random.default_rng(4)
    w = rng.standard_normal((8, 8, 3, 3, 3))
    base = oracle.group_reweight(w, 4, 4, norm=2)["norms"]
    assert np.allclose(oracle.group_reweight(-2.5 * w, 4, 4, norm=2)["norms"], 2.5 * base,
                       rtol=1e-14)
    perm = w[[1, 0, 3, 2, 4, 5, 6, 7]][:, [3, 1, 2, 0, 7, 6, 5, 4]]
    assert np.allclose(oracle.group_reweight(perm, 4, 4, norm=2)["norms"], base, rtol=1e-14)


def test_reweighting_iteration_reaches_its_fixed_point():
    """Reweighted group lasso on F(W) = 1/2 |W - W0|^2 (a stand-in for the
    training loss): each iteration solves the penalised problem exactly with
    the proximal map and then updates P (Section 4).  A unit that survives
    converges to n* with n0 - n* = lam / (n*^2 + eps) (the stationarity
    condition of the reweighted problem); small units are pruned to 0."""
    rng = np.random.default_rng(21)
    w0 = rng.standard_normal((8, 8, 1, 1, 4)) * 0.1
    w0[:4, :4, 0, 0, 0] *= 20.0  # a strong unit (norm ~8)
    w0[4:, 4:, 0, 0, 2] *= 5.0   # a medium one (norm ~2); the rest have norm ~0.4
    lam, eps = 0.1, 1e-4
    pen = None
    for _ in range(60):
        r = oracle.group_reweight(w0, 4, 4, norm=2, scope=0, pen=pen, lam=lam, eps=eps)
        wt = r["w_prox"]
        pen = oracle.group_reweight(wt, 4, 4, norm=2, scope=0, lam=lam, eps=eps)["pen_next"]
    n0 = oracle.group_reweight(w0, 4, 4, norm=2, scope=0)["norms"]
    nt = oracle.group_reweight(wt, 4, 4, norm=2, scope=0)["norms"]
    alive = nt > 0
    assert alive[0, 0, 0] and alive[1, 1, 2] and alive.sum() == 2
    assert np.allclose(n0[alive] - nt[alive], lam / (nt[alive] ** 2 + eps), rtol=1e-8, atol=0)
