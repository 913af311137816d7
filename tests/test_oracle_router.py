"""Pins of the router oracle (oracle/router.py) against things other than
itself: brute-force top-k, the k = E and k = 1 special cases, float64 torch
autograd of an independently written forward, central finite differences,
softmax invariants, and a planted mistake that one of them must catch."""
import itertools

import numpy as np
import pytest
import torch

from oracle import router as orr


def case(T=13, h=9, E=6, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, h))
    Wr = rng.standard_normal((E, h)) * scale
    dg = rng.standard_normal((T, min(E, 3)))
    return X, Wr, dg


def test_topk_brute_force_and_ties():
    rng = np.random.default_rng(1)
    z = rng.integers(-3, 4, size=(50, 7)).astype(np.float64)   # many exact ties
    for k in (1, 2, 3, 7):
        got = orr.topk(z, k)
        for t in range(z.shape[0]):
            want = sorted(range(7), key=lambda e: (-z[t, e], e))[:k]
            assert got[t].tolist() == want


def test_k_equals_E_gates_are_the_softmax():
    X, Wr, _ = case()
    f = orr.router_fwd(X, Wr, Wr.shape[0])
    p_sorted = np.take_along_axis(f["p"], f["idx"], axis=1)
    assert np.allclose(f["gates"], p_sorted, rtol=0, atol=1e-15)
    assert np.allclose(f["p"].sum(axis=1), 1.0, atol=1e-15)


def test_k1_gate_is_one_and_gradient_zero():
    X, Wr, _ = case()
    f = orr.router_fwd(X, Wr, 1)
    assert np.array_equal(f["gates"], np.ones((X.shape[0], 1)))
    b = orr.router_bwd(X, Wr, f["idx"], f["logits"], np.random.default_rng(2).standard_normal((X.shape[0], 1)))
    assert np.max(np.abs(b["dlogits"])) < 1e-15


def _torch_grads(X, Wr, idx, dg):
    """Independent forward in torch (float64), selection held fixed."""
    Xt = torch.tensor(X, requires_grad=True)
    Wt = torch.tensor(Wr, requires_grad=True)
    z = Xt @ Wt.T
    z.retain_grad()
    p = torch.softmax(z, dim=1)
    sel = torch.gather(p, 1, torch.tensor(idx, dtype=torch.int64))
    g = sel / sel.sum(dim=1, keepdim=True)
    (g * torch.tensor(dg)).sum().backward()
    return z.grad.numpy(), Xt.grad.numpy(), Wt.grad.numpy(), g.detach().numpy()


@pytest.mark.parametrize("T,h,E,k", [(13, 9, 6, 3), (40, 16, 8, 2), (7, 5, 4, 4), (20, 12, 16, 8)])
def test_against_torch_autograd(T, h, E, k):
    X, Wr, _ = case(T, h, E, seed=T + E)
    dg = np.random.default_rng(k).standard_normal((T, k))
    f = orr.router_fwd(X, Wr, k)
    zg, Xg, Wg, g = _torch_grads(X, Wr, f["idx"], dg)
    assert np.allclose(f["gates"], g, rtol=0, atol=1e-14)
    b = orr.router_bwd(X, Wr, f["idx"], f["logits"], dg)
    assert np.allclose(b["dlogits"], zg, rtol=0, atol=1e-13)
    assert np.allclose(b["dX"], Xg, rtol=0, atol=1e-12)
    assert np.allclose(b["dWr"], Wg, rtol=0, atol=1e-12)


def test_finite_differences():
    X, Wr, _ = case(6, 5, 5, seed=9, scale=3.0)      # well separated logits
    k = 2
    dg = np.random.default_rng(4).standard_normal((6, k))
    f = orr.router_fwd(X, Wr, k)
    b = orr.router_bwd(X, Wr, f["idx"], f["logits"], dg)
    eps = 1e-6

    def L(Xv, Wv):
        g = orr.router_fwd(Xv, Wv, k)
        assert np.array_equal(g["idx"], f["idx"])       # selection unchanged
        return float((g["gates"] * dg).sum())

    for t, j in itertools.product(range(6), range(5)):
        Xp, Xm = X.copy(), X.copy()
        Xp[t, j] += eps
        Xm[t, j] -= eps
        assert abs((L(Xp, Wr) - L(Xm, Wr)) / (2 * eps) - b["dX"][t, j]) < 1e-7
    for e, j in itertools.product(range(5), range(5)):
        Wp, Wm = Wr.copy(), Wr.copy()
        Wp[e, j] += eps
        Wm[e, j] -= eps
        assert abs((L(X, Wp) - L(X, Wm)) / (2 * eps) - b["dWr"][e, j]) < 1e-7


def test_softmax_invariants():
    X, Wr, _ = case(30, 7, 9, seed=5)
    k = 3
    f = orr.router_fwd(X, Wr, k)
    shifted = orr.router_fwd(None, None, k, logits=f["logits"] + 17.25)
    assert np.array_equal(shifted["idx"], f["idx"])
    assert np.allclose(shifted["gates"], f["gates"], rtol=0, atol=1e-14)
    dg = np.random.default_rng(6).standard_normal((30, k))
    b = orr.router_bwd(X, Wr, f["idx"], f["logits"], dg)
    assert np.max(np.abs(b["dlogits"].sum(axis=1))) < 1e-14     # rows of dz sum to 0
    nonsel = np.ones_like(b["dlogits"], dtype=bool)
    nonsel[np.arange(30)[:, None], f["idx"]] = False
    # unselected experts receive p_e * (0 - <p, dp>) = 0 since <p, dp> = 0
    assert np.max(np.abs(b["dlogits"][nonsel])) < 1e-14


def test_planted_mistake_missing_renormalisation_term():
    """Dropping the -p_i/S^2 term of the renormalisation Jacobian must fail
    the autograd pin."""
    X, Wr, _ = case(13, 9, 6, seed=13)
    k = 3
    dg = np.random.default_rng(7).standard_normal((13, k))
    f = orr.router_fwd(X, Wr, k)
    zg, _, _, _ = _torch_grads(X, Wr, f["idx"], dg)

    def broken(X, Wr, idx, logits, dgates):
        z, d = np.asarray(logits, dtype=np.float64), np.asarray(dgates, dtype=np.float64)
        p = orr.softmax(z)
        sel = np.take_along_axis(p, idx, axis=1)
        dp = np.zeros_like(z)
        np.add.at(dp, (np.arange(z.shape[0])[:, None], idx), d / sel.sum(axis=1, keepdims=True))
        return p * (dp - (p * dp).sum(axis=1, keepdims=True))

    assert not np.allclose(broken(X, Wr, f["idx"], f["logits"], dg), zg, atol=1e-6)
