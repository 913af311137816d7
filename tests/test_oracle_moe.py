"""Pins for the oracle's MoE forward and chunked-recompute backward (no GPU).

Each check compares the oracle with something other than itself:
* a brute-force per-token, per-slot Python loop written here (forward);
* float64 autograd of a dense formulation written here with torch ops
  (every expert on every token, then a gather of the routed ones): it yields
  the gradients without any hand-derived backward;
* central finite differences of <Y, dY> (directional derivatives);
* special cases that reduce to a textbook dense SwiGLU MLP (E = k = 1, and
  identical experts with gates summing to one), built from torch's own SiLU;
* Eq. (6)/(7) chunk invariance for every chunk count;
* a few planted mistakes, each of which must make one of these pins fail.
"""
import math

import numpy as np
import pytest
import torch

from oracle import moe as om


def tiny_case(T=8, h=8, F=16, E=4, k=2, seed=0, dup=True):
    rng = np.random.default_rng(seed)
    if dup:
        idx = rng.integers(0, E, size=(T, k))
    else:
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    g = rng.uniform(0.1, 1.0, size=(T, k))
    X = rng.standard_normal((T, h))
    W1 = rng.standard_normal((E, 2 * F, h)) / math.sqrt(h)
    W2 = rng.standard_normal((E, h, F)) / math.sqrt(F)
    dY = rng.standard_normal((T, h))
    return X, idx, g, W1, W2, dY


def brute_forward(X, idx, g, W1, W2):
    T, h = X.shape
    E, twoF, _ = W1.shape
    F = twoF // 2
    k = idx.shape[1]
    Y = [[0.0] * h for _ in range(T)]
    for t in range(T):
        for j in range(k):
            e = int(idx[t, j])
            u = [sum(W1[e, r, c] * X[t, c] for c in range(h)) for r in range(twoF)]
            a = [u[f] / (1.0 + math.exp(-u[f])) * u[F + f] for f in range(F)]
            for o in range(h):
                y = sum(W2[e, o, f] * a[f] for f in range(F))
                Y[t][o] += g[t, j] * y
    return np.array(Y)


def autograd_reference(X, idx, g, W1, W2, dY):
    """Dense masked formulation: all experts on all tokens, gather, gate-sum."""
    tX = torch.tensor(X, dtype=torch.float64, requires_grad=True)
    tg = torch.tensor(g, dtype=torch.float64, requires_grad=True)
    tW1 = torch.tensor(W1, dtype=torch.float64, requires_grad=True)
    tW2 = torch.tensor(W2, dtype=torch.float64, requires_grad=True)
    F = W1.shape[1] // 2
    u = torch.einsum("th,efh->tef", tX, tW1)                   # [T,E,2F]
    a = torch.nn.functional.silu(u[..., :F]) * u[..., F:]     # [T,E,F]
    yall = torch.einsum("tef,ehf->teh", a, tW2)                # [T,E,h]
    tidx = torch.tensor(idx, dtype=torch.int64)
    ysel = torch.gather(yall, 1, tidx[:, :, None].expand(-1, -1, X.shape[1]))
    Y = (tg[:, :, None] * ysel).sum(1)
    Y.backward(torch.tensor(dY, dtype=torch.float64))
    return (Y.detach().numpy(), tX.grad.numpy(), tg.grad.numpy(),
            tW1.grad.numpy(), tW2.grad.numpy())


def rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ------------------------------------------------------------------ forward
@pytest.mark.parametrize("C", [1, 2, 3, 8])
def test_forward_matches_brute_force(C):
    X, idx, g, W1, W2, _ = tiny_case(T=7, h=5, F=6, E=3, k=2, seed=C)
    assert rel(om.moe_fwd(X, idx, g, W1, W2, C), brute_forward(X, idx, g, W1, W2)) < 1e-12


# ----------------------------------------------------------------- backward
@pytest.mark.parametrize("seed,dup", [(0, True), (1, False), (2, True)])
@pytest.mark.parametrize("C", [1, 3])
def test_backward_matches_autograd(seed, dup, C):
    X, idx, g, W1, W2, dY = tiny_case(T=9, h=8, F=12, E=4, k=3, seed=seed, dup=dup)
    Y_ref, dX_ref, dg_ref, dW1_ref, dW2_ref = autograd_reference(X, idx, g, W1, W2, dY)
    assert rel(om.moe_fwd(X, idx, g, W1, W2, C), Y_ref) < 1e-12
    out = om.moe_bwd(X, idx, g, W1, W2, dY, C)
    assert rel(out["dX"], dX_ref) < 1e-12
    assert rel(out["dgates"], dg_ref) < 1e-12
    assert rel(out["dW1"], dW1_ref) < 1e-12
    assert rel(out["dW2"], dW2_ref) < 1e-12


def fd_error(seed=0, C=2, eps=1e-6):
    """Largest relative gap between the oracle's gradient and a central
    finite difference of L = <Y, dY> along random directions."""
    X, idx, g, W1, W2, dY = tiny_case(seed=seed)
    rng = np.random.default_rng(100 + seed)
    grads = om.moe_bwd(X, idx, g, W1, W2, dY, C)
    worst = 0.0
    for name in ("X", "g", "W1", "W2"):
        base = {"X": X, "g": g, "W1": W1, "W2": W2}
        V = rng.standard_normal(base[name].shape)

        def L(s):
            args = dict(base)
            args[name] = base[name] + s * V
            Y = om.moe_fwd(args["X"], idx, args["g"], args["W1"], args["W2"], C)
            return float(np.sum(Y * dY))

        fd = (L(eps) - L(-eps)) / (2 * eps)
        gname = {"X": "dX", "g": "dgates", "W1": "dW1", "W2": "dW2"}[name]
        an = float(np.sum(grads[gname] * V))
        worst = max(worst, abs(fd - an) / max(abs(an), 1e-3))
    return worst


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_finite_differences(seed):
    assert fd_error(seed) < 1e-7


# ------------------------------------------------------------ special cases
def textbook_swiglu_mlp(x, Wg, Wu, Wd):
    tx = torch.tensor(x, dtype=torch.float64)
    return (torch.nn.functional.silu(tx @ torch.tensor(Wg).T) * (tx @ torch.tensor(Wu).T)
            @ torch.tensor(Wd).T).numpy()


def test_single_expert_is_dense_swiglu():
    X, _, _, W1, W2, _ = tiny_case(T=11, h=8, F=16, E=1, k=1, seed=3)
    idx = np.zeros((11, 1), dtype=np.int64)
    g = np.ones((11, 1))
    F = 16
    ref = textbook_swiglu_mlp(X, W1[0, :F], W1[0, F:], W2[0])
    for C in (1, 4):
        assert rel(om.moe_fwd(X, idx, g, W1, W2, C), ref) < 1e-12


def test_identical_experts_sum_to_dense():
    T, h, F, E, k = 10, 8, 16, 5, 3
    X, idx, g, W1, W2, _ = tiny_case(T=T, h=h, F=F, E=E, k=k, seed=4)
    W1 = np.repeat(W1[:1], E, axis=0)
    W2 = np.repeat(W2[:1], E, axis=0)
    g = g / g.sum(axis=1, keepdims=True)
    ref = textbook_swiglu_mlp(X, W1[0, :F], W1[0, F:], W2[0])
    assert rel(om.moe_fwd(X, idx, g, W1, W2, 2), ref) < 1e-12


def test_dgate_identity():
    """<dY[t], y> equals <W2^T dY[t], a> for every slot (used by the GPU
    path to get the gate gradient without recomputing FC2)."""
    X, idx, g, W1, W2, dY = tiny_case(seed=5)
    F = W1.shape[1] // 2
    for t in range(X.shape[0]):
        for j in range(idx.shape[1]):
            e = idx[t, j]
            u = W1[e] @ X[t]
            a = om.silu(u[:F]) * u[F:]
            assert abs(dY[t] @ (W2[e] @ a) - (W2[e].T @ dY[t]) @ a) < 1e-12


# --------------------------------------------------------- chunk invariance
def test_chunk_invariance():
    X, idx, g, W1, W2, dY = tiny_case(T=13, h=8, F=8, E=4, k=2, seed=6)
    Y1 = om.moe_fwd(X, idx, g, W1, W2, 1)
    B1 = om.moe_bwd(X, idx, g, W1, W2, dY, 1)
    for C in (2, 3, 4, 5, 8, 13, 16):
        assert rel(om.moe_fwd(X, idx, g, W1, W2, C), Y1) < 1e-13
        B = om.moe_bwd(X, idx, g, W1, W2, dY, C)
        for key in ("dX", "dgates", "dW1", "dW2"):
            assert rel(B[key], B1[key]) < 1e-12, (C, key)


# ---------------------------------------------------- sampled-output forms
def test_token_forms_match_chunked():
    X, idx, g, W1, W2, dY = tiny_case(T=12, h=8, F=8, E=4, k=3, seed=8)
    Y = om.moe_fwd(X, idx, g, W1, W2, 3)
    B = om.moe_bwd(X, idx, g, W1, W2, dY, 3)
    toks = [0, 5, 11]
    assert rel(om.moe_fwd_tokens(X, idx, g, W1, W2, toks), Y[toks]) < 1e-12
    dX, dg = om.moe_bwd_tokens(X, idx, g, W1, W2, dY, toks)
    assert rel(dX, B["dX"][toks]) < 1e-12
    assert rel(dg, B["dgates"][toks]) < 1e-12
    for e in range(4):
        dW1e, dW2e = om.moe_dW_expert(X, idx, g, W1, W2, dY, e)
        assert rel(dW1e, B["dW1"][e]) < 1e-12
        assert rel(dW2e, B["dW2"][e]) < 1e-12


def test_sigmoid_extremes():
    z = np.array([-800.0, -40.0, 0.0, 40.0, 800.0])
    s = om.sigmoid(z)
    assert np.all(np.isfinite(s))
    assert s[2] == 0.5 and s[0] == 0.0 and s[-1] == 1.0
    ref = torch.sigmoid(torch.tensor(z)).numpy()
    assert np.allclose(s, ref, rtol=1e-15, atol=0)


# ------------------------------------------------------- planted mistakes
def _autograd_gap():
    X, idx, g, W1, W2, dY = tiny_case(T=9, h=8, F=12, E=4, k=3, seed=0)
    Y_ref, dX_ref, dg_ref, dW1_ref, dW2_ref = autograd_reference(X, idx, g, W1, W2, dY)
    out = om.moe_bwd(X, idx, g, W1, W2, dY, 2)
    return max(rel(om.moe_fwd(X, idx, g, W1, W2, 2), Y_ref), rel(out["dX"], dX_ref),
               rel(out["dgates"], dg_ref), rel(out["dW1"], dW1_ref), rel(out["dW2"], dW2_ref))


@pytest.mark.parametrize("mistake", ["silu_grad_drops_term", "silu_sign", "unstable_dispatch",
                                     "chunk_overlap"])
def test_planted_mistakes_are_caught(monkeypatch, mistake):
    if mistake == "silu_grad_drops_term":
        monkeypatch.setattr(om, "silu_grad", lambda z: om.sigmoid(z))
    elif mistake == "silu_sign":
        monkeypatch.setattr(om, "silu", lambda z: z * om.sigmoid(-z))
    elif mistake == "unstable_dispatch":
        real = om.dispatch

        def bad(idx, t0, t1, E):
            d = real(idx, t0, t1, E)
            ss = d["sorted_slot"].copy()
            for e in range(E):           # reverse slot order inside each group
                a, b = d["offsets"][e], d["offsets"][e + 1]
                ss[a:b] = ss[a:b][::-1].copy()
            d["sorted_slot"] = ss
            return d
        monkeypatch.setattr(om, "dispatch", bad)
        rng = np.random.default_rng(1)
        idx = rng.integers(0, 3, size=(6, 2))
        from test_oracle_permute import brute_dispatch
        _, ss, _ = brute_dispatch(idx.tolist(), 0, 6, 3)
        assert om.dispatch(idx, 0, 6, 3)["sorted_slot"].tolist() != ss
        return
    elif mistake == "chunk_overlap":
        monkeypatch.setattr(om, "chunk_ranges",
                            lambda T, C: [(max(0, i * T // C - 1), (i + 1) * T // C) for i in range(C)])
    assert _autograd_gap() > 1e-6 or fd_error() > 1e-6


def test_dW_columns_match_full():
    X, idx, g, W1, W2, dY = tiny_case(T=12, h=8, F=8, E=4, k=3, seed=9)
    B = om.moe_bwd(X, idx, g, W1, W2, dY, 2)
    fs = [0, 3, 7]
    for e in range(4):
        # whole, and summed over blocks of 1, 2 and 5 slots (the form used for
        # experts with half a million slots)
        for block in (32768, 1, 2, 5):
            g1, u1, c2 = om.moe_dW_expert_columns(X, idx, g, W1, W2, dY, e, fs, block=block)
            assert rel(g1, B["dW1"][e][fs]) < 1e-12
            assert rel(u1, B["dW1"][e][[8 + f for f in fs]]) < 1e-12
            assert rel(c2, B["dW2"][e][:, fs]) < 1e-12
