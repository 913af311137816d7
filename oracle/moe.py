"""fp64 oracle of the chunked MoE expert layer (test infrastructure only).

What is computed (paper Section 4.1):

* Eq. (4): Y = F_w(X) = combine(expert(dispatch(X))).
* Eq. (5): X_grad = B_w(Y_grad, F_w(X)).
* Eq. (6): the tokens are cut into c contiguous chunks; each chunk runs
  dispatch -> expert computation -> combine on its own and the outputs are
  concatenated.
* Eq. (7): the backward visits the chunks one after another; for each chunk it
  first recomputes that chunk's forward (recomputation) and then
  back-propagates it; nothing from the forward pass is kept.

The layer itself, as read from Table 2 (rows 11-14: the activated expert
stores its input and a 2*g_e wide FC1 output, then the score multiply and the
add follow the expert):

    for token t and slot j with expert e = idx[t, j] and gate g = gates[t, j]:
        u      = W1[e] @ X[t]                 (2F,)   rows 0..F-1 gate, F..2F-1 up
        a      = silu(u[:F]) * u[F:]          (F,)    SwiGLU
        y_tj   = W2[e] @ a                    (h,)
        Y[t]   = sum_j g * y_tj               j ascending

The backward is the exact derivative of that map (given dY = Y_grad).

Readings of the paper used here (it is silent on these points):
* SwiGLU is not spelled out; the fused FC1 of width 2*g_e (Table 2 row 12) is
  read as [gate | up] with a = silu(gate) * up and no biases.
* The score (gate) multiplies the expert output (Table 2 "score mul" after
  the expert rows); gates need not sum to one.
* Chunk i covers tokens [floor(i*T/C), floor((i+1)*T/C)); empty chunks are
  skipped; backward visits chunks in ascending order and chunk i uses its own
  rows of Y_grad (Eq. (7) writes the whole Y_grad into every term).
* Dispatch orders the chunk's slots (global slot id s = t*k + j) by expert,
  ties by ascending slot id (a stable sort).

Precision: everything is float64.  bf16 inputs are passed in already rounded
(they are exact in float64); intermediate bf16 rounding of the GPU path is not
emulated.

Pins (tests/test_oracle_*.py): brute-force per-token Python loops; float64
autograd of a dense, masked formulation written independently in the test;
central finite differences; the E=k=1 and identical-experts special cases,
which reduce to a textbook dense SwiGLU MLP; chunk invariance for every C;
a brute-force double loop for the dispatch permutation.
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# elementwise pieces of the expert FFN
# ---------------------------------------------------------------------------
def sigmoid(z: np.ndarray) -> np.ndarray:
    """Logistic function, evaluated without overflow for either sign of z."""
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def silu(z: np.ndarray) -> np.ndarray:
    return z * sigmoid(z)


def silu_grad(z: np.ndarray) -> np.ndarray:
    """d/dz [z * sigmoid(z)] = sigmoid(z) * (1 + z * (1 - sigmoid(z)))."""
    s = sigmoid(z)
    return s * (1.0 + z * (1.0 - s))


# ---------------------------------------------------------------------------
# chunking (Eq. (6)) and dispatch (the "dispatch" of Eq. (4))
# ---------------------------------------------------------------------------
def chunk_ranges(T: int, C: int) -> List[Tuple[int, int]]:
    """Token ranges of the C chunks of Eq. (6); empty ranges are dropped."""
    if C < 1:
        raise ValueError("C must be >= 1")
    out = []
    for i in range(C):
        t0, t1 = (i * T) // C, ((i + 1) * T) // C
        if t1 > t0:
            out.append((t0, t1))
    return out


def dispatch(idx: np.ndarray, t0: int, t1: int, E: int) -> Dict[str, np.ndarray]:
    """Group the slots of tokens [t0, t1) by expert.

    Returns
      counts[E]        slots per expert in the chunk
      offsets[E+1]     exclusive prefix sum of counts (offsets[E] = n)
      sorted_slot[n]   global slot ids t*k+j, grouped by expert, ascending
                       slot id within an expert
      row_of_slot[n]   for the chunk's i-th slot (global id t0*k + i): its row
                       in the grouped order (inverse of sorted_slot)
    """
    k = idx.shape[1]
    expert_of = np.asarray(idx[t0:t1], dtype=np.int64).reshape(-1)
    n = expert_of.size
    counts = np.bincount(expert_of, minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    order = np.argsort(expert_of, kind="stable")
    sorted_slot = t0 * k + order
    row_of_slot = np.empty(n, dtype=np.int64)
    row_of_slot[order] = np.arange(n)
    return {"counts": counts, "offsets": offsets,
            "sorted_slot": sorted_slot, "row_of_slot": row_of_slot}


def expert_counts(idx: np.ndarray, E: int) -> np.ndarray:
    """Slots received per local expert over all tokens (the count that the
    paper's "first notification" delivers, Section 4.2)."""
    return np.bincount(np.asarray(idx, dtype=np.int64).reshape(-1),
                       minlength=E).astype(np.int64)


# ---------------------------------------------------------------------------
# one chunk: F_w(X_i) and B_w(Y_grad_i, F_w(X_i))
# ---------------------------------------------------------------------------
def _f64(a):
    return np.asarray(a, dtype=np.float64)


def forward_chunk(X, idx, gates, W1, W2, t0, t1):
    """F_w(X_i) for chunk [t0, t1): dispatch -> expert FFN -> combine.

    Returns Y_i [t1-t0, h] and the chunk's stored activations (which the
    chunked algorithm throws away after use)."""
    E, twoF, h = W1.shape
    F = twoF // 2
    k = idx.shape[1]
    d = dispatch(idx, t0, t1, E)
    sorted_slot, offsets = d["sorted_slot"], d["offsets"]
    tok = sorted_slot // k
    x_perm = _f64(X)[tok]                            # gathered expert inputs
    n = sorted_slot.size
    u = np.zeros((n, twoF))
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            u[r0:r1] = x_perm[r0:r1] @ _f64(W1[e]).T
    a = silu(u[:, :F]) * u[:, F:]
    y = np.zeros((n, h))
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            y[r0:r1] = a[r0:r1] @ _f64(W2[e]).T
    # combine: token t sums g[t, j] * y of its j-th slot, j ascending
    g = _f64(gates)
    row = d["row_of_slot"].reshape(t1 - t0, k)
    Yi = np.zeros((t1 - t0, h))
    for j in range(k):
        Yi += g[t0:t1, j:j + 1] * y[row[:, j]]
    acts = {"dispatch": d, "u": u, "a": a, "y": y}
    return Yi, acts


def backward_chunk(X, idx, gates, W1, W2, dY, t0, t1):
    """B_w(Y_grad_i, F_w(X_i)) with the chunk's forward recomputed first.

    Returns (dX_i [t1-t0, h], dg_i [t1-t0, k], dW1 part [E,2F,h],
    dW2 part [E,h,F])."""
    E, twoF, h = W1.shape
    F = twoF // 2
    k = idx.shape[1]
    _, acts = forward_chunk(X, idx, gates, W1, W2, t0, t1)     # recompute
    d, u, a, y = acts["dispatch"], acts["u"], acts["a"], acts["y"]
    sorted_slot, offsets = d["sorted_slot"], d["offsets"]
    tok = sorted_slot // k
    jj = sorted_slot % k
    g_row = _f64(gates)[tok, jj]                                # gate per row
    dy_row = _f64(dY)[tok]                                      # [n, h]
    x_perm = _f64(X)[tok]

    # combine backward: Y[t] = sum_j g y  ->  dy_e = g * dY[t], dg = <dY[t], y>
    dg_row = np.einsum("nh,nh->n", dy_row, y)
    dy_e = g_row[:, None] * dy_row
    da = np.zeros((sorted_slot.size, F))
    dW1 = np.zeros((E, twoF, h))
    dW2 = np.zeros((E, h, F))
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            da[r0:r1] = dy_e[r0:r1] @ _f64(W2[e])
            dW2[e] = dy_e[r0:r1].T @ a[r0:r1]
    ug, uu = u[:, :F], u[:, F:]
    du = np.concatenate([da * uu * silu_grad(ug), da * silu(ug)], axis=1)
    dx_perm = np.zeros((sorted_slot.size, h))
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            dx_perm[r0:r1] = du[r0:r1] @ _f64(W1[e])
            dW1[e] = du[r0:r1].T @ x_perm[r0:r1]
    # un-permute: token t sums the input gradients of its k slots, j ascending
    row = d["row_of_slot"].reshape(t1 - t0, k)
    dXi = np.zeros((t1 - t0, h))
    for j in range(k):
        dXi += dx_perm[row[:, j]]
    dgi = dg_row[row]
    return dXi, dgi, dW1, dW2


# ---------------------------------------------------------------------------
# FCDA: Eq. (6) forward and Eq. (7) chunked-recompute backward
# ---------------------------------------------------------------------------
def moe_fwd(X, idx, gates, W1, W2, C: int = 1) -> np.ndarray:
    """Y = concat(F_w(X_1), ..., F_w(X_c)) (Eq. (6)); C=1 is Eq. (4)."""
    T, h = X.shape
    Y = np.zeros((T, h))
    for t0, t1 in chunk_ranges(T, C):
        Y[t0:t1], _ = forward_chunk(X, idx, gates, W1, W2, t0, t1)
    return Y


def moe_bwd(X, idx, gates, W1, W2, dY, C: int = 1):
    """Eq. (7): per chunk (ascending), recompute F_w(X_i) then B_w; the input
    gradient is the concatenation, the weight gradients are summed.

    Returns dict dX [T,h], dgates [T,k], dW1 [E,2F,h], dW2 [E,h,F]."""
    T, h = X.shape
    k = idx.shape[1]
    dX = np.zeros((T, h))
    dg = np.zeros((T, k))
    dW1 = np.zeros(W1.shape)
    dW2 = np.zeros(W2.shape)
    for t0, t1 in chunk_ranges(T, C):
        dXi, dgi, dW1i, dW2i = backward_chunk(X, idx, gates, W1, W2, dY, t0, t1)
        dX[t0:t1] = dXi
        dg[t0:t1] = dgi
        dW1 += dW1i
        dW2 += dW2i
    return {"dX": dX, "dgates": dg, "dW1": dW1, "dW2": dW2}


# ---------------------------------------------------------------------------
# Sampled outputs for full-size parity: each token's output depends on that
# token only (Eq. (4) per token), so a few tokens can be checked one by one.
# ---------------------------------------------------------------------------
def _slot_ffn(x, W1e, W2e):
    F = W1e.shape[0] // 2
    u = _f64(W1e) @ _f64(x)
    a = silu(u[:F]) * u[F:]
    return u, a, _f64(W2e) @ a


def moe_fwd_tokens(X, idx, gates, W1, W2, tokens: Iterable[int]) -> np.ndarray:
    """Y rows for the given tokens only (the per-token form of Eq. (4))."""
    tokens = list(tokens)
    k = idx.shape[1]
    out = np.zeros((len(tokens), X.shape[1]))
    for i, t in enumerate(tokens):
        for j in range(k):
            _, _, y = _slot_ffn(X[t], W1[idx[t, j]], W2[idx[t, j]])
            out[i] += float(gates[t, j]) * y
    return out


def moe_bwd_tokens(X, idx, gates, W1, W2, dY, tokens: Iterable[int]):
    """dX and dgates rows for the given tokens only (per-token Eq. (5))."""
    tokens = list(tokens)
    k = idx.shape[1]
    F = W1.shape[1] // 2
    dX = np.zeros((len(tokens), X.shape[1]))
    dg = np.zeros((len(tokens), k))
    for i, t in enumerate(tokens):
        dy = _f64(dY[t])
        for j in range(k):
            e = idx[t, j]
            u, a, y = _slot_ffn(X[t], W1[e], W2[e])
            dg[i, j] = dy @ y
            da = float(gates[t, j]) * (_f64(W2[e]).T @ dy)
            ug, uu = u[:F], u[F:]
            du = np.concatenate([da * uu * silu_grad(ug), da * silu(ug)])
            dX[i] += _f64(W1[e]).T @ du
    return dX, dg


def moe_dW_expert(X, idx, gates, W1, W2, dY, e: int):
    """Full dW1[e], dW2[e]: sums over every slot routed to expert e."""
    k = idx.shape[1]
    F = W1.shape[1] // 2
    slots = np.nonzero(np.asarray(idx).reshape(-1) == e)[0]
    tok = slots // k
    jj = slots % k
    x = _f64(X[tok])
    g = _f64(gates)[tok, jj]
    u = x @ _f64(W1[e]).T
    a = silu(u[:, :F]) * u[:, F:]
    dy_e = g[:, None] * _f64(dY[tok])
    dW2 = dy_e.T @ a
    da = dy_e @ _f64(W2[e])
    ug, uu = u[:, :F], u[:, F:]
    du = np.concatenate([da * uu * silu_grad(ug), da * silu(ug)], axis=1)
    dW1 = du.T @ x
    return dW1, dW2


def moe_dW_expert_columns(X, idx, gates, W1, W2, dY, e: int, fs, block: int = 32768):
    """Selected columns f of expert e's weight gradients, each from its
    definition over the expert's slots: rows f and F+f of dW1[e] and column f
    of dW2[e].  Returns (dW1_gate [len(fs), h], dW1_up [len(fs), h],
    dW2_col [h, len(fs)]).

    The sum over the expert's slots is taken `block` slots at a time (in
    ascending slot order), so that at most `block` gathered rows of X and dY
    are held in fp64 at once: a hot expert of the paper's worst case holds
    half a million slots."""
    k = idx.shape[1]
    F = W1.shape[1] // 2
    fs = np.asarray(list(fs), dtype=np.int64)
    slots = np.nonzero(np.asarray(idx).reshape(-1) == e)[0]
    W1g = _f64(W1[e][fs])                           # [|fs|, h]
    W1u = _f64(W1[e][F + fs])
    W2c = _f64(W2[e][:, fs])                        # [h, |fs|]
    h = W1g.shape[1]
    g1 = np.zeros((len(fs), h))
    u1 = np.zeros((len(fs), h))
    c2 = np.zeros((h, len(fs)))
    gates64 = _f64(gates)
    for b0 in range(0, len(slots), max(1, int(block))):
        sl = slots[b0:b0 + block]
        tok = sl // k
        jj = sl % k
        x = _f64(X[tok])
        g = gates64[tok, jj]
        dy = _f64(dY[tok])
        ug = x @ W1g.T                              # [rows, |fs|]
        uu = x @ W1u.T
        a = silu(ug) * uu
        da = g[:, None] * (dy @ W2c)                # [rows, |fs|]
        du_g = da * uu * silu_grad(ug)
        du_u = da * silu(ug)
        g1 += du_g.T @ x
        u1 += du_u.T @ x
        c2 += (g[:, None] * dy).T @ a
    return g1, u1, c2
