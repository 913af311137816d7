"""Router in front of the MoE expert layer, plain fp64 NumPy (test
infrastructure only: imported by tests/, by the smoke check and by the
benchmark's CPU baseline; the product path never calls it).

Passages followed
-----------------
* Table 2 rows 9-10: the router reads the layer input x (D_t b s h bytes
  stored) and produces e_n logits per token (D_t b s e_n bytes stored).
* Table 2 "score mul" (row 13): the routing scores multiply the expert
  outputs; these are the `gates` the expert layer takes.
* Section 1 and Section 2: every token is routed to its top-k experts by a
  gating network; expert capacity is not capped.

Readings
--------
* The router is a bias-free linear map, logits = X Wr^T with Wr [E, h],
  followed by a softmax over the E experts; the k experts with the largest
  logits are selected (equal logits: the lower expert id first) and their
  probabilities are renormalised to sum to one (the routing recipe of the
  fp32 test workload).
* Selection is decided on the logits; softmax is monotone, so this is the
  order of the probabilities.
* The backward takes dgates (the expert layer's gate gradient) and returns
  dlogits, dX (the router's contribution to the input gradient) and dWr, by
  the chain rule through the renormalisation and the softmax; the selection
  itself is piecewise constant and passes no gradient.
"""
from __future__ import annotations

from typing import Dict

import numpy as np


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def logits_of(X, Wr) -> np.ndarray:
    """logits[t, e] = <X[t], Wr[e]>."""
    return _f64(X) @ _f64(Wr).T


def softmax(z) -> np.ndarray:
    z = _f64(z)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def topk(logits, k: int) -> np.ndarray:
    """Indices of the k largest logits per row, largest first; equal logits
    put the lower expert id first."""
    z = np.asarray(logits)
    T, E = z.shape
    ids = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((ids, -z), axis=-1)   # primary: -logit, then id
    return order[:, :k].astype(np.int32)


def router_fwd(X, Wr, k: int, logits=None) -> Dict[str, np.ndarray]:
    """Forward: logits, probabilities, top-k ids and renormalised gates.
    `logits` may be given to take the selection from another precision's
    logits (the probabilities and gates are still computed in fp64)."""
    z = logits_of(X, Wr) if logits is None else _f64(logits)
    p = softmax(z)
    idx = topk(z, k)
    sel = np.take_along_axis(p, idx, axis=1)
    gates = sel / sel.sum(axis=1, keepdims=True)
    return {"logits": z, "p": p, "idx": idx, "gates": gates}


def router_bwd(X, Wr, idx, logits, dgates) -> Dict[str, np.ndarray]:
    """Backward from dgates [T, k] through gates = p[idx] / sum(p[idx]) and
    p = softmax(logits): returns dlogits [T, E], dX [T, h], dWr [E, h]."""
    X, Wr, z, dg = _f64(X), _f64(Wr), _f64(logits), _f64(dgates)
    idx = np.asarray(idx)
    T, E = z.shape
    p = softmax(z)
    sel = np.take_along_axis(p, idx, axis=1)            # p at the selected ids
    S = sel.sum(axis=1, keepdims=True)
    # renormalisation: d gates_j / d p_m = [m = i_j] / S - p_{i_j} / S^2 for m
    # among the selected ids (and 0 otherwise)
    dp = np.zeros((T, E))
    np.add.at(dp, (np.arange(T)[:, None], idx), dg / S)
    c = (dg * sel).sum(axis=1, keepdims=True) / (S * S)
    mask = np.zeros((T, E), dtype=bool)
    mask[np.arange(T)[:, None], idx] = True
    dp -= np.where(mask, c, 0.0)
    # softmax: dz = p * (dp - <p, dp>)
    dz = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    return {"dlogits": dz, "dX": dz @ Wr, "dWr": dz.T @ X}
