"""Seeded synthetic inputs for the chunked MoE expert layer.

This module is the only code shared by the fp64 oracle side (tests) and the
HIP side (tests, bench).  It draws routing and tensors and does nothing of the
layer's own arithmetic: no dispatch, no expert FFN, no combine, no memory
model.  Routing is always NumPy (PCG64), so that a (config, seed) pair
yields the same routing on every machine; tensors come either from NumPy
(small cases the oracle checks in full) or, for the multi-GB workloads, from
torch's seeded generator directly in device memory (make_tensors_device), and
the oracle then reads the slices it needs back to the host.

Workload recipe (the paper's training corpus and trained weights are not
available; these synthetic draws stand in for the skewed per-GPU token
distributions it describes in its Section 3):

* routing, fixed draw order: expert loads -> slot shuffle -> gate logits;
  then X -> W1 -> W2 -> dY.
* ``softmax_topk`` routing (the tiny fp32 case): router logits ~ N(0,1)[T,E],
  p = softmax, top-k by descending p (ties -> lower expert id), gates are the
  chosen p renormalised to sum to 1.
* load-shaped routing (all bf16 cases): a probability vector over experts is
  turned into exact integer slot counts summing to N = T*k by largest
  remainder (ties -> lower expert id); the multiset of expert ids is shuffled
  and reshaped to [T, k] (one token may send two slots to one expert), and the
  gates are softmax(N(0,1)[T,k]) per token.
* tensors: X, dY ~ N(0,1); weights ~ N(0, 0.02) for bf16 cases and
  N(0, 1/h) / N(0, 1/F) for the fp32 case.  bf16 cases round every tensor to
  bf16 (round-to-nearest-even) and keep it in float32 storage, so the values
  are exactly representable in bf16.

Layouts: idx int32 [T,k]; gates float32 [T,k]; X, dY [T,h]; W1 [E,2F,h]
(rows 0..F-1 feed the SiLU gate, rows F..2F-1 the linear "up" half);
W2 [E,h,F].
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int          # received tokens on this GPU
    h: int          # hidden size
    F: int          # expert FFN (intermediate) size, g_e in the paper
    E: int          # local experts
    k: int          # top-k slots per token
    dtype: str      # "bf16" or "f32"
    routing: str    # "softmax_topk" | "dirichlet" | "zipf" | "hot"
    alpha: float = 1.0          # Dirichlet concentration
    zipf_s: float = 1.2         # Zipf exponent
    hot_frac: float = 0.0       # share of slots on the hottest expert ("hot")
    chunks: Tuple[int, ...] = (1,)
    budget_bytes: Optional[int] = None   # activation budget handed to the planner
    bins: Tuple[int, ...] = (1, 2, 4, 8)

    @property
    def N(self) -> int:
        return self.T * self.k

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads the layer is measured and checked on.
WORKLOADS: Dict[int, Workload] = {
    1: Workload("tiny-f32", T=256, h=64, F=128, E=4, k=2, dtype="f32",
                routing="softmax_topk", chunks=(1, 2, 4)),
    2: Workload("balanced-dirichlet5", T=8192, h=2048, F=1408, E=16, k=4,
                dtype="bf16", routing="dirichlet", alpha=5.0, chunks=(1, 2, 4)),
    3: Workload("skewed-zipf1.2-dense-ffn", T=16384, h=4096, F=14336, E=8, k=2,
                dtype="bf16", routing="zipf", zipf_s=1.2, chunks=(1, 2, 4, 8)),
    4: Workload("fine-grained-32of256", T=8192, h=7168, F=2048, E=32, k=8,
                dtype="bf16", routing="hot", hot_frac=8.0 / 32.0, alpha=1.0,
                chunks=(1, 2, 4, 8), budget_bytes=10**9),
    # Budget sweep at the per-GPU worst case of the paper's own setup
    # (e*s*t_k = 32*4096*8 slots); one expert takes half of all slots.
    5: Workload("budget-sweep-hot50", T=131072, h=7168, F=2048, E=32, k=8,
                dtype="bf16", routing="hot", hot_frac=0.5, alpha=1.0,
                chunks=(1, 2, 4, 8, 16), bins=(1, 2, 4, 8, 16)),
}

BUDGET_SWEEP_GB = (4, 8, 16, 32, 64)


def largest_remainder(p: np.ndarray, total: int) -> np.ndarray:
    """Integer counts summing to ``total`` proportional to ``p``.

    Floors first, then hands the leftover units to the largest fractional
    parts; ties go to the lower index (stable sort on the negated remainder).
    """
    p = np.asarray(p, dtype=np.float64)
    p = p / p.sum()
    raw = p * total
    base = np.floor(raw).astype(np.int64)
    left = int(total - base.sum())
    order = np.argsort(-(raw - base), kind="stable")
    base[order[:left]] += 1
    return base


def expert_probabilities(w: Workload, rng: np.random.Generator) -> np.ndarray:
    E = w.E
    if w.routing == "dirichlet":
        return rng.dirichlet(np.full(E, w.alpha))
    if w.routing == "zipf":
        ranks = np.arange(1, E + 1, dtype=np.float64)
        pr = ranks ** (-w.zipf_s)
        pr /= pr.sum()
        perm = rng.permutation(E)          # rank r -> expert perm[r]
        p = np.empty(E)
        p[perm] = pr
        return p
    if w.routing == "hot":
        hot = int(rng.integers(E))
        rest = rng.dirichlet(np.full(E - 1, w.alpha)) if E > 1 else np.zeros(0)
        p = np.empty(E)
        p[hot] = w.hot_frac
        others = [e for e in range(E) if e != hot]
        p[others] = rest * (1.0 - w.hot_frac)
        return p
    raise ValueError(f"unknown load-shaped routing {w.routing!r}")


def make_routing(w: Workload, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Return (idx int32 [T,k], gates float32 [T,k])."""
    rng = np.random.default_rng(seed)
    T, E, k = w.T, w.E, w.k
    if w.routing == "softmax_topk":
        logits = rng.standard_normal((T, E))
        z = logits - logits.max(axis=1, keepdims=True)
        p = np.exp(z)
        p /= p.sum(axis=1, keepdims=True)
        idx = np.argsort(-p, axis=1, kind="stable")[:, :k]
        g = np.take_along_axis(p, idx, axis=1)
        g = g / g.sum(axis=1, keepdims=True)
        return idx.astype(np.int32), g.astype(np.float32)
    p = expert_probabilities(w, rng)
    counts = largest_remainder(p, w.N)
    flat = np.repeat(np.arange(E, dtype=np.int32), counts)
    rng.shuffle(flat)
    idx = flat.reshape(T, k)
    gl = rng.standard_normal((T, k))
    gl = np.exp(gl - gl.max(axis=1, keepdims=True))
    g = gl / gl.sum(axis=1, keepdims=True)
    return idx.astype(np.int32), g.astype(np.float32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    r = ((u + bias) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def _normal(rng: np.random.Generator, shape, std: float, bf16: bool) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return round_to_bf16(x) if bf16 else x


def make_tensors(w: Workload, seed: int, with_dy: bool = True) -> Dict[str, np.ndarray]:
    """Draw X, W1, W2 (and dY) for workload ``w``; float32 storage."""
    rng = np.random.default_rng([seed, 1])
    bf16 = w.dtype == "bf16"
    if bf16:
        s1 = s2 = 0.02
    else:
        s1, s2 = w.h ** -0.5, w.F ** -0.5
    out = {
        "X": _normal(rng, (w.T, w.h), 1.0, bf16),
        "W1": _normal(rng, (w.E, 2 * w.F, w.h), s1, bf16),
        "W2": _normal(rng, (w.E, w.h, w.F), s2, bf16),
    }
    if with_dy:
        out["dY"] = _normal(rng, (w.T, w.h), 1.0, bf16)
    return out


def make_case(w: Workload, seed: int, with_dy: bool = True) -> Dict[str, np.ndarray]:
    idx, gates = make_routing(w, seed)
    case = make_tensors(w, seed, with_dy=with_dy)
    case["idx"] = idx
    case["gates"] = gates
    return case


def scaled(w: Workload, **kw) -> Workload:
    """A copy of ``w`` with other sizes (same routing recipe), for parity runs."""
    return w.with_(**kw)


def make_tensors_device(w: Workload, seed: int, device, with_dy: bool = True):
    """Draw X, W1, W2 (and dY) directly in device memory with torch's seeded
    generator (for the multi-GB workloads; same distributions as
    make_tensors, bf16 by round-to-nearest-even).  Returns torch tensors in
    the workload's storage dtype."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) * 1000003 + 17)
    bf16 = w.dtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    s1, s2 = (0.02, 0.02) if bf16 else (w.h ** -0.5, w.F ** -0.5)

    def normal(shape, std):
        t = torch.empty(shape, dtype=dt, device=device)
        # fill in slices to bound the float32 staging buffer
        flat = t.view(-1)
        step = 1 << 26
        for i in range(0, flat.numel(), step):
            j = min(flat.numel(), i + step)
            x = torch.randn(j - i, generator=gen, device=device, dtype=torch.float32)
            if std != 1.0:
                x.mul_(std)
            flat[i:j].copy_(x)
        return t

    out = {"X": normal((w.T, w.h), 1.0), "W1": normal((w.E, 2 * w.F, w.h), s1),
           "W2": normal((w.E, w.h, w.F), s2)}
    if with_dy:
        out["dY"] = normal((w.T, w.h), 1.0)
    return out
