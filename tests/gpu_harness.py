"""Helpers for the GPU parity tests: move a seeded case to the device, run the
layer through the C ABI, and compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

import moe_workloads as mw

TOL = {"bf16": 2e-2, "f32": 1e-4}


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch():
    import torch as _t
    return _t


def relerr(got, ref) -> float:
    """max |got - ref| / max |ref| over one output tensor."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if not np.all(np.isfinite(got)):
        return float("inf")
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(got - ref)) if ref.size else 0.0
    return float(num / den) if den > 0 else float(num)


def shape_of(w: mw.Workload):
    import paper_2511_21431_amd as mf
    return mf.make_shape(w.T, w.h, w.F, w.E, w.k, mf.BF16 if w.dtype == "bf16" else mf.F32)


def device_case(w: mw.Workload, case) -> dict:
    """numpy case -> device tensors in the layer's storage dtype."""
    t = torch()
    dt = t.bfloat16 if w.dtype == "bf16" else t.float32
    out = {}
    for key in ("X", "W1", "W2", "dY"):
        if key in case:
            out[key] = t.from_numpy(np.ascontiguousarray(case[key])).to("cuda").to(dt).contiguous()
    out["idx"] = t.from_numpy(np.ascontiguousarray(case["idx"], dtype=np.int32)).to("cuda")
    out["gates"] = t.from_numpy(np.ascontiguousarray(case["gates"], dtype=np.float32)).to("cuda")
    return out


def nan_like(shape, dtype):
    t = torch()
    return t.full(shape, float("nan"), dtype=dtype, device="cuda")


def run_fwd(w, dev, C, allocator=None):
    import paper_2511_21431_amd as mf
    t = torch()
    dt = t.bfloat16 if w.dtype == "bf16" else t.float32
    Y = nan_like((w.T, w.h), dt)
    mf.memfine_moe_fwd(shape_of(w), C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"], Y,
                       allocator=allocator)
    return Y


def run_bwd(w, dev, C, allocator=None, dW=None, accumulate=False):
    import paper_2511_21431_amd as mf
    t = torch()
    dt = t.bfloat16 if w.dtype == "bf16" else t.float32
    dX = nan_like((w.T, w.h), dt)
    dg = nan_like((w.T, w.k), t.float32)
    if dW is None:
        dW1 = nan_like((w.E, 2 * w.F, w.h), t.float32)
        dW2 = nan_like((w.E, w.h, w.F), t.float32)
    else:
        dW1, dW2 = dW
    mf.memfine_moe_bwd(shape_of(w), C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"],
                       dev["dY"], dX, dW1, dW2, dg, accumulate_dW=accumulate, allocator=allocator)
    return {"dX": dX, "dgates": dg, "dW1": dW1, "dW2": dW2}


def host(x) -> np.ndarray:
    return x.float().cpu().numpy()
