"""GPU parity of expert-ordered chunks (launch option chunk_order =
MEMFINE_CHUNK_EXPERTS): chunk c holds rows [c N / C, (c + 1) N / C) of the
layer's slots grouped by expert, so Y and dX are sums over chunks.

* against the fp64 oracle, per tensor max|got - ref| / max|ref| <= 2e-2
  (bf16) and <= 1e-4 (fp32), over chunk counts that split experts across
  chunks, with dropped ids, cold experts and accumulation into dW;
* dgates bit-identical to the token order (each row's products do not depend
  on how rows are grouped), dW equal to it up to the order of the fp32 sums;
* the working memory the layer holds at once equals its declared workspace.
Every output starts as NaN, so an element no chunk writes fails the check.
"""
import gc

import numpy as np
import pytest

import moe_workloads as mw
from gpu_harness import (TOL, device_case, host, log, relerr, run_bwd, run_fwd, shape_of,
                         torch)
from oracle import moe as om

pytestmark = pytest.mark.gpu

W = mw.WORKLOADS
CASES = {
    "cfg1-f32": (W[1], (1, 2, 3, 7)),
    "cfg2-like": (mw.scaled(W[2], T=768, h=256, F=192), (1, 2, 5)),
    "cfg3-like": (mw.scaled(W[3], T=1024, h=384, F=448), (1, 3, 8)),
    "cfg4-like": (mw.scaled(W[4], T=256, h=448, F=128), (2, 4, 256)),
    "cfg5-like": (mw.scaled(W[5], T=512, h=128, F=192), (1, 8, 16)),
    # the ABI's largest expert count: one wave per expert can no longer hold
    # the table, most experts have no row and chunks hold hundreds of them
    "many-1024": (mw.Workload("many-1024", T=640, h=128, F=192, E=1024, k=3, dtype="bf16",
                              routing="dirichlet"), (1, 3)),
}


@pytest.fixture(scope="module")
def mf():
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_21431_amd as m
    m.lib()
    return m


@pytest.fixture
def experts_order(mf):
    mf.memfine_set_launch_options(chunk_order=mf.CHUNK_EXPERTS)
    yield
    mf.memfine_set_launch_options()


_cache = {}


def case_of(name):
    if name not in _cache:
        w = CASES[name][0]
        _cache[name] = (w, mw.make_case(w, 301 + list(CASES).index(name)))
    return _cache[name]


def oracle(case, idx=None, gates=None):
    idx = case["idx"] if idx is None else idx
    gates = case["gates"] if gates is None else gates
    Y = om.moe_fwd(case["X"], idx, gates, case["W1"], case["W2"])
    R = om.moe_bwd(case["X"], idx, gates, case["W1"], case["W2"], case["dY"])
    return Y, R


@pytest.mark.parametrize("name,C", [(n, c) for n in CASES for c in CASES[n][1]])
def test_expert_order_parity(mf, experts_order, name, C):
    w, case = case_of(name)
    dev = device_case(w, case)
    log(f"expert order {name} C={C}")
    Y = host(run_fwd(w, dev, C))
    B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
    Y_ref, R = oracle(case)
    errs = {"Y": relerr(Y, Y_ref)}
    for key in ("dX", "dgates", "dW1", "dW2"):
        errs[key] = relerr(B[key], R[key])
    log(f"  {name} C={C} rel errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= TOL[w.dtype], (key, e)


@pytest.mark.parametrize("name", ["cfg2-like", "cfg4-like"])
def test_expert_order_against_token_order(mf, name):
    """dgates bit-identical to the token order at every C; dW equal up to the
    order of the fp32 sums; Y and dX within one rounding per chunk."""
    w, case = case_of(name)
    dev = device_case(w, case)
    mf.memfine_set_launch_options()
    Y0 = host(run_fwd(w, dev, 1))
    B0 = {k: host(v) for k, v in run_bwd(w, dev, 1).items()}
    try:
        mf.memfine_set_launch_options(chunk_order=mf.CHUNK_EXPERTS)
        for C in (1, 3, 4):
            log(f"expert vs token order {name} C={C}")
            Y = host(run_fwd(w, dev, C))
            B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
            assert np.array_equal(B["dgates"], B0["dgates"]), C
            for key in ("dW1", "dW2"):
                assert relerr(B[key], B0[key]) < 1e-5, (C, key)
            if C == 1:   # one chunk: every token's sum written once, as in the token order
                assert np.array_equal(Y, Y0) and np.array_equal(B["dX"], B0["dX"])
            assert relerr(Y, Y0) < 2.0 ** -6 and relerr(B["dX"], B0["dX"]) < 2.0 ** -6, C
    finally:
        mf.memfine_set_launch_options()


def test_expert_order_dropped_ids_cold_experts_accumulate(mf, experts_order):
    """Slots with ids outside [0, E) (a token may lose every slot: its Y and
    dX rows are 0, written by the first chunk), experts without rows (dW 0
    when overwriting, untouched when accumulating), and accumulation into
    dW across split experts."""
    t = torch()
    w, case = case_of("cfg2-like")
    idx = case["idx"].copy()
    rng = np.random.default_rng(9)
    drop = rng.random(idx.shape) < 0.1
    drop[5, :] = True                      # token 5 loses every slot
    idx[drop] = -1
    idx[idx == 3] = 0                      # expert 3 receives nothing
    ref_idx = np.where(drop, 0, idx).astype(np.int32)
    ref_g = np.where(drop, 0.0, case["gates"]).astype(np.float32)
    dev = device_case(w, dict(case, idx=idx))
    Y_ref, R = oracle(case, ref_idx, ref_g)
    R["dgates"] = np.where(drop, 0.0, R["dgates"])
    for C in (2, 7):
        log(f"expert order dropped / cold C={C}")
        Y = host(run_fwd(w, dev, C))
        B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
        assert relerr(Y, Y_ref) <= TOL["bf16"]
        assert np.all(Y[5] == 0.0) and np.all(B["dX"][5] == 0.0)
        for key in ("dX", "dgates", "dW1", "dW2"):
            assert relerr(B[key], R[key]) <= TOL["bf16"], (C, key)
        assert np.all(B["dgates"][drop] == 0.0)
        assert np.all(B["dW1"][3] == 0.0) and np.all(B["dW2"][3] == 0.0)
        base1 = t.randn((w.E, 2 * w.F, w.h), device="cuda")
        base2 = t.randn((w.E, w.h, w.F), device="cuda")
        dW = (base1.clone(), base2.clone())
        run_bwd(w, dev, C, dW=dW, accumulate=True)
        assert relerr(host(dW[0] - base1), B["dW1"]) < 1e-5
        assert relerr(host(dW[1] - base2), B["dW2"]) < 1e-5
        assert t.equal(dW[0][3], base1[3]) and t.equal(dW[1][3], base2[3])


def test_expert_order_allocator_peak(mf, experts_order):
    """The working memory held at once (the allocator hook's high-water mark
    and torch's statistics) equals the declared expert-order workspace: the
    layer's routing tables plus one chunk's intermediates."""
    t = torch()
    w, case = case_of("cfg4-like")
    dev = device_case(w, case)
    s = shape_of(w)
    dX = t.empty((w.T, w.h), dtype=t.bfloat16, device="cuda")
    dg = t.empty((w.T, w.k), device="cuda")
    dW1 = t.empty((w.E, 2 * w.F, w.h), device="cuda")
    dW2 = t.empty((w.E, w.h, w.F), device="cuda")
    for C in (1, 3, 8):
        alloc = mf.TorchAllocator()
        t.cuda.synchronize()
        t.cuda.empty_cache()
        gc.collect()                 # no frees of earlier garbage inside the window
        t.cuda.reset_peak_memory_stats()
        base = t.cuda.memory_allocated()
        log(f"expert order allocator peak C={C}")
        mf.memfine_moe_bwd(s, C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"],
                           dev["dY"], dX, dW1, dW2, dg, allocator=alloc)
        t.cuda.synchronize()
        peak = t.cuda.max_memory_allocated() - base
        pred = mf.memfine_workspace_bytes(s, C, mf.PASS_BWD)
        assert alloc.live == {} and alloc.live_bytes == 0
        assert alloc.high_water == pred, (C, alloc.high_water, pred)
        assert pred <= peak <= pred + (4 << 20), (C, peak, pred)


def test_expert_order_launch_options_bitwise(mf):
    """Expert-ordered chunks under the other launch options (paired FC1
    backward launch, side streams, 128 x 128 tiles): the same results, bit
    for bit (each output element keeps its order of fp32 sums)."""
    w, case = case_of("cfg4-like")
    dev = device_case(w, case)
    res = {}
    try:
        for name, kw in (("default", {}), ("pair", dict(pair=True)), ("streams", dict(streams=True)),
                         ("tile128", dict(tile=mf.TILE_128))):
            mf.memfine_set_launch_options(chunk_order=mf.CHUNK_EXPERTS, **kw)
            log(f"expert order, launch options {name}")
            Y = host(run_fwd(w, dev, 3))
            B = {k: host(v) for k, v in run_bwd(w, dev, 3).items()}
            res[name] = (Y, B)
    finally:
        mf.memfine_set_launch_options()
    Y0, B0 = res["default"]
    for name, (Y, B) in res.items():
        assert np.array_equal(Y, Y0), name
        for key in B0:
            assert np.array_equal(B[key], B0[key]), (name, key)

