"""GPU parity: the HIP layer, called through the C ABI, against the fp64
oracle on the same seeded inputs.

* counts and the dispatch permutation: bit-exact;
* outputs and gradients: max|got - ref| / max|ref| <= 2e-2 (bf16 inputs,
  fp32 accumulation) and <= 1e-4 (fp32 path), per tensor;
* Y, dX and dgates bit-identical for every chunk count (each row's dot
  products do not depend on how rows are grouped into tiles or chunks), and
  the whole layer bitwise deterministic run to run;
* full-size workloads in the launch configuration the benchmark times, on
  sampled tokens and sampled weight-gradient columns the oracle computes one
  by one, and on 512 tokens plus whole experts' weight gradients.
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
SMALL = {
    "cfg1-f32": W[1],
    "cfg2-like": mw.scaled(W[2], T=768, h=256, F=192),
    "cfg3-like": mw.scaled(W[3], T=1024, h=384, F=448),
    "cfg4-like": mw.scaled(W[4], T=256, h=448, F=128),
    "cfg5-like": mw.scaled(W[5], T=512, h=128, F=192),
}


@pytest.fixture(scope="module")
def mf():
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_21431_amd as m
    m.lib()
    return m


_cache = {}


def small_case(name, seed=None):
    key = (name, seed)
    if key not in _cache:
        w = SMALL[name]
        s = seed if seed is not None else 101 + list(SMALL).index(name)
        _cache[key] = (w, mw.make_case(w, s))
    return _cache[key]


# ------------------------------------------------------------------ dispatch
@pytest.mark.parametrize("name", list(SMALL))
def test_count_matches_oracle(mf, name):
    w, case = small_case(name)
    t = torch()
    log(f"count {name}")
    idx = t.from_numpy(case["idx"]).cuda()
    work = t.zeros(w.E + 1, dtype=t.int32, device="cuda")
    got = mf.memfine_count(shape_of(w), idx, work)
    assert got.tolist() == om.expert_counts(case["idx"], w.E).tolist()


def test_count_rejects_bad_ids(mf):
    t = torch()
    w = SMALL["cfg2-like"]
    idx = t.zeros((w.T, w.k), dtype=t.int32, device="cuda")
    idx[5, 1] = w.E
    idx[7, 0] = -3
    work = t.zeros(w.E + 1, dtype=t.int32, device="cuda")
    with pytest.raises(mf.MemfineError) as ei:
        mf.memfine_count(shape_of(w), idx, work)
    assert ei.value.code == -1
    assert int(work[w.E]) == 2


def _dispatch_check(mf, w, idx_np, t0, t1):
    t = torch()
    n = (t1 - t0) * w.k
    idx = t.from_numpy(np.ascontiguousarray(idx_np, dtype=np.int32)).cuda()
    counts = t.full((w.E,), -7, dtype=t.int32, device="cuda")
    offsets = t.full((w.E + 1,), -7, dtype=t.int32, device="cuda")
    ss = t.full((n,), -7, dtype=t.int32, device="cuda")
    rs = t.full((n,), -7, dtype=t.int32, device="cuda")
    mf.memfine_dispatch(shape_of(w), idx, t0, t1, counts, offsets, ss, rs)
    ref = om.dispatch(idx_np, t0, t1, w.E)
    assert counts.cpu().numpy().tolist() == ref["counts"].tolist()
    assert offsets.cpu().numpy().tolist() == ref["offsets"].tolist()
    assert ss.cpu().numpy().tolist() == ref["sorted_slot"].tolist()
    assert rs.cpu().numpy().tolist() == ref["row_of_slot"].tolist()


@pytest.mark.parametrize("name", list(SMALL))
def test_dispatch_bit_exact_every_chunk(mf, name):
    w, case = small_case(name)
    for C in (1, 2, 3, 4, 8):
        for t0, t1 in om.chunk_ranges(w.T, C):
            log(f"dispatch {name} C={C} [{t0},{t1})")
            _dispatch_check(mf, w, case["idx"], t0, t1)


@pytest.mark.parametrize("E,k,T", [(1, 1, 1), (1, 3, 5000), (1024, 8, 3000), (1000, 1, 777),
                                   (7, 2, 0), (64, 6, 4096)])
def test_dispatch_edge_shapes(mf, E, k, T):
    w = mw.Workload("edge", T=T, h=64, F=64, E=E, k=k, dtype="bf16", routing="dirichlet")
    rng = np.random.default_rng(E * 7 + k)
    idx = rng.integers(0, E, size=(T, k)).astype(np.int32)
    if E > 4 and T > 0:
        idx[: T // 2] = E - 1            # a hot expert and long runs of equal ids
    log(f"dispatch edge E={E} k={k} T={T}")
    _dispatch_check(mf, w, idx, 0, T)
    if T > 3:
        _dispatch_check(mf, w, idx, 1, T - 2)


def test_dispatch_full_size_config4(mf):
    w = W[4]
    idx, _ = mw.make_routing(w, 4)
    for C in (1, 4, 8):
        for t0, t1 in om.chunk_ranges(w.T, C)[:2]:
            log(f"dispatch cfg4 C={C} [{t0},{t1})")
            _dispatch_check(mf, w, idx, t0, t1)


# ------------------------------------------------------------- layer parity
CHUNKS = {"cfg1-f32": (1, 2, 4), "cfg2-like": (1, 2, 4), "cfg3-like": (1, 3, 8),
          "cfg4-like": (1, 4), "cfg5-like": (1, 16)}


@pytest.mark.parametrize("name,C", [(n, c) for n in SMALL for c in CHUNKS[n]])
def test_layer_parity(mf, name, C):
    w, case = small_case(name)
    tol = TOL[w.dtype]
    dev = device_case(w, case)
    log(f"fwd {name} C={C}")
    Y = run_fwd(w, dev, C)
    log(f"bwd {name} C={C}")
    B = run_bwd(w, dev, C)
    torch().cuda.synchronize()
    Y_ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
    R = om.moe_bwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], case["dY"], C)
    errs = {"Y": relerr(host(Y), Y_ref)}
    for key in ("dX", "dgates", "dW1", "dW2"):
        errs[key] = relerr(host(B[key]), R[key])
    log(f"  {name} C={C} rel errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= tol, (key, e)


@pytest.mark.parametrize("E,C", [(80, 1), (80, 3), (200, 2), (1024, 2)])
def test_layer_parity_many_experts(mf, E, C):
    """More experts than one wave's lanes: the GEMMs locate their row tiles
    by walking the experts instead of a one-wave table (up to the ABI's
    1024 experts, most of them with no row)."""
    w = mw.Workload(f"many-{E}", T=640, h=128, F=192, E=E, k=3, dtype="bf16", routing="dirichlet")
    case = mw.make_case(w, 17 + E)
    dev = device_case(w, case)
    log(f"many experts E={E} C={C}")
    Y = run_fwd(w, dev, C)
    B = run_bwd(w, dev, C)
    torch().cuda.synchronize()
    Y_ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
    R = om.moe_bwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], case["dY"], C)
    assert relerr(host(Y), Y_ref) <= TOL["bf16"]
    for key in ("dX", "dgates", "dW1", "dW2"):
        assert relerr(host(B[key]), R[key]) <= TOL["bf16"], key


@pytest.mark.parametrize("h,k,dtype,C", [(64, 12, "bf16", 2), (128, 12, "bf16", 1),
                                         (64, 20, "f32", 2), (128, 9, "bf16", 3)])
def test_layer_parity_large_k(mf, h, k, dtype, C):
    """More slots per token than 16-byte vectors per row (k > h / 8 in bf16,
    h / 4 in fp32): the gate-gradient sums run as their own kernel instead of
    inside the unpermute kernel; and k > 8 takes the combine's slot groups
    twice."""
    w = mw.Workload(f"k{k}-h{h}", T=300, h=h, F=128, E=24, k=k, dtype=dtype, routing="dirichlet")
    case = mw.make_case(w, 7 + k + h)
    dev = device_case(w, case)
    log(f"large k: h={h} k={k} {dtype} C={C}")
    Y = run_fwd(w, dev, C)
    B = run_bwd(w, dev, C)
    torch().cuda.synchronize()
    Y_ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
    R = om.moe_bwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], case["dY"], C)
    assert relerr(host(Y), Y_ref) <= TOL[dtype]
    for key in ("dX", "dgates", "dW1", "dW2"):
        assert relerr(host(B[key]), R[key]) <= TOL[dtype], key


@pytest.mark.parametrize("name", ["cfg1-f32", "cfg3-like", "cfg4-like"])
def test_chunk_invariance_and_determinism(mf, name):
    w, case = small_case(name)
    dev = device_case(w, case)
    ref_Y = host(run_fwd(w, dev, 1))
    ref_B = {k: host(v) for k, v in run_bwd(w, dev, 1).items()}
    for C in (1, 2, 5, w.T, w.T + 3):
        log(f"invariance {name} C={C}")
        Y = host(run_fwd(w, dev, C))
        B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
        assert np.array_equal(Y, ref_Y), C
        assert np.array_equal(B["dX"], ref_B["dX"]), C
        assert np.array_equal(B["dgates"], ref_B["dgates"]), C
        for key in ("dW1", "dW2"):
            if C == 1:
                assert np.array_equal(B[key], ref_B[key])      # run-to-run determinism
            else:
                assert relerr(B[key], ref_B[key]) < 1e-5, (C, key)


def test_side_stream_backward_bitwise(mf):
    """The optional side-stream schedule of the backward (weight gradients
    beside the FC1 dgrad) gives bit-identical results to the serial one."""
    w, case = small_case("cfg2-like")
    dev = device_case(w, case)
    for C in (1, 3):
        log(f"side streams C={C}")
        mf.memfine_set_launch_options()
        ref = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
        try:
            mf.memfine_set_launch_options(streams=True)
            got = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
        finally:
            mf.memfine_set_launch_options()
        for key in ref:
            assert np.array_equal(got[key], ref[key]), (C, key)


def test_internal_workspace_per_stream(mf):
    """Calls without an allocator take their chunk buffers from a cached
    block per (device, stream).  Work enqueued on two streams at once, and a
    call with larger chunks after one with smaller chunks on the same stream
    (the stream's block grows), give bit-identical results to the same calls
    run one by one on the default stream."""
    t = torch()
    wa, ca = small_case("cfg2-like")
    wb, cb = small_case("cfg4-like")
    da, db = device_case(wa, ca), device_case(wb, cb)
    ref = {}
    for name, w, d in (("a", wa, da), ("b", wb, db)):
        ref[name] = {"Y": host(run_fwd(w, d, 3)), **{k: host(v) for k, v in run_bwd(w, d, 3).items()}}
    t.cuda.synchronize()
    s1, s2 = t.cuda.Stream(), t.cuda.Stream()
    got = {}
    with t.cuda.stream(s1):
        run_fwd(wa, da, 7)                   # smaller chunks first: the block grows below
    for rep in range(2):
        log(f"two streams, repetition {rep}")
        with t.cuda.stream(s1):
            got["a"] = {"Y": run_fwd(wa, da, 3), **run_bwd(wa, da, 3)}
        with t.cuda.stream(s2):
            got["b"] = {"Y": run_fwd(wb, db, 3), **run_bwd(wb, db, 3)}
        t.cuda.synchronize()
        for name in ("a", "b"):
            for key, v in got[name].items():
                assert np.array_equal(host(v), ref[name][key]), (rep, name, key)


def test_workspace_held_and_trim(mf):
    """The cached workspace block of a stream (calls without an allocator)
    grows to the largest chunk asked for, is reported by
    memfine_workspace_held, and memfine_workspace_trim shrinks it to the
    workspace of the chunk count in use: a C = 1 call, then a C = 4 call,
    then a trim to the C = 4 workspace leaves exactly that block, and later
    C = 4 calls run in it with bit-identical results (Section 4.1: the peak
    is the largest chunk's)."""
    t = torch()
    w, case = small_case("cfg4-like")
    dev = device_case(w, case)
    s = shape_of(w)
    ws1 = mf.memfine_workspace_bytes(s, 1, mf.PASS_BWD)
    ws4 = mf.memfine_workspace_bytes(s, 4, mf.PASS_BWD)
    st = t.cuda.Stream()
    with t.cuda.stream(st):
        log("workspace held / trim")
        mf.memfine_workspace_trim(0)
        assert mf.memfine_workspace_held() == 0
        mf.memfine_pool_high_water(reset=True)
        run_bwd(w, dev, 1)
        assert mf.memfine_workspace_held() == ws1
        first4 = {k: host(v) for k, v in run_bwd(w, dev, 4).items()}
        assert mf.memfine_workspace_held() == ws1          # kept, not shrunk by itself
        mf.memfine_workspace_trim(ws4)
        assert mf.memfine_workspace_held() == ws4
        again4 = {k: host(v) for k, v in run_bwd(w, dev, 4).items()}
        assert mf.memfine_workspace_held() == ws4
        for key in first4:
            assert np.array_equal(first4[key], again4[key]), key
        mf.memfine_workspace_trim(ws4 + 1)                  # larger than held: no change
        assert mf.memfine_workspace_held() == ws4
        mf.memfine_workspace_trim(0)
        assert mf.memfine_workspace_held() == 0
    st.synchronize()
    assert mf.memfine_pool_high_water() >= ws1


def test_accumulate_dW(mf):
    w, case = small_case("cfg2-like")
    t = torch()
    dev = device_case(w, case)
    base1 = t.randn((w.E, 2 * w.F, w.h), device="cuda")
    base2 = t.randn((w.E, w.h, w.F), device="cuda")
    dW = (base1.clone(), base2.clone())
    log("accumulate dW")
    run_bwd(w, dev, 3, dW=dW, accumulate=True)
    plain = run_bwd(w, dev, 3)
    assert relerr(host(dW[0] - base1), host(plain["dW1"])) < 1e-5
    assert relerr(host(dW[1] - base2), host(plain["dW2"])) < 1e-5


def test_degenerate_cases(mf):
    t = torch()
    # one token, one slot, one expert
    w = mw.Workload("one", T=1, h=64, F=64, E=1, k=1, dtype="f32", routing="dirichlet")
    case = mw.make_case(w, 3)
    dev = device_case(w, case)
    log("degenerate T=1")
    Y = host(run_fwd(w, dev, 4))
    B = run_bwd(w, dev, 4)
    assert relerr(Y, om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"])) < 1e-4
    R = om.moe_bwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], case["dY"])
    for key in ("dX", "dgates", "dW1", "dW2"):
        assert relerr(host(B[key]), R[key]) < 1e-4
    # experts that receive nothing get zero weight gradients
    w = mw.Workload("cold", T=64, h=128, F=64, E=6, k=2, dtype="bf16", routing="dirichlet")
    case = mw.make_case(w, 4)
    case["idx"][:] = np.where(case["idx"] % 2 == 0, 0, 3).astype(np.int32)
    dev = device_case(w, case)
    log("degenerate cold experts")
    B = run_bwd(w, dev, 2)
    dW1 = host(B["dW1"])
    for e in (1, 2, 4, 5):
        assert np.all(dW1[e] == 0.0)
    # no tokens at all
    w0 = mw.Workload("empty", T=0, h=64, F=64, E=3, k=2, dtype="bf16", routing="dirichlet")
    import paper_2511_21431_amd as m
    X = t.zeros((0, 64), dtype=t.bfloat16, device="cuda")
    idx = t.zeros((0, 2), dtype=t.int32, device="cuda")
    g = t.zeros((0, 2), dtype=t.float32, device="cuda")
    W1 = t.ones((3, 128, 64), dtype=t.bfloat16, device="cuda")
    W2 = t.ones((3, 64, 64), dtype=t.bfloat16, device="cuda")
    dW1 = t.full((3, 128, 64), 5.0, device="cuda")
    dW2 = t.full((3, 64, 64), 5.0, device="cuda")
    m.memfine_moe_fwd(shape_of(w0), 2, X, idx, g, W1, W2, X)
    m.memfine_moe_bwd(shape_of(w0), 2, X, idx, g, W1, W2, X, X, dW1, dW2, g)
    assert float(dW1.abs().max()) == 0.0 and float(dW2.abs().max()) == 0.0


def test_out_of_range_ids_are_dropped(mf):
    """A slot whose id lies outside [0, E) contributes nothing.  Reference: the
    oracle with that slot sent to expert 0 at gate 0 (a zero gate removes the
    slot from Y, dX and dW), and dgates 0 at the dropped slots."""
    w, case = small_case("cfg2-like")
    bad = case["idx"].copy()
    rng = np.random.default_rng(7)
    drop = rng.random(bad.shape) < 0.1
    bad[drop] = np.where(rng.random(drop.sum()) < 0.5, -1, w.E + 5).astype(np.int32)
    ref_idx = np.where(drop, 0, case["idx"]).astype(np.int32)
    ref_g = np.where(drop, 0.0, case["gates"]).astype(np.float32)
    dev = device_case(w, dict(case, idx=bad))
    for C in (1, 3):
        log(f"dropped ids C={C}")
        Y = host(run_fwd(w, dev, C))
        B = run_bwd(w, dev, C)
        Y_ref = om.moe_fwd(case["X"], ref_idx, ref_g, case["W1"], case["W2"], C)
        R = om.moe_bwd(case["X"], ref_idx, ref_g, case["W1"], case["W2"], case["dY"], C)
        R["dgates"] = np.where(drop, 0.0, R["dgates"])
        assert relerr(Y, Y_ref) <= TOL[w.dtype]
        for key in ("dX", "dgates", "dW1", "dW2"):
            assert relerr(host(B[key]), R[key]) <= TOL[w.dtype], key
        assert np.all(host(B["dgates"])[drop] == 0.0)


def test_split_tail_parity(mf):
    """A shape whose grids run on 256 x 256 tiles with a short last round
    (FC1: 68 m-tiles x 8 = 544 tiles on 256 CUs; FC2 dgrad 272), which the
    row-grouped GEMMs run as quarter tiles: checked in full against the oracle,
    and Y / dX / dgates bit-identical between C = 1 and C = 2 (whose grids
    split differently)."""
    w = mw.scaled(W[2], T=4096, h=512, F=1024, E=8)
    case = mw.make_case(w, 211)
    dev = device_case(w, case)
    res = {}
    for C in (1, 2):
        log(f"split tail C={C}")
        Y = host(run_fwd(w, dev, C))
        B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
        res[C] = (Y, B)
        Y_ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
        R = om.moe_bwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], case["dY"], C)
        assert relerr(Y, Y_ref) <= TOL["bf16"]
        for key in ("dX", "dgates", "dW1", "dW2"):
            assert relerr(B[key], R[key]) <= TOL["bf16"], (C, key)
    assert np.array_equal(res[1][0], res[2][0])
    for key in ("dX", "dgates"):
        assert np.array_equal(res[1][1][key], res[2][1][key]), key


def test_allocator_hook_peak_and_oom(mf):
    """The working memory the layer holds at once, measured two ways (the
    allocator hook's own high-water mark, and torch's allocator statistics),
    against the layer's declared per-chunk workspace."""
    t = torch()
    w, case = small_case("cfg4-like")
    dev = device_case(w, case)
    s = shape_of(w)
    dt = t.bfloat16
    dX = t.empty((w.T, w.h), dtype=dt, device="cuda")
    dg = t.empty((w.T, w.k), device="cuda")
    dW1 = t.empty((w.E, 2 * w.F, w.h), device="cuda")
    dW2 = t.empty((w.E, w.h, w.F), device="cuda")
    for C in (1, 2, 4):
        alloc = mf.TorchAllocator()
        t.cuda.synchronize()
        t.cuda.empty_cache()
        gc.collect()                 # no frees of earlier garbage inside the window
        t.cuda.reset_peak_memory_stats()
        base = t.cuda.memory_allocated()
        log(f"allocator peak C={C}")
        mf.memfine_moe_bwd(s, C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"],
                           dev["dY"], dX, dW1, dW2, dg, allocator=alloc)
        t.cuda.synchronize()
        peak = t.cuda.max_memory_allocated() - base
        pred = mf.memfine_workspace_bytes(s, C, mf.PASS_BWD)
        assert alloc.live == {} and alloc.live_bytes == 0
        assert alloc.high_water == pred, (C, alloc.high_water, pred)
        # torch rounds blocks up (at most to the next 2 MiB segment)
        assert pred <= peak <= pred + (2 << 20), (C, peak, pred)
    alloc = mf.TorchAllocator()
    alloc.fail_at = 2                       # second chunk's allocation fails
    with pytest.raises(mf.MemfineError) as ei:
        run_bwd(w, dev, 3, allocator=alloc)
    assert ei.value.code == -4 and alloc.live == {}


# ---------------------------------------------------- full-size, sampled
def test_full_size_workload2_every_output(mf):
    """The benchmark's workload (T=8192, h=2048, F=1408, E=16, top-4, the
    planner's C=2) checked in full against the oracle: every Y, dX and dgates
    entry and every weight-gradient element (about 6 s of oracle time)."""
    t = torch()
    w, C = W[2], 2
    idx, gates = mw.make_routing(w, 2)
    dev = mw.make_tensors_device(w, 2, "cuda")
    dev["idx"] = t.from_numpy(idx).cuda()
    dev["gates"] = t.from_numpy(gates).cuda()
    log("full check cfg2 C=2: fwd + bwd")
    Y = host(run_fwd(w, dev, C))
    B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
    X = dev["X"].double().cpu().numpy()
    W1 = dev["W1"].double().cpu().numpy()
    W2 = dev["W2"].double().cpu().numpy()
    dY = dev["dY"].double().cpu().numpy()
    log("full check cfg2 C=2: oracle")
    Y_ref = om.moe_fwd(X, idx, gates, W1, W2, C)
    R = om.moe_bwd(X, idx, gates, W1, W2, dY, C)
    errs = {"Y": relerr(Y, Y_ref)}
    for key in ("dX", "dgates", "dW1", "dW2"):
        errs[key] = relerr(B[key], R[key])
    log("  cfg2 C=2 full: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= TOL["bf16"], (key, e)


# the benchmark's workload 2 at its planner C and C = 1; workloads 3 and 5 at
# the chunk counts their planner picks at the benchmark budgets (C = 8 for
# both), workload 3 at C = 4, workload 4 at its planner C, and the budget
# sweep's largest chunk count on workload 5's 131072 tokens
FULL = [(2, 2, 0), (2, 1, 0), (3, 4, 0), (3, 8, 0), (4, 4, 0), (5, 8, 0), (5, 16, 0),
        (4, 4, 1), (5, 8, 1)]   # last field: chunk order (1: expert-ordered chunks)


@pytest.mark.parametrize("cfg,C,order", FULL)
def test_full_size_sampled(mf, cfg, C, order):
    mf.memfine_set_launch_options(chunk_order=order)
    try:
        _full_size_sampled(mf, cfg, C)
    finally:
        mf.memfine_set_launch_options()


def _full_size_sampled(mf, cfg, C, w=None):
    t = torch()
    w = W[cfg] if w is None else w
    log(f"full-size cfg{cfg} C={C}: generating inputs")
    idx, gates = mw.make_routing(w, cfg)
    dev = mw.make_tensors_device(w, cfg, "cuda")
    dev["idx"] = t.from_numpy(idx).cuda()
    dev["gates"] = t.from_numpy(gates).cuda()
    log(f"full-size cfg{cfg} C={C}: fwd")
    Y = run_fwd(w, dev, C)
    log(f"full-size cfg{cfg} C={C}: bwd")
    B = run_bwd(w, dev, C)
    t.cuda.synchronize()
    rng = np.random.default_rng(1000 + cfg)
    toks = sorted(set(rng.choice(w.T, size=12, replace=False).tolist()) | {0, w.T - 1})
    X = dev["X"].float().cpu().numpy()
    dY = dev["dY"].float().cpu().numpy()
    counts = np.bincount(idx.reshape(-1), minlength=w.E)
    order = np.argsort(-counts, kind="stable")
    experts = sorted({int(order[0]), int(order[w.E // 2]), int(order[-1])} |
                     {int(e) for e in np.unique(idx[toks])})
    W1 = {e: dev["W1"][e].double().cpu().numpy() for e in experts}
    W2 = {e: dev["W2"][e].double().cpu().numpy() for e in experts}

    class Lazy(dict):           # W1[e] lookups for the token forms
        def __getitem__(self, e):
            return dict.__getitem__(self, int(e))

    W1l, W2l = Lazy(W1), Lazy(W2)
    W1l.shape = (w.E, 2 * w.F, w.h)
    log(f"full-size cfg{cfg} C={C}: oracle on {len(toks)} tokens")
    Y_ref = om.moe_fwd_tokens(X, idx, gates, W1l, W2l, toks)
    dX_ref, dg_ref = om.moe_bwd_tokens(X, idx, gates, W1l, W2l, dY, toks)
    tol = TOL[w.dtype]
    errs = {"Y": relerr(host(Y[toks]), Y_ref), "dX": relerr(host(B["dX"][toks]), dX_ref),
            "dgates": relerr(host(B["dgates"][toks]), dg_ref)}
    fs = sorted(set(rng.choice(w.F, size=3, replace=False).tolist()) | {0, w.F - 1})
    # the hottest, the median and the coldest expert; the oracle's column
    # form sums over blocks of 32768 slots, so the hot expert of workload 5
    # (524288 slots: weight-gradient tiles with K up to 524288 rows) is
    # checked too
    dw_experts = [int(order[0]), int(order[w.E // 2]), int(order[-1])]
    for e in dw_experts:
        log(f"full-size cfg{cfg} C={C}: weight-gradient columns of expert {e} "
            f"({int(counts[e])} slots)")
        g1, u1, c2 = om.moe_dW_expert_columns(X, idx, gates, W1l, W2l, dY, e, fs)
        errs[f"dW1g[{e}]"] = relerr(host(B["dW1"][e][fs]), g1)
        errs[f"dW1u[{e}]"] = relerr(host(B["dW1"][e][[w.F + f for f in fs]]), u1)
        errs[f"dW2[{e}]"] = relerr(host(B["dW2"][e][:, fs]), c2)
    log(f"  cfg{cfg} C={C}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= tol, (key, e)


# 512 seeded tokens (the first and the last among them) and whole weight
# gradients of the hottest, median and coldest experts, at the planner's chunk
# counts of workloads 3 (C = 8), 4 (C = 4) and 5 (C = 8).  Each token's Y, dX and
# dgates depend on that token's row and slots only (Eq. (4)/(5) per token),
# so the oracle's forward and backward run on the sub-batch of those tokens;
# an expert's dW sums over all its slots (oracle.moe.moe_dW_expert).  The
# hot expert of workload 5 (524288 slots, about two minutes of fp64 host
# work in whole) is checked on sampled columns by test_full_size_sampled.
@pytest.mark.parametrize("cfg,C", [(3, 8), (4, 4), (5, 8)])
def test_full_size_512_tokens_whole_dW(mf, cfg, C):
    t = torch()
    w = W[cfg]
    log(f"512-token check cfg{cfg} C={C}: generating inputs")
    idx, gates = mw.make_routing(w, cfg)
    dev = mw.make_tensors_device(w, cfg, "cuda")
    dev["idx"] = t.from_numpy(idx).cuda()
    dev["gates"] = t.from_numpy(gates).cuda()
    log(f"512-token check cfg{cfg} C={C}: fwd + bwd")
    Y = run_fwd(w, dev, C)
    B = run_bwd(w, dev, C)
    t.cuda.synchronize()
    rng = np.random.default_rng(2000 + cfg)
    toks = np.array(sorted(set(rng.choice(w.T - 2, size=510, replace=False) + 1) |
                           {0, w.T - 1}), dtype=np.int64)
    assert len(toks) == 512
    X = dev["X"].float().cpu().numpy()
    dY = dev["dY"].float().cpu().numpy()
    W1 = dev["W1"].float().cpu().numpy()
    W2 = dev["W2"].float().cpu().numpy()
    tol = TOL[w.dtype]
    log(f"512-token check cfg{cfg} C={C}: oracle on the 512-token sub-batch")
    Y_ref = om.moe_fwd(X[toks], idx[toks], gates[toks], W1, W2, 1)
    R = om.moe_bwd(X[toks], idx[toks], gates[toks], W1, W2, dY[toks], 1)
    tk = t.from_numpy(toks).cuda()
    errs = {"Y": relerr(host(Y[tk]), Y_ref), "dX": relerr(host(B["dX"][tk]), R["dX"]),
            "dgates": relerr(host(B["dgates"][tk]), R["dgates"])}
    del R
    counts = np.bincount(idx.reshape(-1), minlength=w.E)
    order = np.argsort(-counts, kind="stable")
    experts = [int(order[w.E // 2]), int(order[-1])]
    if cfg != 5:
        experts.insert(0, int(order[0]))
    for e in experts:
        log(f"512-token check cfg{cfg} C={C}: whole dW of expert {e} ({int(counts[e])} slots)")
        d1, d2 = om.moe_dW_expert(X, idx, gates, W1, W2, dY, e)
        errs[f"dW1[{e}]"] = relerr(host(B["dW1"][e]), d1)
        errs[f"dW2[{e}]"] = relerr(host(B["dW2"][e]), d2)
    log(f"  cfg{cfg} C={C}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= tol, (key, e)
    del X, dY, W1, W2, dev, Y, B
    gc.collect()


# The largest token count the ABI takes at h = 7168 in bf16: X and dY are
# addressed with 31-bit byte offsets, and T h 2 = 2147475456 leaves 8 KB
# below 2^31, so the last token's row sits at the top of that range.
T_MAX_H7168 = (2 ** 31 - 1) // (7168 * 2)


def test_largest_token_count_sampled(mf):
    """Sampled parity (the first and the last token among them) at the
    largest T for h = 7168, k = 1, 8 experts, C = 2; one more token is
    refused on the host."""
    w = mw.scaled(W[4], T=T_MAX_H7168, E=8, k=1)
    _full_size_sampled(mf, 4, 2, w=w)
    big = mf.make_shape(T_MAX_H7168 + 1, 7168, 2048, 8, 1, mf.BF16)
    with pytest.raises(mf.MemfineError):
        mf.memfine_workspace_bytes(big, 2, mf.PASS_FWD)

