"""GPU parity of the router (memfine_router_fwd / memfine_router_bwd) against
oracle/router.py, and of the trainable block router -> expert layer ->
router backward.

* idx: bit-exact against the oracle's top-k taken on the kernel's own fp32
  logits (the decision is made in the kernel's precision);
* logits against fp64 logits of the same bf16 inputs: 2e-2 (bf16) / 1e-4
  (fp32) of max |logit|; gates against the oracle's from the kernel logits:
  1e-5;
* dX, dWr: max|got - ref| / max|ref| <= 2e-2 (bf16: dlogits enter the weight
  gradient GEMM as bf16) / 1e-4 (fp32).
* against the fp64 logits alone: the kernel's selection is a valid top-k of
  them up to the logit tolerance (every selected logit is at least every
  unselected one minus twice the tolerance), and on the tokens whose
  selection agrees with the fp64 top-k, the backward (run again with the
  gate gradients of the other tokens set to zero) matches the oracle chain
  that starts from the fp64 logits.
"""
import numpy as np
import pytest

import moe_workloads as mw
from gpu_harness import TOL, host, log, relerr, shape_of, torch
from oracle import moe as om
from oracle import router as orr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_21431_amd as m
    m.lib()
    return m


def make(T, h, E, k, dtype, seed):
    rng = np.random.default_rng(seed)
    X = mw.round_to_bf16(rng.standard_normal((T, h))) if dtype == "bf16" else rng.standard_normal((T, h))
    Wr = rng.standard_normal((E, h)) / np.sqrt(h)
    if dtype == "bf16":
        Wr = mw.round_to_bf16(Wr)
    dg = rng.standard_normal((T, k))
    w = mw.Workload("router", T=T, h=h, F=64, E=E, k=k, dtype=dtype, routing="dirichlet")
    return w, X.astype(np.float32), Wr.astype(np.float32), dg.astype(np.float32)


def dev(a, dtype):
    t = torch()
    d = t.bfloat16 if dtype == "bf16" else t.float32
    return t.from_numpy(np.ascontiguousarray(a)).cuda().to(d).contiguous()


def run_router(mf, w, X, Wr, dg, accumulate_dX=None):
    t = torch()
    Xd, Wd = dev(X, w.dtype), dev(Wr, w.dtype)
    idx = t.full((w.T, w.k), -1, dtype=t.int32, device="cuda")
    gates = t.full((w.T, w.k), float("nan"), device="cuda")
    logits = t.full((w.T, w.E), float("nan"), device="cuda")
    mf.memfine_router_fwd(shape_of(w), Xd, Wd, idx, gates, logits)
    dgd = t.from_numpy(dg).cuda()
    if accumulate_dX is None:
        dX = t.full((w.T, w.h), float("nan"), device="cuda").to(Xd.dtype)
    else:
        dX = dev(accumulate_dX, w.dtype)
    dWr = t.full((w.E, w.h), float("nan"), device="cuda")
    mf.memfine_router_bwd(shape_of(w), Xd, Wd, idx, gates, dgd, dX, dWr,
                          accumulate_dX=accumulate_dX is not None)
    t.cuda.synchronize()
    return {"idx": idx.cpu().numpy(), "gates": host(gates), "logits": host(logits),
            "dX": host(dX), "dWr": host(dWr)}


# (T, h, E, k, dtype): narrow routers (E <= 64, one fused kernel), wide ones
# (64 < E <= 256: a fused kernel, or, for E a multiple of 32, the logits as a
# grouped GEMM and a top-k kernel), and the router of the paper's Table 3
# models at one GPU's token count (T = 8192, h = 7168, 256 routed experts,
# top-8)
CASES = [(1000, 512, 16, 4, "bf16"), (777, 256, 6, 2, "bf16"), (513, 128, 33, 8, "bf16"),
         (256, 64, 64, 16, "bf16"), (300, 192, 4, 4, "bf16"), (200, 128, 5, 1, "bf16"),
         (1000, 512, 16, 4, "f32"), (129, 64, 40, 3, "f32"),
         (700, 256, 100, 6, "bf16"), (513, 128, 256, 8, "bf16"), (333, 64, 65, 16, "bf16"),
         (300, 64, 129, 16, "f32"), (1000, 512, 200, 4, "f32"), (8192, 7168, 256, 8, "bf16"),
         (600, 256, 96, 5, "bf16"), (700, 128, 160, 4, "f32"), (2048, 1024, 128, 8, "bf16"),
         (4099, 512, 224, 16, "bf16")]


def check_against_fp64_logits(mf, w, X, Wr, dg, got, tol):
    """The kernel's decisions against the fp64 logits (not the kernel's own):
    a valid top-k up to the logit tolerance, and the backward of the tokens
    whose selection agrees with the fp64 top-k against the fp64 chain."""
    t = torch()
    k = w.k
    z64 = orr.logits_of(X, Wr)
    delta = tol * np.max(np.abs(z64))
    sel = got["idx"].astype(np.int64)
    rows = np.arange(w.T)[:, None]
    assert np.all((sel >= 0) & (sel < w.E))
    assert np.all(np.sort(sel, axis=1)[:, 1:] != np.sort(sel, axis=1)[:, :-1])   # k distinct ids
    if w.E > k:
        zsel = z64[rows, sel].min(axis=1)
        unsel = z64.copy()
        unsel[rows, sel] = -np.inf
        gap = zsel - unsel.max(axis=1)
        assert np.all(gap >= -2 * delta), float(gap.min())
    ref64 = orr.router_fwd(X, Wr, k)
    agree = np.all(ref64["idx"] == sel, axis=1)
    assert agree.mean() > 0.5, agree.mean()
    # a renormalised gate moves by at most 2 g_j max|dz| <= 2 delta when the
    # logits move by delta
    assert np.max(np.abs(got["gates"][agree] - ref64["gates"][agree])) <= 2 * delta
    if k == 1:
        return
    dgm = np.where(agree[:, None], dg, 0.0).astype(np.float32)
    Xd, Wd = dev(X, w.dtype), dev(Wr, w.dtype)
    idx = t.from_numpy(np.ascontiguousarray(got["idx"])).cuda()
    gates = t.from_numpy(np.ascontiguousarray(got["gates"])).cuda()
    dX = t.full((w.T, w.h), float("nan"), device="cuda").to(Xd.dtype)
    dWr = t.full((w.E, w.h), float("nan"), device="cuda")
    mf.memfine_router_bwd(shape_of(w), Xd, Wd, idx, gates, t.from_numpy(dgm).cuda(), dX, dWr)
    t.cuda.synchronize()
    ref = orr.router_bwd(X, Wr, ref64["idx"], z64, dgm)
    assert relerr(host(dX)[agree], ref["dX"][agree]) <= tol
    assert relerr(host(dWr), ref["dWr"]) <= tol


@pytest.mark.parametrize("T,h,E,k,dtype", CASES)
def test_router_parity(mf, T, h, E, k, dtype):
    w, X, Wr, dg = make(T, h, E, k, dtype, seed=T + E + k)
    log(f"router T={T} h={h} E={E} k={k} {dtype}")
    got = run_router(mf, w, X, Wr, dg)
    tol = TOL[dtype]
    ref_logits = orr.logits_of(X, Wr)
    assert relerr(got["logits"], ref_logits) <= tol
    own = orr.router_fwd(None, None, k, logits=got["logits"].astype(np.float64))
    assert np.array_equal(got["idx"], own["idx"])
    assert np.max(np.abs(got["gates"] - own["gates"])) <= 1e-5
    ref = orr.router_bwd(X, Wr, own["idx"], got["logits"], dg)
    if k == 1:
        # one selected expert: its gate is 1 whatever the logits, no gradient
        assert np.max(np.abs(ref["dX"])) < 1e-12 and np.max(np.abs(ref["dWr"])) < 1e-12
        assert np.max(np.abs(got["dX"])) == 0.0 and np.max(np.abs(got["dWr"])) == 0.0
    else:
        assert relerr(got["dX"], ref["dX"]) <= tol
        assert relerr(got["dWr"], ref["dWr"]) <= tol
    check_against_fp64_logits(mf, w, X, Wr, dg, got, tol)


def test_router_ties_take_the_lower_id(mf):
    """Equal logits (Wr rows repeated): the lower expert id is selected first,
    on the narrow and on the wide kernel."""
    for E, k in ((48, 6), (256, 8)):
        w, X, Wr, dg = make(256, 128, E, k, "bf16", seed=E)
        Wr[1::2] = Wr[0::2][: E // 2]           # expert 2i+1 repeats expert 2i
        got = run_router(mf, w, X, Wr, dg)
        own = orr.router_fwd(None, None, k, logits=got["logits"].astype(np.float64))
        assert np.array_equal(got["logits"][:, 1::2], got["logits"][:, 0::2])
        assert np.array_equal(got["idx"], own["idx"])
        assert np.all(got["idx"][:, 0] % 2 == 0)   # of each tied pair, the even id first


@pytest.mark.parametrize("E", [96, 256])
def test_router_without_logits_output(mf, E):
    """Without a logits output the wide router keeps its logits in working
    memory: the same ids and gates, bit for bit, as with the output."""
    t = torch()
    w, X, Wr, dg = make(1500, 256, E, 8, "bf16", seed=E + 3)
    Xd, Wd = dev(X, "bf16"), dev(Wr, "bf16")
    out = []
    for with_logits in (True, False):
        idx = t.full((w.T, w.k), -1, dtype=t.int32, device="cuda")
        gates = t.full((w.T, w.k), float("nan"), device="cuda")
        logits = t.empty((w.T, w.E), device="cuda") if with_logits else None
        mf.memfine_router_fwd(shape_of(w), Xd, Wd, idx, gates, logits)
        t.cuda.synchronize()
        out.append((idx.cpu().numpy(), host(gates)))
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


def test_router_accumulates_into_dX(mf):
    w, X, Wr, dg = make(600, 256, 16, 4, "bf16", seed=5)
    base = mw.round_to_bf16(np.random.default_rng(1).standard_normal((600, 256))).astype(np.float32)
    got = run_router(mf, w, X, Wr, dg, accumulate_dX=base)
    own = orr.router_fwd(None, None, 4, logits=got["logits"].astype(np.float64))
    ref = orr.router_bwd(X, Wr, own["idx"], got["logits"], dg)
    # the output tensor is base + contribution, rounded once to bf16
    assert relerr(got["dX"], base + ref["dX"]) <= 2e-2
    assert relerr(got["dX"], base) > 1e-3          # the contribution is there


def test_router_bwd_drops_out_of_range_ids(mf):
    t = torch()
    w, X, Wr, dg = make(300, 128, 8, 2, "bf16", seed=8)
    Xd, Wd = dev(X, "bf16"), dev(Wr, "bf16")
    idx = t.zeros((300, 2), dtype=t.int32, device="cuda")
    gates = t.full((300, 2), 0.5, device="cuda")
    idx[:, 0] = t.arange(300, device="cuda", dtype=t.int32) % 8
    idx[:, 1] = t.where(t.arange(300, device="cuda") % 3 == 0, -5, 99).to(t.int32)
    dX = t.zeros((300, 128), dtype=t.bfloat16, device="cuda")
    dWr = t.zeros((8, 128), device="cuda")
    dgd = t.from_numpy(dg).cuda()
    mf.memfine_router_bwd(shape_of(w), Xd, Wd, idx, gates, dgd, dX, dWr)
    t.cuda.synchronize()
    # only the valid slot j = 0 counts: c = g0 dg0, dz0 = g0 (dg0 - c)
    g0 = 0.5
    dz0 = g0 * (dg[:, 0] - g0 * dg[:, 0])
    Wr64 = Wr.astype(np.float64)
    ref_dX = dz0[:, None] * Wr64[np.arange(300) % 8]
    assert relerr(host(dX), ref_dX) <= 2e-2
    ref_dWr = np.zeros((8, 128))
    for tt in range(300):
        ref_dWr[tt % 8] += dz0[tt] * X[tt]
    assert relerr(host(dWr), ref_dWr) <= 2e-2


def test_router_full_size_sampled(mf):
    """The router at the benchmark's shapes (workload 2: T = 8192, h = 2048,
    E = 16, top-4), in the launch configuration the benchmark times: sampled
    tokens for logits / idx / gates / dX, sampled columns of dWr."""
    t = torch()
    w = mw.WORKLOADS[2]
    rng = np.random.default_rng(2)
    Xd = mw.make_tensors_device(w, 2, "cuda", with_dy=False)["X"]
    Wr = mw.round_to_bf16(rng.standard_normal((w.E, w.h)) / np.sqrt(w.h)).astype(np.float32)
    Wd = dev(Wr, "bf16")
    idx = t.empty((w.T, w.k), dtype=t.int32, device="cuda")
    gates = t.empty((w.T, w.k), device="cuda")
    logits = t.empty((w.T, w.E), device="cuda")
    log("router full size: fwd")
    mf.memfine_router_fwd(shape_of(w), Xd, Wd, idx, gates, logits)
    dg = rng.standard_normal((w.T, w.k)).astype(np.float32)
    dX = t.empty((w.T, w.h), dtype=t.bfloat16, device="cuda")
    dWr = t.empty((w.E, w.h), device="cuda")
    log("router full size: bwd")
    mf.memfine_router_bwd(shape_of(w), Xd, Wd, idx, gates, t.from_numpy(dg).cuda(), dX, dWr)
    t.cuda.synchronize()
    X = Xd.float().cpu().numpy()
    L = host(logits)
    toks = sorted(set(rng.choice(w.T, 24, replace=False).tolist()) | {0, w.T - 1})
    assert relerr(L[toks], orr.logits_of(X[toks], Wr)) <= 2e-2
    own = orr.router_fwd(None, None, w.k, logits=L.astype(np.float64))
    assert np.array_equal(idx.cpu().numpy(), own["idx"])
    assert np.max(np.abs(host(gates) - own["gates"])) <= 1e-5
    ref = orr.router_bwd(X, Wr, own["idx"], L, dg)
    assert relerr(host(dX)[toks], ref["dX"][toks]) <= 2e-2
    cols = sorted(rng.choice(w.h, 16, replace=False).tolist())
    assert relerr(host(dWr)[:, cols], ref["dWr"][:, cols]) <= 2e-2


def test_trainable_block(mf):
    """Router -> chunked expert layer -> layer backward -> router backward on
    the GPU, against the same chain of oracles (selection from the kernel's
    logits): Y, dX (layer + router), dW1, dW2, dWr."""
    t = torch()
    w = mw.Workload("block", T=512, h=256, F=192, E=8, k=2, dtype="bf16", routing="dirichlet")
    rng = np.random.default_rng(77)
    X = mw.round_to_bf16(rng.standard_normal((w.T, w.h))).astype(np.float32)
    Wr = mw.round_to_bf16(rng.standard_normal((w.E, w.h)) / np.sqrt(w.h)).astype(np.float32)
    W1 = mw.round_to_bf16(rng.standard_normal((w.E, 2 * w.F, w.h)) * 0.05).astype(np.float32)
    W2 = mw.round_to_bf16(rng.standard_normal((w.E, w.h, w.F)) * 0.05).astype(np.float32)
    dY = mw.round_to_bf16(rng.standard_normal((w.T, w.h))).astype(np.float32)
    Xd, Wrd, W1d, W2d, dYd = (dev(a, "bf16") for a in (X, Wr, W1, W2, dY))
    S = shape_of(w)
    idx = t.empty((w.T, w.k), dtype=t.int32, device="cuda")
    gates = t.empty((w.T, w.k), device="cuda")
    logits = t.empty((w.T, w.E), device="cuda")
    mf.memfine_router_fwd(S, Xd, Wrd, idx, gates, logits)
    Y = t.empty((w.T, w.h), dtype=t.bfloat16, device="cuda")
    mf.memfine_moe_fwd(S, 2, Xd, idx, gates, W1d, W2d, Y)
    dX = t.empty_like(Y)
    dW1 = t.empty((w.E, 2 * w.F, w.h), device="cuda")
    dW2 = t.empty((w.E, w.h, w.F), device="cuda")
    dg = t.empty((w.T, w.k), device="cuda")
    mf.memfine_moe_bwd(S, 2, Xd, idx, gates, W1d, W2d, dYd, dX, dW1, dW2, dg)
    dWr = t.empty((w.E, w.h), device="cuda")
    mf.memfine_router_bwd(S, Xd, Wrd, idx, gates, dg, dX, dWr, accumulate_dX=True)
    t.cuda.synchronize()
    own = orr.router_fwd(None, None, w.k, logits=host(logits).astype(np.float64))
    assert np.array_equal(idx.cpu().numpy(), own["idx"])
    Y_ref = om.moe_fwd(X, own["idx"], own["gates"], W1, W2, 2)
    R = om.moe_bwd(X, own["idx"], own["gates"], W1, W2, dY, 2)
    RR = orr.router_bwd(X, Wr, own["idx"], host(logits), R["dgates"])
    errs = {"Y": relerr(host(Y), Y_ref), "dX": relerr(host(dX), R["dX"] + RR["dX"]),
            "dW1": relerr(host(dW1), R["dW1"]), "dW2": relerr(host(dW2), R["dW2"]),
            "dWr": relerr(host(dWr), RR["dWr"])}
    log("block: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for key, e in errs.items():
        assert e <= 2e-2, (key, e)


def test_trainable_block_wide_router_32_local_experts(mf):
    """The router of a 256-expert model (top-8, h = 7168) in front of this
    GPU's slice of 32 local experts (experts 0..31; slots routed to the other
    224 are another GPU's and are dropped here, passing no gradient back from
    this layer), against the chain of oracles started from the kernel's
    logits: Y, dX (layer + router), dW1, dW2, dWr."""
    t = torch()
    T, h, F, Er, El, k = 2048, 7168, 256, 256, 32, 8
    rng = np.random.default_rng(91)
    X = mw.round_to_bf16(rng.standard_normal((T, h))).astype(np.float32)
    Wr = mw.round_to_bf16(rng.standard_normal((Er, h)) / np.sqrt(h)).astype(np.float32)
    W1 = mw.round_to_bf16(rng.standard_normal((El, 2 * F, h)) * 0.02).astype(np.float32)
    W2 = mw.round_to_bf16(rng.standard_normal((El, h, F)) * 0.05).astype(np.float32)
    dY = mw.round_to_bf16(rng.standard_normal((T, h))).astype(np.float32)
    Xd, Wrd, W1d, W2d, dYd = (dev(a, "bf16") for a in (X, Wr, W1, W2, dY))
    wr = mw.Workload("router", T=T, h=h, F=64, E=Er, k=k, dtype="bf16", routing="dirichlet")
    wl = mw.Workload("layer", T=T, h=h, F=F, E=El, k=k, dtype="bf16", routing="dirichlet")
    Sr, Sl = shape_of(wr), shape_of(wl)
    idx = t.empty((T, k), dtype=t.int32, device="cuda")
    gates = t.empty((T, k), device="cuda")
    logits = t.empty((T, Er), device="cuda")
    log("wide block: router fwd")
    mf.memfine_router_fwd(Sr, Xd, Wrd, idx, gates, logits)
    local = t.where(idx < El, idx, t.full_like(idx, -1))
    Y = t.empty((T, h), dtype=t.bfloat16, device="cuda")
    log("wide block: layer fwd / bwd")
    mf.memfine_moe_fwd(Sl, 2, Xd, local, gates, W1d, W2d, Y)
    dX = t.empty_like(Y)
    dW1 = t.empty((El, 2 * F, h), device="cuda")
    dW2 = t.empty((El, h, F), device="cuda")
    dg = t.empty((T, k), device="cuda")
    mf.memfine_moe_bwd(Sl, 2, Xd, local, gates, W1d, W2d, dYd, dX, dW1, dW2, dg)
    dWr = t.empty((Er, h), device="cuda")
    log("wide block: router bwd")
    mf.memfine_router_bwd(Sr, Xd, Wrd, idx, gates, dg, dX, dWr, accumulate_dX=True)
    t.cuda.synchronize()
    L = host(logits)
    own = orr.router_fwd(None, None, k, logits=L.astype(np.float64))
    assert np.array_equal(idx.cpu().numpy(), own["idx"])
    remote = own["idx"] >= El
    assert 0.5 < remote.mean() < 0.95            # most slots go to the other GPUs' experts
    ref_idx = np.where(remote, 0, own["idx"]).astype(np.int32)
    ref_g = np.where(remote, 0.0, own["gates"])
    log("wide block: oracle")
    Y_ref = om.moe_fwd(X, ref_idx, ref_g, W1, W2, 2)
    R = om.moe_bwd(X, ref_idx, ref_g, W1, W2, dY, 2)
    R["dgates"] = np.where(remote, 0.0, R["dgates"])
    assert np.all(host(dg)[remote] == 0.0)
    RR = orr.router_bwd(X, Wr, own["idx"], L, R["dgates"])
    errs = {"Y": relerr(host(Y), Y_ref), "dX": relerr(host(dX), R["dX"] + RR["dX"]),
            "dW1": relerr(host(dW1), R["dW1"]), "dW2": relerr(host(dW2), R["dW2"]),
            "dWr": relerr(host(dWr), RR["dWr"]), "dgates": relerr(host(dg), R["dgates"])}
    log("wide block: " + ", ".join(f"{kk}={v:.2e}" for kk, v in errs.items()))
    for key, e in errs.items():
        assert e <= 2e-2, (key, e)
