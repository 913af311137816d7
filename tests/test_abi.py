"""The C ABI without a GPU: the library loads, exports every declared symbol,
and its host-side logic (planner, workspace sizes, argument checks, status
strings) behaves as documented.  No device work is launched here."""
import ctypes
import os
import random
import re

import numpy as np
import pytest

import paper_2511_21431_amd as mf
from paper_2511_21431_amd import _lib
from oracle import memory_model as mm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "memfine.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(memfine_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 9
    L = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib._SIGS), "binding and header disagree"


def test_binding_shares_torch_hip_runtime():
    """Whatever the import order, the process maps one HIP runtime: the
    binding loads torch before the library (a library loaded first would bring
    in a second runtime, and its launches on torch's tensors fail)."""
    import subprocess
    import sys
    code = ("import paper_2511_21431_amd._lib as L; L.memfine_set_launch_options(); import torch; "
            "print(len({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=600)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_launch_options_roundtrip_and_validation():
    L = _lib.lib()
    mf.memfine_set_launch_options()
    assert mf.memfine_get_launch_options() == {"tile": 0, "raster": -1, "split_tail": 1,
                                               "pair": 0, "streams": 0, "chunk_order": 0}
    mf.memfine_set_launch_options(tile=mf.TILE_256_REG, raster=3, split_tail=False, pair=True,
                                  chunk_order=mf.CHUNK_EXPERTS)
    assert mf.memfine_get_launch_options() == {"tile": 3, "raster": 3, "split_tail": 0,
                                               "pair": 1, "streams": 0, "chunk_order": 1}
    for bad in (dict(tile=4), dict(tile=-1), dict(raster=5), dict(raster=-2),
                dict(chunk_order=2), dict(chunk_order=-1)):
        with pytest.raises(mf.MemfineError):
            mf.memfine_set_launch_options(**bad)
    assert mf.memfine_get_launch_options()["tile"] == 3       # unchanged by the rejected calls
    assert L.memfine_set_launch_options(None) == 0
    assert mf.memfine_get_launch_options()["tile"] == 0
    assert L.memfine_get_launch_options(None) == -1


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert mf.memfine_status_str(code)
    assert mf.memfine_status_str(12345) == "unknown status"


def _shape(T=8192, h=7168, F=2048, E=32, k=8, dtype=mf.BF16):
    return mf.make_shape(T, h, F, E, k, dtype)


def test_plan_matches_oracle_randomised():
    rng = random.Random(1)
    for _ in range(400):
        E = rng.randint(1, 64)
        h = 64 * rng.randint(1, 120)
        F = 64 * rng.randint(1, 60)
        dtype = rng.choice([mf.BF16, mf.F32])
        T = rng.randint(0, 50000)
        k = rng.randint(1, 8)
        counts = np.random.default_rng(rng.randint(0, 10**6)).multinomial(T * k, np.ones(E) / E)
        beta = (2 if dtype == mf.BF16 else 4) * (2 * h + 2 * F)
        s2 = int(counts.sum())
        # budgets spread around the bin edges, including exact edges
        choice = rng.random()
        if choice < 0.3 and s2 > 0:
            b = rng.choice([1, 2, 4, 8])
            budget = -(-s2 * beta // b) + rng.choice([-1, 0, 1])
        else:
            budget = rng.randint(-10, 4 * 10**10)
        fixed = rng.choice([0, 0, rng.randint(0, 10**9)])
        bins = sorted(rng.sample([1, 2, 3, 4, 6, 8, 16], rng.randint(1, 4)))
        shape = mf.make_shape(T, h, F, E, k, dtype)
        # the paper's model alone: beta = Table 2 rows 11-13
        rc, C, info = mf.memfine_plan(shape, counts, budget, bins=bins, fixed_bytes=fixed,
                                      beta_bytes=beta)
        ref = mm.plan(counts, budget, beta, bins=bins, fixed=fixed)
        assert C == ref["C"], (budget, fixed, s2, bins, ref)
        assert (rc == 0) == ref["ok"]
        assert info["s_recv"] == s2 and info["beta"] == beta
        if ref["c_theory"] is not None:
            assert info["c_theory"] == ref["c_theory"]
        else:
            assert info["c_theory"] == -1


def test_plan_default_keeps_eq3_for_the_implementation():
    """Default beta: max(Table 2's, the library's own) and the workspace check.
    On the dense-FFN shape (F > h: the backward holds more per slot than
    Table 2's rows) every budget the planner accepts holds the chunk's whole
    workspace, the chosen bin is the smallest such bin at or above Eq. (9)'s
    c, and the paper-model bin is reported beside it (Eq. (3), Eq. (8)/(9))."""
    import moe_workloads as mw
    w = mw.WORKLOADS[3]
    idx, _ = mw.make_routing(w, 3)
    counts = np.bincount(idx.reshape(-1), minlength=w.E)
    shape = mf.make_shape(w.T, w.h, w.F, w.E, w.k, mf.BF16)
    beta_paper = 2 * (2 * w.h + 2 * w.F)
    bins = (1, 2, 4, 8)
    ws = {b: mf.memfine_workspace_bytes(shape, b, mf.PASS_BWD) for b in bins}
    rng = np.random.default_rng(7)
    budgets = sorted(set(np.linspace(0.30e9, 3.15e9, 3000).astype(np.int64).tolist()
                         + [ws[b] + d for b in bins for d in (-1, 0, 1)]
                         + rng.integers(10**8, 4 * 10**9, 1000).tolist()))
    n_ok = n_paper_over = 0
    for budget in budgets:
        rc, C, info = mf.memfine_plan(shape, counts, budget, bins=bins)
        assert info["beta_paper"] == beta_paper and info["beta_impl"] > beta_paper
        assert info["beta"] == info["beta_impl"]
        assert info["workspace_bytes"] == ws[C]
        c = info["c_theory"]
        feasible = [b for b in bins if b >= c and ws[b] <= budget]
        if rc == 0:
            n_ok += 1
            assert ws[C] <= budget, (budget, C, ws[C])
            assert C == min(feasible), (budget, C, feasible)
        else:
            assert rc == _lib.ERR_BUDGET and not feasible and C == max(bins)
        ref = mm.plan(counts, budget, beta_paper, bins=bins)
        assert info["paper_chunks"] == ref["C"]
        if ref["ok"] and ws[ref["C"]] > budget:
            n_paper_over += 1           # where Table 2's beta alone would overshoot
    assert n_ok > 1000 and n_paper_over > 100


def test_plan_handworked_config5():
    shape = _shape(T=131072)
    counts = [0] * 32
    counts[3] = 131072 * 8 // 2
    counts[0] = 131072 * 8 - counts[3]
    want = {4: 16, 8: 8, 16: 4, 32: 2, 64: 1}
    for gb, C in want.items():
        rc, got, info = mf.memfine_plan(shape, counts, gb * 10**9, bins=(1, 2, 4, 8, 16))
        assert rc == 0 and got == C


def test_plan_beta_override_and_errors():
    shape = _shape()
    counts = [2048] * 32
    rc, C, info = mf.memfine_plan(shape, counts, 10**9, beta_bytes=100)
    assert info["beta"] == 100 and C == 1
    rc, C, info = mf.memfine_plan(shape, counts, 10**6)
    assert rc == _lib.ERR_BUDGET and C == 8 and info["fits"] == 0
    L = _lib.lib()
    out = ctypes.c_int32(0)
    bins = (ctypes.c_int32 * 2)(1, 0)
    c = (ctypes.c_int64 * 32)(*counts)
    assert L.memfine_plan(ctypes.byref(shape), c, 10**9, 0, 0, bins, 2, ctypes.byref(out), None) == -1
    bins = (ctypes.c_int32 * 1)(2)
    assert L.memfine_plan(ctypes.byref(shape), None, 10**9, 0, 0, bins, 1, ctypes.byref(out), None) == -1
    assert L.memfine_plan(ctypes.byref(shape), c, 10**9, 0, 0, bins, 0, ctypes.byref(out), None) == -1
    assert L.memfine_plan(ctypes.byref(shape), c, 10**9, -1, 0, bins, 1, ctypes.byref(out), None) == -1


@pytest.mark.parametrize("T,h,F,E,k,dtype", [(8192, 7168, 2048, 32, 8, mf.BF16),
                                             (256, 64, 128, 4, 2, mf.F32),
                                             (10, 128, 64, 3, 3, mf.BF16)])
def test_workspace_bytes(T, h, F, E, k, dtype):
    s = mf.make_shape(T, h, F, E, k, dtype)
    for p in (mf.PASS_FWD, mf.PASS_BWD):
        vals = [mf.memfine_workspace_bytes(s, C, p) for C in (1, 2, 3, 4, 8, 16, T, T + 5)]
        assert all(a >= b for a, b in zip(vals, vals[1:]))
        assert vals[-1] == vals[-2]           # more chunks than tokens: one token per chunk
        es = 2 if dtype == mf.BF16 else 4
        # at least the per-slot intermediates: a and y forward; u, g*a and the
        # input gradient backward
        per_slot = es * (F + h) if p == mf.PASS_FWD else es * (3 * F + h)
        assert vals[0] >= T * k * per_slot
    # the backward holds more per slot than the forward
    assert mf.memfine_workspace_bytes(s, 1, mf.PASS_BWD) > mf.memfine_workspace_bytes(s, 1, mf.PASS_FWD)


def test_workspace_bytes_expert_order():
    """Expert-ordered chunks: the layer's routing tables for all N = T k slots
    (16 bytes per slot and more) are held for the whole call, beside one
    chunk's intermediates for at most ceil(N / C) rows; the planner's
    workspace check follows the option."""
    T, h, F, E, k = 8192, 7168, 2048, 32, 8
    s = mf.make_shape(T, h, F, E, k, mf.BF16)
    N = T * k
    tok = {C: mf.memfine_workspace_bytes(s, C, mf.PASS_BWD) for C in (1, 2, 4, 8, 16)}
    try:
        mf.memfine_set_launch_options(chunk_order=mf.CHUNK_EXPERTS)
        ex = {C: mf.memfine_workspace_bytes(s, C, mf.PASS_BWD) for C in (1, 2, 3, 4, 8, 16, T, T + 9)}
        vals = list(ex.values())
        assert all(a >= b for a, b in zip(vals, vals[1:])) and ex[T] == ex[T + 9]
        tables = ex[T]                          # at C = T a chunk holds k rows
        assert tables >= 16 * N
        per_row = 2 * (3 * F + h)               # u, g*a and the input gradient, bf16
        for C in (1, 2, 4, 8, 16):
            rows = -(-N // C)
            assert ex[C] - tables >= (rows - k) * per_row
            # the same intermediates as the token order's chunk, plus the tables
            assert abs((ex[C] - tables) - (tok[C] - 16 * rows)) < 0.01 * tok[C] + 2 ** 20
        counts = [N // E] * E
        for budget in (5e9, 1e10, 2e10, 4e10):
            rc, C, info = mf.memfine_plan(s, counts, int(budget), bins=(1, 2, 4, 8, 16))
            assert info["workspace_bytes"] == ex[C]
            if rc == 0:
                assert ex[C] <= budget
    finally:
        mf.memfine_set_launch_options()


def test_workspace_scales_with_chunks():
    s = _shape()
    w1 = mf.memfine_workspace_bytes(s, 1, mf.PASS_BWD)
    for C in (2, 4, 8):
        wc = mf.memfine_workspace_bytes(s, C, mf.PASS_BWD)
        assert abs(wc / w1 - 1.0 / C) < 0.01


@pytest.mark.parametrize("bad", [dict(h=100), dict(F=96), dict(h=0), dict(E=0), dict(E=2000),
                                 dict(k=0), dict(T=-1), dict(dtype=7), dict(T=2**28, k=8)])
def test_invalid_shapes_rejected_on_host(bad):
    kw = dict(T=16, h=64, F=64, E=4, k=2, dtype=mf.BF16)
    kw.update(bad)
    s = mf.make_shape(**kw)
    L = _lib.lib()
    expect = (-2,) if ("dtype" in bad or "T" in bad and bad.get("k") == 8) else (-1,)
    assert L.memfine_workspace_bytes(ctypes.byref(s), 1, 0) < 0
    rc = L.memfine_moe_fwd(ctypes.byref(s), 1, None, None, None, None, None, None, None, None)
    assert rc in expect
    rc = L.memfine_moe_bwd(ctypes.byref(s), 1, *([None] * 10), 0, None, None)
    assert rc in expect


def test_null_pointers_rejected_on_host():
    s = mf.make_shape(16, 64, 64, 4, 2, mf.BF16)
    L = _lib.lib()
    fake = ctypes.c_void_p(0x1000)
    assert L.memfine_moe_fwd(ctypes.byref(s), 1, fake, fake, fake, fake, None, fake, None, None) == -1
    assert L.memfine_moe_fwd(ctypes.byref(s), 0, fake, fake, fake, fake, fake, fake, None, None) == -1
    args = [fake] * 10
    args[7] = None   # dW1
    assert L.memfine_moe_bwd(ctypes.byref(s), 1, *args, 0, None, None) == -1
    assert L.memfine_moe_bwd(ctypes.byref(s), 1, *([fake] * 10), 2, None, None) == -1
    assert L.memfine_count(None, fake, fake, None, None) == -1
    assert L.memfine_dispatch(ctypes.byref(s), fake, 5, 3, fake, fake, fake, fake, None, None) == -1
    assert L.memfine_dispatch(ctypes.byref(s), fake, 0, 17, fake, fake, fake, fake, None, None) == -1


def test_binding_checks_tensor_shapes():
    torch = pytest.importorskip("torch")
    s = mf.make_shape(16, 64, 64, 4, 2, mf.BF16)
    X = torch.zeros(16, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        mf.memfine_moe_fwd(s, 1, X[:, :32], None, None, None, None, None)
    with pytest.raises(ValueError):
        mf.memfine_moe_fwd(s, 1, X.float(), None, None, None, None, None)
    with pytest.raises(ValueError):     # host tensors are refused
        mf.memfine_moe_fwd(s, 1, X, torch.zeros(16, 2, dtype=torch.int32),
                           torch.zeros(16, 2), torch.zeros(4, 128, 64, dtype=torch.bfloat16),
                           torch.zeros(4, 64, 64, dtype=torch.bfloat16), X)


def test_router_limits_and_null_pointers_rejected_on_host():
    L = _lib.lib()
    fake = ctypes.c_void_p(0x1000)
    ok = mf.make_shape(16, 64, 64, 8, 2, mf.BF16)
    for bad in (mf.make_shape(16, 64, 64, 257, 2, mf.BF16),   # E > 256
                mf.make_shape(16, 64, 64, 32, 17, mf.BF16),   # k > 16
                mf.make_shape(16, 64, 64, 3, 4, mf.BF16)):    # k > E
        assert L.memfine_router_fwd(ctypes.byref(bad), fake, fake, fake, fake, None, None) == -2
        assert L.memfine_router_bwd(ctypes.byref(bad), *([fake] * 7), 0, 0, None, None) == -2
    assert L.memfine_router_fwd(ctypes.byref(ok), None, fake, fake, fake, None, None) == -1
    assert L.memfine_router_fwd(ctypes.byref(ok), fake, fake, fake, None, None, None) == -1
    args = [fake] * 7
    args[5] = None   # dX
    assert L.memfine_router_bwd(ctypes.byref(ok), *args, 0, 0, None, None) == -1
    assert L.memfine_router_bwd(ctypes.byref(ok), *([fake] * 7), 2, 0, None, None) == -1
    assert L.memfine_router_bwd(ctypes.byref(ok), *([fake] * 7), 0, -1, None, None) == -1
    assert L.memfine_router_fwd(None, fake, fake, fake, fake, None, None) == -1


def test_missing_library_fails_loudly():
    """Without the built library every entry point raises: there is no CPU
    fallback behind the binding."""
    import subprocess
    import sys
    code = ("import paper_2511_21431_amd._lib as L\n"
            "L.LIB_PATH = '/nonexistent/libmemfine.so'\n"
            "try:\n"
            "    L.memfine_status_str(0)\n"
            "except ImportError as e:\n"
            "    print('raised', 'no fallback' in str(e))\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))), timeout=300)
    assert "raised True" in out.stdout, out.stdout + out.stderr
