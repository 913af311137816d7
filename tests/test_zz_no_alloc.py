"""The allocation-free forward (memfine_moe_fwd_noalloc, for callers that
cannot allocate: HIP graph capture, tight serving loops) against the
allocating forward, through the C ABI: bit-identical outputs on two calls in
a row, the second with a smaller input, both also within the bf16 tolerance
of the oracle; nothing is allocated (the torch allocator, the library's pool
and its per-stream workspace stay as they were); a call whose largest chunk
needs more than the static scratch is refused before anything runs."""
import gc

import numpy as np
import pytest

import moe_workloads as mw
from gpu_harness import TOL, device_case, host, log, nan_like, relerr, shape_of, torch
from oracle import moe as om

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_21431_amd as m
    m.lib()
    return m


def _fwd_both(mf, w, dev, C, stream):
    t = torch()
    s = shape_of(w)
    Y_ref = nan_like((w.T, w.h), t.bfloat16)
    mf.memfine_moe_fwd(s, C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"], Y_ref)
    t.cuda.synchronize()
    Y = nan_like((w.T, w.h), t.bfloat16)
    # tensors of earlier tests that only the cycle collector frees (a caught
    # exception's traceback holds their frames) go now, not inside the window
    gc.collect()
    t.cuda.synchronize()
    torch_before = t.cuda.memory_allocated()
    pool_before = mf.memfine_pool_high_water()
    with t.cuda.stream(stream):
        mf.memfine_moe_fwd_noalloc(s, C, dev["X"], dev["idx"], dev["gates"], dev["W1"], dev["W2"], Y)
        assert mf.memfine_workspace_held() == 0       # no workspace block for this stream
    stream.synchronize()
    assert t.cuda.memory_allocated() == torch_before
    assert mf.memfine_pool_high_water() == pool_before
    return host(Y_ref), host(Y)


def test_fwd_noalloc_matches_fwd_two_calls(mf):
    t = torch()
    stream = t.cuda.Stream()
    # first call, then a smaller input (fewer tokens, other sizes)
    for name, w, C, seed in (("larger", mw.scaled(mw.WORKLOADS[2], T=3000, h=512, F=384), 2, 71),
                             ("smaller", mw.scaled(mw.WORKLOADS[4], T=333, h=256, F=128), 3, 72)):
        s = shape_of(w)
        assert mf.memfine_workspace_bytes(s, C, mf.PASS_FWD) <= mf.NOALLOC_SCRATCH_BYTES
        case = mw.make_case(w, seed, with_dy=False)
        dev = device_case(w, case)
        log(f"no-alloc forward, {name} input T={w.T} h={w.h} F={w.F} C={C}")
        Y_ref, Y = _fwd_both(mf, w, dev, C, stream)
        assert np.array_equal(Y, Y_ref)
        ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
        assert relerr(Y, ref) <= TOL["bf16"]


def test_fwd_noalloc_refuses_chunks_beyond_the_scratch(mf):
    t = torch()
    w = mw.scaled(mw.WORKLOADS[2], T=8192, h=2048, F=1408)
    s = shape_of(w)
    assert mf.memfine_workspace_bytes(s, 1, mf.PASS_FWD) > mf.NOALLOC_SCRATCH_BYTES
    X = t.zeros((w.T, w.h), dtype=t.bfloat16, device="cuda")
    idx = t.zeros((w.T, w.k), dtype=t.int32, device="cuda")
    g = t.zeros((w.T, w.k), device="cuda")
    W1 = t.zeros((w.E, 2 * w.F, w.h), dtype=t.bfloat16, device="cuda")
    W2 = t.zeros((w.E, w.h, w.F), dtype=t.bfloat16, device="cuda")
    Y = nan_like((w.T, w.h), t.bfloat16)
    with pytest.raises(mf.MemfineError) as ei:
        mf.memfine_moe_fwd_noalloc(s, 1, X, idx, g, W1, W2, Y)
    assert ei.value.code == mf.ERR_SCRATCH
    t.cuda.synchronize()
    assert bool(t.isnan(Y.float()).all())             # nothing ran
    # enough chunks make it fit
    C = next(c for c in (2, 4, 8, 16) if mf.memfine_workspace_bytes(s, c, mf.PASS_FWD)
             <= mf.NOALLOC_SCRATCH_BYTES)
    mf.memfine_moe_fwd_noalloc(s, C, X, idx, g, W1, W2, Y)
    t.cuda.synchronize()
    assert bool((Y.float() == 0).all())


def test_fwd_noalloc_expert_order(mf):
    """Expert-ordered chunks (launch option chunk_order): the layer's routing
    tables and the chunk's buffers both come from the static scratch; the
    same output, bit for bit, as the allocating forward in that order, and
    nothing allocated."""
    t = torch()
    stream = t.cuda.Stream()
    w = mw.scaled(mw.WORKLOADS[2], T=3000, h=512, F=384)
    case = mw.make_case(w, 73, with_dy=False)
    dev = device_case(w, case)
    try:
        mf.memfine_set_launch_options(chunk_order=mf.CHUNK_EXPERTS)
        for C in (2, 5):
            assert mf.memfine_workspace_bytes(shape_of(w), C, mf.PASS_FWD) <= mf.NOALLOC_SCRATCH_BYTES
            log(f"no-alloc forward, expert order, C={C}")
            Y_ref, Y = _fwd_both(mf, w, dev, C, stream)
            assert np.array_equal(Y, Y_ref)
            ref = om.moe_fwd(case["X"], case["idx"], case["gates"], case["W1"], case["W2"], C)
            assert relerr(Y, ref) <= TOL["bf16"]
    finally:
        mf.memfine_set_launch_options()
