"""Every GEMM launch configuration computes the same numbers.

Each output element of every grouped GEMM is one thread's fp32 sum over K in
increasing K order (MFMA steps of 16 or 2), whatever the tile shape, the tile
order over the chip (XCD blocks, row-major), the persistent or one-tile-per-
workgroup launch, the quarter-tile tail, the paired dgrad/wgrad launch or
the side-stream schedule.  So all of them must give bit-identical outputs
and gradients; the default configuration is checked against the oracle in
test_gpu_parity.py.  The options are set through memfine_set_launch_options
(a layer call reads them once when it starts).
"""
import numpy as np
import pytest

import moe_workloads as mw
from gpu_harness import device_case, host, log, run_bwd, run_fwd, torch

pytestmark = pytest.mark.gpu

# large enough for the 256 x 256 tiles' persistent and split-tail launches
# (FC1: 64 m-tiles x 8 n-tiles at C = 1), ragged per expert
W_BIG = mw.scaled(mw.WORKLOADS[2], T=4096, h=512, F=1024, E=8)
W_F32 = mw.WORKLOADS[1]

# memfine_set_launch_options keyword arguments
CONFIGS = ([{"raster": r} for r in range(5)]
           + [{"tile": t} for t in (1, 2, 3)]
           + [{"split_tail": False}, {"pair": True}, {"streams": True},
              {"split_tail": False, "raster": 2}, {"tile": 3, "raster": 0}])


def _ids(c):
    return ",".join(f"{k}={v}" for k, v in c.items())


@pytest.fixture(scope="module")
def mf():
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_21431_amd as m
    m.lib()
    return m


def _run(w, dev, C):
    Y = host(run_fwd(w, dev, C))
    B = {k: host(v) for k, v in run_bwd(w, dev, C).items()}
    return {"Y": Y, **B}


_cache = {}


def _reference(w, seed, C):
    key = (w.name, seed, C)
    if key not in _cache:
        import paper_2511_21431_amd as m
        m.memfine_set_launch_options()
        case = mw.make_case(w, seed)
        dev = device_case(w, case)
        _cache[key] = (dev, _run(w, dev, C))
    return _cache[key]


@pytest.mark.parametrize("C", [1, 3])
@pytest.mark.parametrize("cfg", CONFIGS, ids=_ids)
def test_bitwise_across_launch_configs(mf, cfg, C):
    dev, ref = _reference(W_BIG, 61, C)
    log(f"launch config {cfg} C={C}")
    try:
        mf.memfine_set_launch_options(**cfg)
        got = _run(W_BIG, dev, C)
    finally:
        mf.memfine_set_launch_options()
    for key in ref:
        assert np.array_equal(got[key], ref[key]), (cfg, C, key)


@pytest.mark.parametrize("cfg", [{"raster": 3}, {"split_tail": False}, {"streams": True}], ids=_ids)
def test_bitwise_across_launch_configs_f32(mf, cfg):
    dev, ref = _reference(W_F32, 5, 2)
    log(f"launch config f32 {cfg}")
    try:
        mf.memfine_set_launch_options(**cfg)
        got = _run(W_F32, dev, 2)
    finally:
        mf.memfine_set_launch_options()
    for key in ref:
        assert np.array_equal(got[key], ref[key]), (cfg, key)
