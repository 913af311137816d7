"""The seeded input generator: exact counts, determinism, bf16 values."""
import numpy as np
import pytest

import moe_workloads as mw


def test_largest_remainder():
    c = mw.largest_remainder([0.5, 0.25, 0.25], 7)
    assert c.sum() == 7 and c.tolist() == [3, 2, 2]


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_routing_shapes_and_determinism(cfg):
    w = mw.WORKLOADS[cfg]
    if cfg >= 3:
        w = mw.scaled(w, T=512)
    idx, g = mw.make_routing(w, seed=cfg)
    idx2, g2 = mw.make_routing(w, seed=cfg)
    assert idx.shape == (w.T, w.k) and idx.dtype == np.int32
    assert np.array_equal(idx, idx2) and np.array_equal(g, g2)
    assert idx.min() >= 0 and idx.max() < w.E
    assert np.allclose(g.sum(1), 1.0, atol=1e-6)


def test_hot_expert_share():
    w = mw.WORKLOADS[4]
    idx, _ = mw.make_routing(w, seed=4)
    counts = np.bincount(idx.reshape(-1), minlength=w.E)
    assert counts.sum() == w.N and counts.max() == w.N // 4   # 8x the mean of N/32


def test_zipf_share():
    w = mw.WORKLOADS[3]
    idx, _ = mw.make_routing(mw.scaled(w, T=4096), seed=3)
    counts = np.bincount(idx.reshape(-1), minlength=w.E)
    assert 3.3 < counts.max() / counts.mean() < 3.6


def test_bf16_rounding():
    x = np.array([1.0, 1.00390625, 1.005859375, -3.14159, 65504.0], dtype=np.float32)
    r = mw.round_to_bf16(x)
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    assert r[1] == 1.0                 # tie -> even
    assert r[2] == np.float32(1.0078125)
    t = mw.make_tensors(mw.scaled(mw.WORKLOADS[2], T=64, h=128, F=64, E=2), seed=0)
    for v in t.values():
        assert np.all((v.view(np.uint32) & 0xFFFF) == 0)
