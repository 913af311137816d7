"""Pins for the oracle's chunking and dispatch (no GPU).

The oracle's dispatch (a stable grouping of slots by expert) is checked
against a brute-force double loop written here, and against the invariants a
grouping must satisfy; the chunk split against the Eq. (6) properties.
"""
import numpy as np
import pytest

from oracle import moe as om


def brute_dispatch(idx, t0, t1, E):
    k = len(idx[0])
    sorted_slot = []
    counts = []
    for e in range(E):
        c = 0
        for t in range(t0, t1):
            for j in range(k):
                if int(idx[t][j]) == e:
                    sorted_slot.append(t * k + j)
                    c += 1
        counts.append(c)
    row_of_slot = [None] * ((t1 - t0) * k)
    for r, s in enumerate(sorted_slot):
        row_of_slot[s - t0 * k] = r
    return counts, sorted_slot, row_of_slot


@pytest.mark.parametrize("seed", range(6))
def test_dispatch_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 40))
    k = int(rng.integers(1, 5))
    E = int(rng.integers(1, 9))
    idx = rng.integers(0, E, size=(T, k))
    t0 = int(rng.integers(0, T))
    t1 = int(rng.integers(t0 + 1, T + 1))
    d = om.dispatch(idx, t0, t1, E)
    counts, sorted_slot, row_of_slot = brute_dispatch(idx.tolist(), t0, t1, E)
    assert d["counts"].tolist() == counts
    assert d["sorted_slot"].tolist() == sorted_slot
    assert d["row_of_slot"].tolist() == row_of_slot
    assert d["offsets"][0] == 0 and d["offsets"][-1] == (t1 - t0) * k


def test_dispatch_invariants_large():
    rng = np.random.default_rng(7)
    T, k, E = 3000, 8, 32
    idx = rng.integers(0, E, size=(T, k))
    t0, t1 = 517, 2911
    d = om.dispatch(idx, t0, t1, E)
    n = (t1 - t0) * k
    ss, rs, off = d["sorted_slot"], d["row_of_slot"], d["offsets"]
    assert d["counts"].sum() == n
    assert np.all(np.diff(off) >= 0)
    ex = idx.reshape(-1)[ss]
    assert np.all(np.diff(ex) >= 0)                      # grouped by expert
    for e in range(E):                                   # stable inside a group
        seg = ss[off[e]:off[e + 1]]
        assert np.all(np.diff(seg) > 0)
        assert np.all(ex[off[e]:off[e + 1]] == e)
    assert np.array_equal(ss[rs], t0 * k + np.arange(n))  # inverse
    assert sorted(ss.tolist()) == list(range(t0 * k, t1 * k))


def test_expert_counts():
    idx = np.array([[0, 2], [2, 2], [1, 0]])
    assert om.expert_counts(idx, 4).tolist() == [2, 1, 3, 0]


@pytest.mark.parametrize("T,C", [(10, 1), (10, 3), (10, 4), (7, 7), (5, 8), (256, 4), (8191, 16)])
def test_chunk_ranges(T, C):
    r = om.chunk_ranges(T, C)
    # contiguous, disjoint, covering [0, T)
    assert r[0][0] == 0 and r[-1][1] == T
    for (a0, a1), (b0, b1) in zip(r, r[1:]):
        assert a1 == b0
    sizes = [b - a for a, b in r]
    assert all(s > 0 for s in sizes)
    assert max(sizes) - min(sizes) <= 1
    assert len(r) == min(C, T)
