"""MACT from the model configuration (Section 3 and Section 4.2): the library's
host entry points against the oracle, and the oracle's threshold method
pinned against Eq. (9) + the bin choice and against Eq. (3).  No GPU."""
import itertools
import time
from fractions import Fraction

import numpy as np
import pytest

from oracle import memory_model as mm

BINS = (1, 2, 4, 8, 16)


@pytest.fixture(scope="module")
def mf():
    import paper_2511_21431_amd as m
    m.lib()
    return m


def model_I(**kw):
    """Model I of Table 3 with the paper's parallel setup (t = c = b = 1, p = 4,
    full recomputation); MLA-style k_a = a is a reading, e_n = 256 router
    logits."""
    d = dict(b=1, s=4096, h=7168, a=128, h_d=128, k_a=128, e_n=256, g_e=2048, t=1, c=1, v=1, p=4,
             D_t=2, full_recompute=1)
    d.update(kw)
    return d


def smax_of(d, r_pp, M_gpu, alpha, M_sta):
    m = mm.m_g(d["v"], d["p"], r_pp, bool(d["full_recompute"]))
    return mm.s_max(alpha, M_gpu, M_sta, m, d["t"], d["c"], d["D_t"], d["b"], d["s"], d["h"], d["a"],
                    d["h_d"], d["k_a"], d["e_n"], d["g_e"])


def act_of(d, r_pp, s_recv):
    m = mm.m_g(d["v"], d["p"], r_pp, bool(d["full_recompute"]))
    return mm.activation_memory(m, d["t"], d["c"], d["D_t"], d["b"], d["s"], s_recv, d["h"], d["a"],
                                d["h_d"], d["k_a"], d["e_n"], d["g_e"])


def random_models(n, seed):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        p = int(rng.integers(1, 9))
        yield dict(b=int(rng.integers(1, 5)), s=int(rng.integers(1, 8193)),
                   h=int(rng.integers(1, 9000)), a=int(rng.integers(1, 129)),
                   h_d=int(rng.integers(1, 257)), k_a=int(rng.integers(1, 129)),
                   e_n=int(rng.integers(0, 300)), g_e=int(rng.integers(1, 20000)),
                   t=int(rng.integers(1, 9)), c=int(rng.integers(1, 5)), v=int(rng.integers(1, 4)),
                   p=p, D_t=int(rng.choice([1, 2, 4])), full_recompute=int(rng.integers(0, 2)))


# ------------------------------------------------------- oracle pins
def test_threshold_method_equals_eq9_and_bins():
    """For every s'' the threshold lookup picks the bin that Eq. (9) followed
    by the smallest-bin->=c choice picks (two different formulations)."""
    for smax in (Fraction(1), Fraction(7, 3), Fraction(1000), Fraction(12345, 7), Fraction(0)):
        th = mm.mact_thresholds(smax, BINS)
        top = 20 * max(1, int(smax) + 1)
        for s2 in range(0, top):
            got = mm.mact_select(BINS, th, s2)
            if smax == 0:
                want = (min(BINS), True) if s2 == 0 else (max(BINS), False)
            else:
                want = mm.select_bin(mm.theoretical_chunks(s2, smax), BINS) if s2 else (min(BINS), True)
            assert got == want, (smax, s2, got, want)


def test_selected_bin_keeps_eq3_and_smaller_bin_breaks_it():
    """Chunking s'' slots into C leaves s''/C live (Section 4.1): the chosen C
    satisfies Eq. (3) exactly, and the next smaller bin does not."""
    alpha, M_gpu = Fraction(9, 10), 64 * 10**9
    for d in itertools.islice(random_models(200, 5), 200):
        for r in {0, d["p"] - 1}:
            M_sta = 10**9
            smax = smax_of(d, r, M_gpu, alpha, M_sta)
            th = mm.mact_thresholds(smax, BINS)
            for s2 in (0, 1, 1000, 65536, 10**6):
                C, ok = mm.mact_select(BINS, th, s2)
                fits = mm.fits(M_sta, act_of(d, r, Fraction(s2, C)), alpha, M_gpu)
                assert fits == ok
                smaller = [b for b in BINS if b < C]
                if ok and smaller:
                    assert not mm.fits(M_sta, act_of(d, r, Fraction(s2, max(smaller))), alpha, M_gpu)


def test_pipeline_rank_pressure():
    """Without full recomputation, m_g = v p + p - 2 r - 1 shrinks with the
    rank: earlier stages hold more micro-batches and get lower thresholds."""
    d = model_I(full_recompute=0, s=1024)
    th = [mm.mact_thresholds(smax_of(d, r, 64 * 10**9, Fraction(9, 10), 30 * 10**9), BINS)
          for r in range(d["p"])]
    for r in range(d["p"] - 1):
        assert all(a <= b for a, b in zip(th[r], th[r + 1]))
    assert th[0][0] < th[-1][0]


# ------------------------------------------------------- library vs oracle
def test_activation_memory_matches_oracle(mf):
    for d in random_models(300, 11):
        m = mf.make_model(**d)
        for r in range(d["p"]):
            if mm.m_g(d["v"], d["p"], r, bool(d["full_recompute"])) < 1:
                continue
            for s2 in (0, 1, 4097, 10**6):
                want = act_of(d, r, s2)
                want = -((-want.numerator) // want.denominator)     # whole bytes, rounded up
                assert mf.memfine_activation_memory(m, r, s2) == want


def test_thresholds_and_select_match_oracle(mf):
    rng = np.random.default_rng(3)
    for d in random_models(300, 17):
        m = mf.make_model(**d)
        r = int(rng.integers(0, d["p"]))
        if mm.m_g(d["v"], d["p"], r, bool(d["full_recompute"])) < 1:
            continue
        M_gpu = int(rng.integers(10**9, 300 * 10**9))
        an, ad = int(rng.integers(1, 100)), 100
        M_sta = int(rng.integers(0, M_gpu))
        got = mf.memfine_mact_thresholds(m, r, M_gpu, an, ad, M_sta, BINS)
        want = mm.mact_thresholds(smax_of(d, r, M_gpu, Fraction(an, ad), M_sta), BINS)
        assert got == want
        for s2 in {0, 1, *[max(0, x) for x in want], *[x + 1 for x in want if x >= 0]}:
            rc, C = mf.memfine_mact_select(BINS, got, s2)
            C2, ok = mm.mact_select(BINS, want, s2)
            assert C == C2 and (rc == 0) == ok


def test_static_memory_matches_oracle(mf):
    rng = np.random.default_rng(23)
    for _ in range(200):
        S = rng.integers(0, 10**9, size=int(rng.integers(0, 12))).tolist()
        v, l = int(rng.integers(1, 4)), int(rng.integers(1, 17))
        D = [int(x) for x in rng.choice([1, 2, 4], size=3)]
        assert mf.memfine_static_memory(S, v, l, *D) == mm.static_memory(S, v, l, *D)


def test_mact_errors(mf):
    m = mf.make_model(**model_I())
    with pytest.raises(mf.MemfineError):
        mf.memfine_activation_memory(m, 4, 10)            # rank outside [0, p)
    with pytest.raises(mf.MemfineError):
        mf.memfine_activation_memory(mf.make_model(**model_I(t=0)), 0, 10)
    with pytest.raises(mf.MemfineError):
        mf.memfine_mact_thresholds(m, 0, 10**10, 9, 0, 0, BINS)   # alpha_den = 0
    with pytest.raises(mf.MemfineError):
        mf.memfine_mact_thresholds(m, 0, 10**10, 9, 10, 0, (1, 0))
    with pytest.raises(mf.MemfineError):
        mf.memfine_static_memory([1, -2], 1, 1)
    with pytest.raises(mf.MemfineError):
        mf.memfine_static_memory([2**62, 2**62], 1, 1)     # beyond int64
    # the fixed part alone over budget: nothing fits, largest bin + budget error
    th = mf.memfine_mact_thresholds(m, 0, 10**9, 1, 1, 10**9, BINS)
    assert th == [-1] * len(BINS)
    assert mf.memfine_mact_select(BINS, th, 0) == (-3, max(BINS))


# ------------------------------------------------------- replay
def skew_schedule(iters=30, layers=16, base=32768, peak=1048576):
    """Synthetic received-slot counts per (iteration, layer) with the shape the
    paper describes for its runs: imbalance grows with depth and peaks early
    in training (iterations ~5-15), then the distribution settles."""
    out = np.zeros((iters, layers), dtype=np.int64)
    for i in range(iters):
        burst = np.exp(-((i - 10) / 4.0) ** 2)
        for l in range(layers):
            depth = (l / (layers - 1)) ** 2
            out[i, l] = min(peak, int(base * (1 + (peak / base - 1) * depth * burst)))
    return out


def test_replay_skew_schedule(mf):
    """Per-iteration, per-layer MACT over a synthetic skew schedule on Model I
    (16 layers on p = 4 stages, 64 GB GPUs, alpha = 0.9, 43 GB static as in
    Table 4): every choice keeps Eq. (3); larger chunk counts appear in the
    later layers during the imbalanced iterations and vanish afterwards; the
    fixed C = 1 method breaks Eq. (3) exactly where MACT chunks."""
    d = model_I()
    m = mf.make_model(**d)
    M_gpu, an, ad, M_sta = 64 * 10**9, 9, 10, 43 * 10**9
    th = {r: mf.memfine_mact_thresholds(m, r, M_gpu, an, ad, M_sta, BINS) for r in range(d["p"])}
    sched = skew_schedule()
    C = np.zeros_like(sched)
    t0 = time.perf_counter()
    for (i, l), s2 in np.ndenumerate(sched):
        rc, C[i, l] = mf.memfine_mact_select(BINS, th[l // 4], int(s2))
        assert rc == 0
    per_call_us = (time.perf_counter() - t0) / sched.size * 1e6
    print(f"mact_select: {per_call_us:.2f} us per call (ctypes included)")
    for (i, l), s2 in np.ndenumerate(sched):
        act = act_of(d, l // 4, Fraction(int(s2), int(C[i, l])))
        assert mm.fits(M_sta, act, Fraction(an, ad), M_gpu)
        one_fits = mm.fits(M_sta, act_of(d, l // 4, int(s2)), Fraction(an, ad), M_gpu)
        assert one_fits == (C[i, l] == 1)
    early, late = C[5:16, :8], C[5:16, 8:]
    assert late.mean() > early.mean() and C.max() > 1
    assert (C[25:] == 1).all() and (C[:2] == 1).all()


@pytest.mark.gpu
def test_mact_model_I_in_the_gpu_suite(mf):
    """The library's MACT entry points for Model I at every pipeline rank,
    with and without full recomputation, against the oracle (the same check
    smoke() runs)."""
    import __graft_entry__ as entry
    entry._smoke_mact(mf)
