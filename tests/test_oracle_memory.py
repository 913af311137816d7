"""Pins for the oracle's memory model and chunk planner (no GPU).

Checked against numbers the paper prints (tests/golden, each file cites its
table or section) and hand-worked Eq. (8)/(9) tables.
"""
import random
from fractions import Fraction

import pytest

from conftest import read_golden
from oracle import memory_model as mm


def test_table2_rows_sum_to_printed_total():
    """Table 2: the per-module rows must add up to the printed Total row, and
    Eq. (2) with m_g = 1 must equal that total."""
    total = {r[0]: [int(x) for x in r[1:]] for r in read_golden("table2_total.txt")}
    rng = random.Random(0)
    for _ in range(200):
        p = dict(D_t=rng.choice([1, 2, 4]), b=rng.randint(1, 4), s=rng.randint(1, 9000),
                 s_recv=rng.randint(0, 90000), h=rng.randint(1, 9000), a=rng.randint(1, 200),
                 h_d=rng.randint(1, 256), k_a=rng.randint(1, 200), e_n=rng.randint(1, 512),
                 g_e=rng.randint(1, 9000), t=rng.randint(1, 8), c=rng.randint(1, 4))
        rows = mm.table2_rows(**p)
        assert len(rows) == 14 and rows[7] == 0 and rows[14] == 0
        cs, cr = total["s"], total["s_recv"]
        printed = Fraction(p["D_t"] * p["b"], p["t"] * p["c"]) * (
            p["s"] * (cs[0] * p["h"] + cs[1] * p["a"] * p["h_d"] + cs[2] * p["k_a"] * p["h_d"]
                      + cs[3] * p["e_n"] + cs[4] * p["g_e"])
            + p["s_recv"] * (cr[0] * p["h"] + cr[1] * p["a"] * p["h_d"]
                             + cr[2] * p["k_a"] * p["h_d"] + cr[3] * p["e_n"] + cr[4] * p["g_e"]))
        assert sum(rows.values()) == printed
        eq2 = mm.activation_memory(1, p["t"], p["c"], p["D_t"], p["b"], p["s"], p["s_recv"],
                                   p["h"], p["a"], p["h_d"], p["k_a"], p["e_n"], p["g_e"])
        assert eq2 == printed
        # the MoE part (rows 11-13) is beta bytes per received slot
        moe = rows[11] + rows[12] + rows[13]
        assert moe == Fraction(p["b"] * p["s_recv"] * mm.moe_bytes_per_slot(p["D_t"], p["h"], p["g_e"]),
                               p["t"] * p["c"])


def test_beta_at_table3_shapes():
    for r in read_golden("table3_models.txt"):
        h, g_e = int(r[3]), int(r[6])
        assert mm.moe_bytes_per_slot(2, h, g_e) == 36864


def test_table4_rows_are_consistent():
    for model, method, sta, act, tot, trains in read_golden("table4_memory.txt"):
        assert abs(float(sta) + float(act) - float(tot)) < 0.05
    # Model I Method 1 does not train on a 64 GB GPU, the others do
    rows = {(r[0], r[1]): r for r in read_golden("table4_memory.txt")}
    assert rows[("I", "1")][5] == "0" and float(rows[("I", "1")][4]) > 64.0
    assert all(float(r[4]) <= 64.0 for key, r in rows.items() if key != ("I", "1"))


def test_section5_reductions():
    """The percentages printed in Section 5 follow from Table 4."""
    act = {r[1]: Fraction(r[3]) for r in read_golden("table4_memory.txt") if r[0] == "I"}
    for method, chunks, pct in read_golden("section5_reductions.txt"):
        got = mm.reduction(act["1"], act[method]) * 100
        assert abs(float(got) - float(pct)) < 0.005, (method, float(got), pct)


def test_chunked_peak_scales_like_table4():
    """Section 4.1: chunking replaces the layer's MoE peak by the largest
    chunk's.  Fitting A(C) = A0 + A1 * n(C)/n(1) through Table 4's C=1 and
    C=2 activation figures must reproduce its C=8 figure (to its rounding)."""
    act = {r[1]: float(r[3]) for r in read_golden("table4_memory.txt") if r[0] == "I"}
    T, k, beta = 4096 * 32, 8, 36864            # any T divisible by 8 works
    n = {C: mm.chunk_activation_bytes(T, k, C, beta) for C in (1, 2, 8)}
    A1 = (act["1"] - act["3"]) / (1 - n[2] / n[1])
    A0 = act["1"] - A1
    pred8 = A0 + A1 * n[8] / n[1]
    assert abs(pred8 - act["2"]) <= 0.05 + 1e-9


def test_plan_handworked():
    for s2, budget, c, C, ok in read_golden("plan_handworked.txt"):
        p = mm.plan([int(s2)], int(budget), 36864, bins=(1, 2, 4, 8, 16))
        assert p["c_theory"] == int(c) and p["C"] == int(C) and p["ok"] == bool(int(ok)), (s2, budget, p)


def test_plan_bins_methods():
    """Section 5: Method 2 is a fixed chunk count of 8 (bins {8}); Method 1 is
    no chunking (bins {1})."""
    for s2 in (1, 1000, 10**6):
        assert mm.plan([s2], 10**12, 36864, bins=(8,))["C"] == 8
        assert mm.plan([s2], 10**12, 36864, bins=(1,))["C"] == 1


def test_plan_exact_at_bin_edge():
    beta = 36864
    s2 = 65536
    # budget that fits exactly half of the slots: c = 2 exactly, not 3
    budget = s2 * beta // 2
    assert mm.plan([s2], budget, beta)["c_theory"] == 2
    assert mm.plan([s2], budget - 1, beta)["c_theory"] == 3


def test_plan_no_budget():
    p = mm.plan([100], 0, 36864, bins=(1, 2, 4, 8))
    assert p["C"] == 8 and not p["ok"]
    p = mm.plan([100], 1000, 36864, bins=(1, 2, 4, 8), fixed=1000)
    assert p["C"] == 8 and not p["ok"]


def test_eq8_matches_budget_form():
    """Eq. (8) with m_g=t=c=b=1 equals the planner's budget/beta form when the
    budget is alpha*M_GPU - M_sta - non-MoE term."""
    h, g_e, D_t, s, a, h_d, k_a, e_n = 7168, 2048, 2, 4096, 128, 128, 128, 256
    alpha, M_gpu, M_sta = Fraction(9, 10), 64 * 10**9, 43 * 10**9
    smax = mm.s_max(alpha, M_gpu, M_sta, 1, 1, 1, D_t, 1, s, h, a, h_d, k_a, e_n, g_e)
    non_moe = D_t * s * (5 * h + a * h_d + 2 * k_a * h_d + e_n)
    budget = alpha * M_gpu - M_sta - non_moe
    assert smax == budget / mm.moe_bytes_per_slot(D_t, h, g_e)
    # Eq. (3) holds at s' = floor(s'_max) and fails one slot above it
    sfl = int(smax)
    act = mm.activation_memory(1, 1, 1, D_t, 1, s, sfl, h, a, h_d, k_a, e_n, g_e)
    assert mm.fits(M_sta, act, alpha, M_gpu)
    act = mm.activation_memory(1, 1, 1, D_t, 1, s, sfl + 1, h, a, h_d, k_a, e_n, g_e)
    assert not mm.fits(M_sta, act, alpha, M_gpu)


def test_m_g():
    assert mm.m_g(full_recompute=True) == 1
    assert mm.m_g(v=1, p=4, r_pp=0, full_recompute=False) == 7   # v p + p - 2 r_pp - 1
    assert mm.m_g(v=1, p=4, r_pp=3, full_recompute=False) == 1


@pytest.mark.parametrize("T,C,expect", [(8, 3, 3), (8192, 4, 2048), (5, 8, 1), (10, 4, 3)])
def test_max_chunk_tokens(T, C, expect):
    assert mm.max_chunk_tokens(T, C) == expect


def _adam_state_bytes(sizes, copies):
    """Bytes a mixed-precision Adam training state holds for `copies` sets of
    weight tensors of the given element counts, measured on real tensors:
    bf16 weights with their bf16 gradients from a backward pass, fp32 master
    weights with fp32 gradients, and torch.optim.Adam's state after one step
    (its per-weight tensors; the scalar step counters are not per-weight
    memory)."""
    import torch
    torch.manual_seed(0)
    weights = [torch.randn(n, dtype=torch.bfloat16, requires_grad=True)
               for _ in range(copies) for n in sizes]
    sum((w.float() ** 2).sum() for w in weights).backward()
    master = [w.detach().float().clone().requires_grad_() for w in weights]
    for m, w in zip(master, weights):
        m.grad = w.grad.float()
    opt = torch.optim.Adam(master, lr=1e-3)
    opt.step()
    held = [*weights, *(w.grad for w in weights), *master, *(m.grad for m in master)]
    for m in master:
        held += [v for v in opt.state[m].values()
                 if torch.is_tensor(v) and v.shape == m.shape]
    assert all(t is not None for t in held)
    return sum(t.numel() * t.element_size() for t in held)


@pytest.mark.parametrize("sizes,v,l", [([128, 128, 8], 1, 1), ([96, 40, 7, 1], 2, 3),
                                       ([1000], 4, 1)])
def test_static_memory_is_mixed_precision_adam_state(sizes, v, l):
    """Eq. (1) against the memory that a bf16 model trained with Adam holds,
    counted on real tensors (torch on the CPU): weights (D_para = 2) and
    gradients (D_grad = 2) in bf16, and four fp32 copies per weight
    (D_opt = 4): the master weight, its gradient and Adam's two moment
    estimates.  v l copies of the modules' weights stand for the v virtual
    stages of l layers.  A wrong factor or a dropped term of Eq. (1) changes
    the count."""
    got = mm.static_memory(sizes, v, l)
    assert got == _adam_state_bytes(sizes, v * l)
    assert got == 20 * v * l * sum(sizes)
