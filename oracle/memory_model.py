"""The paper's memory cost model and MACT chunk choice (test infrastructure only).

Everything is exact (``fractions.Fraction`` / Python integers) so that bin
edges are decided without rounding.

Passages followed
-----------------
* Section 3, Eq. (1): static memory = parameters + gradients + 4x optimizer
  states, each D * v * l * sum(S_i).
* Section 3, Table 2: stored activation bytes per module of one MoE
  transformer layer; rows 11-13 are the activated expert's input
  (D_t b s' h), its FC1 output (2 D_t b s' g_e) and the score-multiply input
  (D_t b s' h), all divided by t*c.
* Section 3, Eq. (2): peak activation = m_g/(t c) * D_t b (s(5h + a h_d +
  2 k_a h_d + e_n) + s'(2h + 2 g_e)); m_g = v p + p - 2 r_pp - 1, and 1 under
  full recomputation.
* Section 3, Eq. (3): feasibility M_sta + M_act <= alpha * M_GPU.
* Section 4.2, Eq. (8): s'_max, the most received slots the budget allows;
  Eq. (9): c = ceil(s'' / s'_max); then the chunk count is taken from a set of
  bins.
* Section 4.2, threshold method: before training, each pipeline stage turns
  Eq. (8) into one s'' threshold per bin; at run time the chunk count is the
  smallest bin whose threshold admits the received slots.
* Section 4.1: the chunked layer's peak is the largest chunk's activation.

Readings (the paper is ambiguous here)
--------------------------------------
* s' and s'' count token-slots (rows after dispatch), not distinct tokens.
* Section 4.2's bin choice after Eq. (9) (a bin near c, on the large side)
  is read as the smallest bin >= c, so that the chosen chunk count keeps the
  chunk under the budget; when no bin is large enough the largest bin is
  returned with a budget error.
* The planner's budget is the numerator of Eq. (8) (alpha*M_GPU - M_sta -
  the non-MoE activation term), minus an optional fixed allowance, for one
  layer with m_g = t = c = b = 1.
* Table 2 glosses e_n as an FFN size, but it sits in the router-output row;
  it is read as the router's logit width.  It only enters the non-MoE term.
* Eq. (1)'s four optimizer-state copies of D_opt bytes per weight are read
  as the fp32 state mixed-precision Adam keeps per bf16 weight: the master
  weight, its gradient and the two moment estimates (D_para = D_grad = 2,
  D_opt = 4: 20 bytes per weight).

Pins: Eq. (1) equals the bytes a bf16 model trained with Adam holds, counted
on real tensors after one optimizer step (the reading above); Table 2's
rows must add up to its printed Total row and to Eq. (2);
the Table 4 percentages printed in Section 5 (48.03 %, 83.84 %); the 1/C
scaling of the chunked MoE term against Table 4's three activation figures;
hand-worked Eq. (8)/(9) tables; the threshold method selects, for every s'',
the same bin as Eq. (9) followed by the bin choice, and that bin keeps Eq. (3)
while the next smaller one breaks it.  The absolute 22.9 GB of Table 4 is
parity unpinned: the received-slot count and the attention shapes of that
run are not printed.  So are Table 4's absolute static-memory figures: the
per-module weight sizes and layer placement behind them are not printed.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Dict, Iterable, Optional, Sequence, Tuple


def _F(x) -> Fraction:
    return x if isinstance(x, Fraction) else Fraction(x)


# --- Eq. (1) ----------------------------------------------------------------
def static_memory(S_para: Iterable[int], v: int, l: int,
                  D_para: int = 2, D_grad: int = 2, D_opt: int = 4) -> Fraction:
    """Eq. (1): weights + gradients + four optimizer-state copies, over the
    v l copies of the modules' weights S_i held by one GPU."""
    S = sum(_F(s) for s in S_para)
    return D_para * v * l * S + D_grad * v * l * S + 4 * D_opt * v * l * S


# --- Table 2 ------------------------------------------------------------------
def table2_rows(D_t, b, s, s_recv, h, a, h_d, k_a, e_n, g_e, t=1, c=1) -> Dict[int, Fraction]:
    """Stored activation bytes of Table 2, by input ID (7 and 14 store none)."""
    D_t, b, s, sr = _F(D_t), _F(b), _F(s), _F(s_recv)
    tc = _F(t) * _F(c)
    rows = {
        1: D_t * b * s * h,            # norm
        2: D_t * b * s * h,            # q, k, v
        3: D_t * b * s * a * h_d,      # attention (queries)
        4: D_t * b * s * k_a * h_d,    # attention (keys)
        5: D_t * b * s * k_a * h_d,    # attention (values)
        6: D_t * b * s * h,            # o
        7: Fraction(0),                # add
        8: D_t * b * s * h,            # norm
        9: D_t * b * s * h,            # router input
        10: D_t * b * s * e_n,         # router output
        11: D_t * b * sr * h,          # activated expert input
        12: 2 * D_t * b * sr * g_e,    # activated expert FC1 output (2 g_e)
        13: D_t * b * sr * h,          # score-mul input
        14: Fraction(0),               # add
    }
    return {key: val / tc for key, val in rows.items()}


def moe_bytes_per_slot(D_t: int, h: int, g_e: int) -> int:
    """Bytes Table 2 stores per received slot: rows 11-13 = D_t (2h + 2 g_e)."""
    return D_t * (2 * h + 2 * g_e)


# --- Eq. (2) ------------------------------------------------------------------
def m_g(v: int = 1, p: int = 1, r_pp: int = 0, full_recompute: bool = True) -> int:
    """Stored-activation multiplicity under pipeline parallelism (Section 3)."""
    return 1 if full_recompute else v * p + p - 2 * r_pp - 1


def activation_memory(m, t, c, D_t, b, s, s_recv, h, a, h_d, k_a, e_n, g_e) -> Fraction:
    """Eq. (2): peak activation bytes."""
    non_moe = _F(s) * (5 * h + a * h_d + 2 * k_a * h_d + e_n)
    moe = _F(s_recv) * (2 * h + 2 * g_e)
    return Fraction(m, t * c) * D_t * b * (non_moe + moe)


# --- Eq. (3) ------------------------------------------------------------------
def fits(M_sta, M_act, alpha, M_gpu) -> bool:
    """Eq. (3)."""
    return _F(M_sta) + _F(M_act) <= _F(alpha) * _F(M_gpu)


# --- Eq. (8), Eq. (9), bins -----------------------------------------------------
def s_max(alpha, M_gpu, M_sta, m, t, c, D_t, b, s, h, a, h_d, k_a, e_n, g_e) -> Fraction:
    """Eq. (8): most received slots that still satisfy Eq. (3)."""
    scale = Fraction(m, t * c) * D_t * b
    num = _F(alpha) * _F(M_gpu) - _F(M_sta) - scale * s * (5 * h + a * h_d + 2 * k_a * h_d + e_n)
    return num / (scale * (2 * h + 2 * g_e))


def theoretical_chunks(s2: int, smax: Fraction) -> int:
    """Eq. (9): c = ceil(s'' / s'_max), with s'_max > 0."""
    q = Fraction(s2) / _F(smax)
    return -((-q.numerator) // q.denominator)


def select_bin(c: int, bins: Sequence[int]) -> Tuple[int, bool]:
    """Smallest bin >= c; (max(bins), False) when none is large enough."""
    ok = sorted(b for b in bins if b >= c)
    if ok:
        return ok[0], True
    return max(bins), False


def plan(counts: Sequence[int], budget: int, beta: int,
         bins: Sequence[int] = (1, 2, 4, 8), fixed: int = 0) -> Dict[str, object]:
    """MACT for one layer: s'' from the expert counts, s'_max = (budget -
    fixed) / beta (Eq. (8) with m_g = t = c = b = 1 and the non-MoE term
    folded into the budget), c by Eq. (9), the chunk count from the bins.

    Returns dict(C, ok, c_theory, s2, s_max)."""
    s2 = int(sum(int(x) for x in counts))
    avail = int(budget) - int(fixed)
    if avail <= 0:
        return {"C": max(bins), "ok": False, "c_theory": None, "s2": s2, "s_max": Fraction(0)}
    smax = Fraction(avail, int(beta))
    c = theoretical_chunks(s2, smax)
    C, ok = select_bin(c, bins)
    return {"C": C, "ok": ok, "c_theory": c, "s2": s2, "s_max": smax}


# --- MACT's threshold method (Section 4.2) ---------------------------------------
def mact_thresholds(smax: Fraction, bins: Sequence[int]) -> List[int]:
    """Before training, per pipeline stage: for every bin, the largest s''
    that the bin's chunk count keeps within Eq. (3).  Splitting s'' received
    slots into b chunks leaves s''/b of them live, so bin b admits s'' while
    s''/b <= s'_max, i.e. s'' <= floor(b s'_max); a negative s'_max (the part
    of Eq. (2) that does not depend on s'' already breaks Eq. (3)) admits
    nothing (-1)."""
    smax = _F(smax)
    if smax < 0:
        return [-1 for _ in bins]
    return [int((b * smax).numerator // (b * smax).denominator) for b in bins]


def mact_select(bins: Sequence[int], thresholds: Sequence[int], s2: int) -> Tuple[int, bool]:
    """At run time: the smallest bin whose threshold admits s''; (max(bins),
    False) when none does."""
    ok = [b for b, th in zip(bins, thresholds) if s2 <= th]
    if ok:
        return min(ok), True
    return max(bins), False


# --- the chunked layer's peak (Section 4.1) -------------------------------------
def max_chunk_tokens(T: int, C: int) -> int:
    """Largest chunk of the floor-balanced split of T tokens into C chunks."""
    return max(((i + 1) * T) // C - (i * T) // C for i in range(C))


def chunk_activation_bytes(T: int, k: int, C: int, beta: int) -> int:
    """Peak MoE activation of the chunked layer: beta bytes for every slot of
    the largest chunk (the maximum over chunks replaces the whole layer)."""
    return beta * max_chunk_tokens(T, C) * k


def reduction(before, after) -> Fraction:
    """Relative saving (before - after) / before."""
    return (_F(before) - _F(after)) / _F(before)
