"""Budget-to-threshold mapping of App. C.1 (test infrastructure only).

One unlabeled score pass collects the ACE contribution c of every routed
slot.  N_all counts every routed slot; N_cand excludes the slots the top-1
and minimum-active safeguards protect.  For a skip ratio q,
m_q = clip(round(q N_all), 0, N_cand), and tau is placed between the m_q-th
and (m_q+1)-th smallest candidate scores.

Readings where the appendix is not explicit:
  * round() is round-half-to-even (numpy's rint);
  * "between" is the midpoint of the two values;
  * m_q = 0 gives tau = 0 (nothing skipped, since c >= 0); m_q = N_cand gives
    tau = +inf (every candidate skipped);
  * on a tie at the boundary, tau goes just below the tied value (tau = v,
    realising #{c < v}) or just above it (midpoint to the next larger value,
    realising #{c <= v}), whichever realised count is closer to m_q, the lower
    count on a draw;
  * with m_min > 1 the protected slots are the top-1 slot and the m_min-1
    highest-c other slots of each token (ties to the lower slot index): the
    restore step of Alg. 4 never lets those be skipped, so the realised skip
    set is exactly {candidates with c < tau}.
"""
from __future__ import annotations

import numpy as np


def candidate_mask(c, m_min: int = 1):
    """[T,k] bool: True for slots that may be skipped (not top-1, not min-keep protected).
    Slot 0 is the top-1 slot (slots are in descending gate order)."""
    c = np.asarray(c, dtype=np.float64)
    T, k = c.shape
    cand = np.ones((T, k), dtype=bool)
    cand[:, 0] = False
    if m_min > 1:
        for t in range(T):
            others = sorted(range(1, k), key=lambda i: (-c[t, i], i))
            for i in others[: m_min - 1]:
                cand[t, i] = False
    return cand


def tau_for_budget(cand_scores, n_all: int, q: float) -> float:
    """tau_q from the collected candidate scores (App. C.1)."""
    s = np.sort(np.asarray(cand_scores, dtype=np.float64).ravel())
    n_cand = s.size
    m_q = int(np.clip(np.rint(q * n_all), 0, n_cand))
    if m_q == 0:
        return 0.0
    if m_q == n_cand:
        return float("inf")
    lo, hi = s[m_q - 1], s[m_q]           # c_(m_q), c_(m_q+1) in 1-based order
    if lo < hi:
        return 0.5 * (lo + hi)
    v = lo
    below = int(np.searchsorted(s, v, side="left"))     # #{c < v}
    above = int(np.searchsorted(s, v, side="right"))    # #{c <= v}
    if abs(below - m_q) <= abs(above - m_q):
        return float(v)
    if above == n_cand:
        return float("inf")
    return 0.5 * (v + s[above])


def tau_table(c_list, m_min: int, qs):
    """One score collection -> {q: tau} for every requested budget (App. C.1).

    c_list: iterable of [T,k] contribution arrays (one per layer); tau is global."""
    cands = []
    n_all = 0
    for c in c_list:
        c = np.asarray(c, dtype=np.float64)
        n_all += c.size
        cands.append(c[candidate_mask(c, m_min)])
    pool = np.concatenate(cands) if cands else np.zeros(0)
    return {q: tau_for_budget(pool, n_all, q) for q in qs}


def realised_skip_ratio(keep) -> float:
    """Fraction of routed top-k slots that are not executed (Sec. 4.1)."""
    keep = np.asarray(keep, dtype=bool)
    return float((~keep).sum()) / keep.size
