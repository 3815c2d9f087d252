"""Decision margins, tie accounting and admissibility (test infrastructure only).

Routing indices and skip masks are compared bit-exactly, except on tokens whose
decisions sit within a band (1e-6) of a tie in the oracle's fp64 numbers.  A
token is tied when
  1. its k-th and (k+1)-th largest logits differ by less than the band
     (the top-k set is ambiguous), or
  2. two consecutive logits inside its top-k differ by less than the band
     (slot order, and so top-1, is ambiguous), or
  3. a non-top-1 slot has |c - tau| below the band (c < tau is the only skip
     decision, Eq. app_ace_skip_condition), or
  4. with m_min > 1, two non-top-1 contributions c are within the band (the
     restore order of Alg. 4 is ambiguous).
A tied token's GPU decisions must still be admissible: some resolution of
its near-ties must produce them.
"""
from __future__ import annotations

from itertools import combinations

import numpy as np

BAND = 1e-6


def _alg4_scores(g, a_gsp_e, a_rcr_e, eps, fusion="max"):
    from .forward import contributions
    return contributions(g, a_gsp_e, a_rcr_e, eps, fusion)[0]


def token_margins(z_row, idx_row, c_row, tau: float, m_min: int):
    """Smallest decision margins of one token (fp64 oracle values)."""
    z_row = np.asarray(z_row, dtype=np.float64)
    k = len(idx_row)
    zs = np.sort(z_row)[::-1]
    boundary = zs[k - 1] - zs[k] if k < len(zs) else np.inf
    ztop = z_row[np.asarray(idx_row)]
    order = np.min(ztop[:-1] - ztop[1:]) if k > 1 else np.inf
    c = np.asarray(c_row, dtype=np.float64)[1:]
    if np.isfinite(tau) and c.size:
        tau_m = np.min(np.abs(c - tau))
    else:
        tau_m = np.inf
    restore = np.inf
    if m_min > 1 and c.size > 1:
        cs = np.sort(c)
        restore = np.min(cs[1:] - cs[:-1])
    return dict(boundary=boundary, order=order, tau=tau_m, restore=restore)


def is_tied(m: dict, band: float = BAND) -> bool:
    return min(m.values()) < band


def admissible_token(z_row, pi_row, gpu_idx_row, gpu_keep_row, a_gsp, a_rcr, tau: float,
                     m_min: int, eps: float, band: float = BAND, fusion: str = "max"):
    """Can some resolution of the token's near-ties yield the GPU's decisions?"""
    z_row = np.asarray(z_row, dtype=np.float64)
    idx = np.asarray(gpu_idx_row, dtype=np.int64)
    keep = np.asarray(gpu_keep_row, dtype=bool)
    k = idx.size
    N = z_row.size
    if len(set(idx.tolist())) != k or idx.min() < 0 or idx.max() >= N:
        return False, "topk ids not distinct / out of range"
    zt = z_row[idx]
    if k > 1 and np.any(zt[:-1] < zt[1:] - band):
        return False, "slot order violates descending logits beyond the band"
    others = np.setdiff1d(np.arange(N), idx)
    if others.size and zt.min() < z_row[others].max() - band:
        return False, "top-k set excludes a clearly larger logit"
    if not keep[0]:
        return False, "top-1 slot skipped"
    top = np.asarray(pi_row, dtype=np.float64)[idx]
    g = top / top.sum()
    c = _alg4_scores(g, np.asarray(a_gsp, np.float64)[idx], np.asarray(a_rcr, np.float64)[idx], eps, fusion)
    skip_final = {i for i in range(1, k) if not keep[i]}
    # every non-top-1 slot is exactly one of: ambiguous (|c - tau| inside the band),
    # clearly skippable (c < tau outside the band) or clearly kept (c >= tau outside it)
    ambiguous = [i for i in range(1, k) if abs(c[i] - tau) < band]
    clear_skip = {i for i in range(1, k) if c[i] < tau and i not in ambiguous}
    for r in range(len(ambiguous) + 1):
        for extra in combinations(ambiguous, r):
            s0 = clear_skip | set(extra)            # one resolution of the strict c < tau tests
            need = max(0, m_min - (k - len(s0)))    # slots the m_min safeguard restores
            if not skip_final <= s0:
                continue
            restored = s0 - skip_final
            if len(restored) != need:
                continue
            # restore order: descending c, so no final skip may clearly beat a restored slot
            if all(c[a] >= c[b] - band for a in restored for b in skip_final):
                return True, "ok"
    return False, "keep mask not reachable from any near-tie resolution"


def compare_decisions(z, pi, oracle_idx, oracle_keep, c, gpu_idx, gpu_keep, a_gsp, a_rcr,
                      tau: float, m_min: int, eps: float, band: float = BAND, fusion: str = "max"):
    """Bit-exact comparison of routing and masks with tie accounting.

    Returns dict(n_tokens, tied [list of token ids], mismatch_untied [ids whose
    decisions differ without a tie], inadmissible [tied ids whose GPU decisions
    no near-tie resolution explains], differing_tied [tied ids that differ])."""
    T = len(oracle_idx)
    tied, mism, inadm, diff_tied = [], [], [], []
    for t in range(T):
        m = token_margins(z[t], oracle_idx[t], c[t], tau, m_min)
        same = (np.array_equal(np.asarray(gpu_idx[t]), np.asarray(oracle_idx[t]))
                and np.array_equal(np.asarray(gpu_keep[t], bool), np.asarray(oracle_keep[t], bool)))
        if is_tied(m, band):
            tied.append(t)
            if not same:
                diff_tied.append(t)
                ok, _ = admissible_token(z[t], pi[t], gpu_idx[t], gpu_keep[t], a_gsp, a_rcr,
                                         tau, m_min, eps, band, fusion)
                if not ok:
                    inadm.append(t)
        elif not same:
            mism.append(t)
    return dict(n_tokens=T, tied=tied, mismatch_untied=mism, inadmissible=inadm,
                differing_tied=diff_tied)
