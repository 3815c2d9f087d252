"""Plant plausible mistakes in the CPU oracle and confirm that the pins catch
each one (a dropped term, a wrong sign, order or index, a swapped operand).
Every mutant lives only inside this test, on the CPU."""
from itertools import combinations

import numpy as np
import pytest

import oracle
import oracle_pins as P

F = oracle.forward
TB = oracle.tables
TAU = oracle.tau
PL = oracle.plan
TIES = oracle.ties


def _rms_abs(x, gamma, rms_eps):
    x = np.asarray(x, float)
    return x / np.sqrt(np.mean(np.abs(x), axis=-1, keepdims=True) + rms_eps) * gamma


def _rms_no_gamma(x, gamma, rms_eps):
    x = np.asarray(x, float)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + rms_eps)


def _topk_high_id(z_row, k):
    z_row = np.asarray(z_row, float)
    ids = sorted(range(len(z_row)), key=lambda e: (-z_row[e], -e))
    return np.array(ids[:k])


def _route_no_renorm(x_in, w_router, b_router, k):
    z = F.router_logits(x_in, w_router, b_router)
    pi = F.softmax(z)
    idx = np.stack([F.topk_order(z[t], k) for t in range(len(z))])
    g = np.take_along_axis(pi, idx, 1)
    return z, pi, idx, g


def _skip_variant(kind):
    orig = F.ace_skip

    def fn(g, a_gsp_e, a_rcr_e, tau, m_min, eps, fusion="max"):
        g = np.asarray(g, float)
        k = len(g)
        s_g, s_r = g * a_gsp_e, g * a_rcr_e
        if kind == "no_eps_in_p":
            p_g, p_r = s_g / s_g.sum(), s_r / s_r.sum()
        else:
            p_g, p_r = s_g / (s_g.sum() + eps), s_r / (s_r.sum() + eps)
        c = np.minimum(p_g, p_r) if kind == "union" else np.maximum(p_g, p_r)
        lt = (lambda a: a <= tau) if kind == "non_strict" else (lambda a: a < tau)
        sg = {i for i in range(k) if lt(p_g[i])}
        sr = {i for i in range(k) if lt(p_r[i])}
        skip = (sg | sr) if kind == "union" else (sg & sr)
        if kind != "no_top1":
            skip.discard(0)
        active = set(range(k)) - skip
        if len(active) < m_min:
            order = sorted(skip, key=lambda i: (c[i], i) if kind == "restore_ascending" else (-c[i], i))
            for i in order[: m_min - len(active)]:
                skip.discard(i)
                active.add(i)
        zg = sum(g[i] for i in active) + (0.0 if kind == "no_eps_final" else eps)
        ghat = np.zeros(k)
        for i in active:
            ghat[i] = g[i] / zg
        return dict(keep=np.array([i in active for i in range(k)]), ghat=ghat, c=c, p_gsp=p_g,
                    p_rcr=p_r, s_gsp_set=sg, s_rcr_set=sr, skip_set=skip)
    fn.orig = orig
    return fn


def _contrib_variant(kind):
    orig = F.contributions

    def fn(g, a_gsp_e, a_rcr_e, eps, fusion="max"):
        c, p_g, p_r = orig(g, a_gsp_e, a_rcr_e, eps, fusion)
        if kind == "min_is_max" and fusion == "min":
            c = np.maximum(p_g, p_r)
        elif kind == "mean_no_half" and fusion == "mean":
            c = p_g + p_r
        elif kind == "score_is_gsp" and fusion == "score":
            c = p_g
        elif kind == "rcr_is_gsp" and fusion == "rcr":
            c = p_g
        return c, p_g, p_r
    return fn


def _ffn_silu_on_up(x, wg, wu, wd):
    x = np.asarray(x, float)
    return np.asarray(wd, float) @ ((np.asarray(wg, float) @ x) * F.silu(np.asarray(wu, float) @ x))


def _ffn_relu(x, wg, wu, wd):
    x = np.asarray(x, float)
    return np.asarray(wd, float) @ (np.maximum(np.asarray(wg, float) @ x, 0) * (np.asarray(wu, float) @ x))


def _gsp_up_only(gamma, wg, wu, wd):
    gam = np.asarray(gamma, float)
    G, U = np.asarray(wg, float) * gam, np.asarray(wu, float) * gam
    return np.linalg.norm(U) * np.linalg.norm(np.asarray(wd, float) @ G)


def _gsp_no_gamma(gamma, wg, wu, wd):
    G, U, Wd = np.asarray(wg, float), np.asarray(wu, float), np.asarray(wd, float)
    return np.sqrt(np.linalg.norm(U) * np.linalg.norm(Wd @ G) * np.linalg.norm(G) * np.linalg.norm(Wd @ U))


def _gsp_swapped_paths(gamma, wg, wu, wd):
    gam = np.asarray(gamma, float)
    G, U, Wd = np.asarray(wg, float) * gam, np.asarray(wu, float) * gam, np.asarray(wd, float)
    return np.sqrt(np.linalg.norm(G) * np.linalg.norm(Wd @ G) * np.linalg.norm(U) * np.linalg.norm(Wd @ G))


def _proto_uncentred(w_router, eps=1e-6, rho=1.0):
    W = np.asarray(w_router, float)
    r = np.sqrt(np.mean(W * W, axis=1, keepdims=True))
    return rho * W / (r + eps)


def _proto_l2(w_router, eps=1e-6, rho=1.0):
    W = np.asarray(w_router, float)
    wt = W - W.mean(0)
    return rho * wt / (np.linalg.norm(wt, axis=1, keepdims=True) + eps)


def _tau_floor(cand_scores, n_all, q):
    s = np.sort(np.asarray(cand_scores, float).ravel())
    m_q = int(np.clip(np.floor(q * n_all), 0, s.size))
    if m_q == 0:
        return 0.0
    if m_q == s.size:
        return float("inf")
    return 0.5 * (s[m_q - 1] + s[m_q])


def _tau_off_by_one(cand_scores, n_all, q):
    s = np.sort(np.asarray(cand_scores, float).ravel())
    m_q = int(np.clip(np.rint(q * n_all), 0, s.size))
    if m_q == 0:
        return 0.0
    if m_q >= s.size - 1:
        return float("inf")
    return 0.5 * (s[m_q] + s[m_q + 1])


def _plan_token_desc(topk_idx, keep, N):
    idx = np.asarray(topk_idx)
    keep = np.asarray(keep, bool)
    T, k = idx.shape
    pairs = sorted((int(idx[t, i]), -t, i) for t in range(T) for i in range(k) if keep[t, i])
    counts = np.bincount([e for e, _, _ in pairs], minlength=N)
    offsets = np.concatenate([[0], np.cumsum(counts)])
    slot_row = np.full((T, k), -1)
    for r, (_, nt, i) in enumerate(pairs):
        slot_row[-nt, i] = r
    return dict(counts=counts, offsets=offsets, perm=np.array([-nt for _, nt, _ in pairs]),
                slot_row=slot_row)


def _margins_variant(kind):
    def fn(z_row, idx_row, c_row, tau, m_min):
        z_row = np.asarray(z_row, float)
        k = len(idx_row)
        zs = np.sort(z_row)[::-1]
        if kind == "boundary_off_by_one":
            boundary = zs[k] - zs[k + 1] if k + 1 < len(zs) else np.inf
        else:
            boundary = zs[k - 1] - zs[k] if k < len(zs) else np.inf
        ids = np.sort(np.asarray(idx_row)) if kind == "order_unsorted" else np.asarray(idx_row)
        ztop = z_row[ids]
        order = np.min(ztop[:-1] - ztop[1:]) if k > 1 else np.inf
        call = np.asarray(c_row, float)
        c = call if kind == "tau_includes_top1" else call[1:]
        tau_m = np.min(np.abs(c - tau)) if np.isfinite(tau) and c.size else np.inf
        restore = np.inf
        if (m_min > 1 or kind == "restore_any_m_min") and c.size > 1:
            cs = np.sort(c)
            restore = np.min(cs[1:] - cs[:-1])
        return dict(boundary=boundary, order=order, tau=tau_m, restore=restore)
    return fn


def _is_tied_inclusive(m, band=TIES.BAND):
    return min(m.values()) <= band


def _admissible_variant(kind):
    def fn(z_row, pi_row, gpu_idx_row, gpu_keep_row, a_gsp, a_rcr, tau, m_min, eps, band=TIES.BAND,
           fusion="max"):
        z_row = np.asarray(z_row, float)
        idx = np.asarray(gpu_idx_row, dtype=np.int64)
        keep = np.asarray(gpu_keep_row, dtype=bool)
        k, N = idx.size, z_row.size
        if len(set(idx.tolist())) != k or idx.min() < 0 or idx.max() >= N:
            return False, "ids"
        zt = z_row[idx]
        if kind != "no_order_check" and k > 1 and np.any(zt[:-1] < zt[1:] - band):
            return False, "order"
        others = np.setdiff1d(np.arange(N), idx)
        if kind != "no_topk_set_check" and others.size and zt.min() < z_row[others].max() - band:
            return False, "set"
        if not keep[0]:
            return False, "top1"
        top = np.asarray(pi_row, float)[idx]
        g = top / top.sum()
        c = F.contributions(g, np.asarray(a_gsp, float)[idx], np.asarray(a_rcr, float)[idx], eps, fusion)[0]
        skip_final = {i for i in range(1, k) if not keep[i]}
        if kind == "band_inclusive":
            ambiguous = [i for i in range(1, k) if abs(c[i] - tau) <= band]
        else:
            ambiguous = [i for i in range(1, k) if abs(c[i] - tau) < band]
        clear_skip = {i for i in range(1, k) if c[i] < tau and i not in ambiguous}
        if kind == "ignore_clear_skip":
            clear_skip = set()
        for r in range(len(ambiguous) + 1):
            for extra in combinations(ambiguous, r):
                s0 = clear_skip | set(extra)
                need = max(0, m_min - (k - len(s0)))
                if kind != "skip_not_subset" and not skip_final <= s0:
                    continue
                restored = s0 - skip_final
                if kind == "skip_not_subset":
                    restored = set()
                    need = 0
                if len(restored) != need:
                    continue
                if kind == "restore_order_ignored" or all(c[a] >= c[b] - band for a in restored for b in skip_final):
                    return True, "ok"
        return False, "mask"
    return fn


def _compare_no_admissibility(z, pi, oracle_idx, oracle_keep, c, gpu_idx, gpu_keep, a_gsp, a_rcr, tau, m_min,
                              eps, band=TIES.BAND, fusion="max"):
    rep = _ORIG_COMPARE(z, pi, oracle_idx, oracle_keep, c, gpu_idx, gpu_keep, a_gsp, a_rcr, tau, m_min, eps,
                        band, fusion)
    rep["inadmissible"] = []
    return rep


_ORIG_COMPARE = TIES.compare_decisions


MUTANTS = {
    "rmsnorm_mean_abs": [(F, "rmsnorm", _rms_abs)],
    "rmsnorm_no_gamma": [(F, "rmsnorm", _rms_no_gamma)],
    "topk_ties_high_id": [(F, "topk_order", _topk_high_id)],
    "gates_not_renormalised": [(F, "route", _route_no_renorm)],
    "skip_union": [(F, "ace_skip", _skip_variant("union"))],
    "skip_non_strict": [(F, "ace_skip", _skip_variant("non_strict"))],
    "skip_no_top1": [(F, "ace_skip", _skip_variant("no_top1"))],
    "skip_restore_ascending": [(F, "ace_skip", _skip_variant("restore_ascending"))],
    "skip_no_eps_final": [(F, "ace_skip", _skip_variant("no_eps_final"))],
    "skip_no_eps_in_p": [(F, "ace_skip", _skip_variant("no_eps_in_p"))],
    "fusion_min_is_max": [(F, "contributions", _contrib_variant("min_is_max"))],
    "fusion_mean_no_half": [(F, "contributions", _contrib_variant("mean_no_half"))],
    "fusion_score_is_gsp": [(F, "contributions", _contrib_variant("score_is_gsp"))],
    "fusion_rcr_is_gsp": [(F, "contributions", _contrib_variant("rcr_is_gsp"))],
    "ffn_silu_on_up": [(F, "expert_ffn", _ffn_silu_on_up), (TB, "expert_ffn", _ffn_silu_on_up)],
    "ffn_relu": [(F, "expert_ffn", _ffn_relu), (TB, "expert_ffn", _ffn_relu)],
    "gsp_up_path_only": [(TB, "gsp_raw", _gsp_up_only)],
    "gsp_no_gamma": [(TB, "gsp_raw", _gsp_no_gamma)],
    "gsp_swapped_paths": [(TB, "gsp_raw", _gsp_swapped_paths)],
    "rcr_uncentred": [(TB, "rcr_prototypes", _proto_uncentred)],
    "rcr_l2_not_rms": [(TB, "rcr_prototypes", _proto_l2)],
    "tau_floor": [(TAU, "tau_for_budget", _tau_floor)],
    "tau_off_by_one": [(TAU, "tau_for_budget", _tau_off_by_one)],
    "plan_token_descending": [(PL, "dispatch_plan", _plan_token_desc)],
    "ties_boundary_off_by_one": [(TIES, "token_margins", _margins_variant("boundary_off_by_one"))],
    "ties_order_unsorted": [(TIES, "token_margins", _margins_variant("order_unsorted"))],
    "ties_tau_includes_top1": [(TIES, "token_margins", _margins_variant("tau_includes_top1"))],
    "ties_restore_any_m_min": [(TIES, "token_margins", _margins_variant("restore_any_m_min"))],
    "ties_band_inclusive": [(TIES, "is_tied", _is_tied_inclusive)],
    "ties_admissible_band_inclusive": [(TIES, "admissible_token", _admissible_variant("band_inclusive"))],
    "ties_admissible_ignores_clear_skip": [(TIES, "admissible_token", _admissible_variant("ignore_clear_skip"))],
    "ties_admissible_skip_not_subset": [(TIES, "admissible_token", _admissible_variant("skip_not_subset"))],
    "ties_admissible_restore_order_ignored": [(TIES, "admissible_token",
                                               _admissible_variant("restore_order_ignored"))],
    "ties_admissible_no_topk_set_check": [(TIES, "admissible_token", _admissible_variant("no_topk_set_check"))],
    "ties_admissible_no_order_check": [(TIES, "admissible_token", _admissible_variant("no_order_check"))],
    "ties_compare_no_admissibility": [(TIES, "compare_decisions", _compare_no_admissibility)],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for mod, attr, fn in MUTANTS[name]:
        monkeypatch.setattr(mod, attr, fn)
    caught = []
    for check in P.ALL_CHECKS:
        try:
            check()
        except Exception as e:  # noqa: BLE001 - any failure counts as caught
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin caught the planted mistake {name}"
