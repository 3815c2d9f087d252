"""Online ACE MoE layer forward in fp64 (test infrastructure only).

Follows the paper's online loop (Alg. 1) and its per-token skipping procedure
(Alg. 4, "ACE: Online Conservative Expert Skipping"), written per token from
the definitions, with no batching across tokens beyond the router matmul.

Notation (HF / nn.Linear layouts):
  x        [T, d]      layer input (before RMSNorm)
  gamma    [d]         RMSNorm scale (the diagonal of Gamma_l, Sec. 3.1)
  w_router [N, d]      row e is the router vector w_e (App. B.2, Eq. app_router_logit)
  w_gate, w_up [N, m, d], w_down [N, d, m]   SwiGLU expert weights (Eq. swiglu_expert)
"""
from __future__ import annotations

import numpy as np


def f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def rmsnorm(x, gamma, rms_eps: float):
    """x_in = x / sqrt(mean(x^2) + eps) * gamma  (Sec. 3.1: x = x_bar Gamma_l)."""
    x = f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + rms_eps) * f64(gamma)


def router_logits(x_in, w_router, b_router=None):
    """z_e = x^T w_e + b_e  (App. B.2, Eq. app_router_logit)."""
    z = f64(x_in) @ f64(w_router).T
    if b_router is not None:
        z = z + f64(b_router)
    return z


def softmax(z):
    """pi_e = exp(z_e) / sum_j exp(z_j)  (App. B.2, Eq. app_router_probability)."""
    z = f64(z)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def topk_order(z_row, k: int):
    """Expert ids of the k largest logits, in descending logit order; equal
    logits go to the lower expert id."""
    z_row = f64(z_row)
    ids = sorted(range(len(z_row)), key=lambda e: (-z_row[e], e))
    return np.array(ids[:k], dtype=np.int64)


def route(x_in, w_router, b_router, k: int):
    """Original top-k candidate set and its gates (Sec. 3.1).

    The gates are the router probabilities of the k selected experts
    renormalised to sum to one (App. B.4 assumes non-negative gates summing to
    one).  Returns (z [T,N], pi [T,N], topk_idx [T,k], g [T,k]).
    """
    z = router_logits(x_in, w_router, b_router)
    pi = softmax(z)
    T = z.shape[0]
    idx = np.zeros((T, k), dtype=np.int64)
    g = np.zeros((T, k), dtype=np.float64)
    for t in range(T):
        idx[t] = topk_order(z[t], k)
        top = pi[t, idx[t]]
        g[t] = top / top.sum()
    return z, pi, idx, g


# Fusion rules of the per-slot contribution score (Sec. 4.3, Tab. fusion_ablation and
# Tab. ablation; Sec. 4.1 baselines):
#   "max"   c = max(p_GSP, p_RCR), the ACE rule (Eq. ace_contribution): skip only if
#           both views are low, i.e. the intersection of the two candidate sets
#           (Eq. ace_candidate_intersection)
#   "min"   c = min(p_GSP, p_RCR): skip if either view is low (the union of the sets)
#   "mean"  c = (p_GSP + p_RCR) / 2
#   "gsp"   c = p_GSP (single view);  "rcr"  c = p_RCR (single view)
#   "score" c = g / (sum g + eps): router-score skipping, the p of Alg. 4 with a
#           table of ones
FUSIONS = ("max", "min", "mean", "gsp", "rcr", "score")


def contributions(g, a_gsp_e, a_rcr_e, eps: float, fusion: str = "max"):
    """Per-slot (c, p_gsp, p_rcr) of one token under a fusion rule."""
    g = f64(g)
    # dual-view scores and their normalisation within the top-k set
    # (Eqs. gsp_contribution, gsp_probability, rcr_contribution, rcr_probability)
    s_gsp = g * f64(a_gsp_e)
    s_rcr = g * f64(a_rcr_e)
    p_gsp = s_gsp / (s_gsp.sum() + eps)
    p_rcr = s_rcr / (s_rcr.sum() + eps)
    if fusion == "max":
        c = np.maximum(p_gsp, p_rcr)                  # Eq. ace_contribution
    elif fusion == "min":
        c = np.minimum(p_gsp, p_rcr)
    elif fusion == "mean":
        c = (p_gsp + p_rcr) / 2.0
    elif fusion == "gsp":
        c = p_gsp.copy()
    elif fusion == "rcr":
        c = p_rcr.copy()
    elif fusion == "score":
        c = g / (g.sum() + eps)
    else:
        raise ValueError(f"unknown fusion rule {fusion!r}")
    return c, p_gsp, p_rcr


def ace_skip(g, a_gsp_e, a_rcr_e, tau: float, m_min: int, eps: float, fusion: str = "max"):
    """Alg. 4 for one token (with the fusion rule replaced for the ablation variants).

    g        [k] gates of the routed slots (slot order)
    a_gsp_e  [k] A^GSP(e_i) looked up for each slot
    a_rcr_e  [k] A^RCR(e_i)
    Returns dict(keep [k] bool, ghat [k] (0 where skipped), c, p_gsp, p_rcr,
                 s_gsp_set, s_rcr_set, skip_set).
    """
    g = f64(g)
    k = g.shape[0]
    c, p_gsp, p_rcr = contributions(g, a_gsp_e, a_rcr_e, eps, fusion)
    # low-contribution candidate sets of the two views
    s_gsp_set = {i for i in range(k) if p_gsp[i] < tau}
    s_rcr_set = {i for i in range(k) if p_rcr[i] < tau}
    if fusion == "max":
        skip = s_gsp_set & s_rcr_set                  # Eq. ace_candidate_intersection
    elif fusion == "min":
        skip = s_gsp_set | s_rcr_set
    else:
        skip = {i for i in range(k) if c[i] < tau}
    # the top-1 routed expert is always retained
    top1 = max(range(k), key=lambda i: (g[i], -i))
    skip.discard(top1)
    active = set(range(k)) - skip
    # minimum-active safeguard: restore skipped slots by descending c (ties -> lower slot)
    if len(active) < m_min:
        order = sorted(skip, key=lambda i: (-c[i], i))
        for i in order[: m_min - len(active)]:
            skip.discard(i)
            active.add(i)
    z_gate = sum(g[i] for i in active) + eps
    ghat = np.zeros(k)
    for i in active:
        ghat[i] = g[i] / z_gate
    keep = np.array([i in active for i in range(k)])
    return dict(keep=keep, ghat=ghat, c=c, p_gsp=p_gsp, p_rcr=p_rcr,
                s_gsp_set=s_gsp_set, s_rcr_set=s_rcr_set, skip_set=skip)


def silu(v):
    v = f64(v)
    return v / (1.0 + np.exp(-v))


def expert_ffn(x_in_row, w_gate_e, w_up_e, w_down_e):
    """SwiGLU expert f(x) = (SiLU(x W_gate) * (x W_up)) W_down (Eq. swiglu_expert),
    written for nn.Linear layouts: W_down @ (SiLU(W_gate @ x) * (W_up @ x))."""
    x = f64(x_in_row)
    h = silu(f64(w_gate_e) @ x) * (f64(w_up_e) @ x)
    return f64(w_down_e) @ h


def moe_forward(layer: dict, k: int, a_gsp, a_rcr, tau: float, m_min: int = 1,
                eps: float = 1e-6, rms_eps: float = 1e-6, skip_disable: bool = False,
                tokens=None, decisions=None, fusion: str = "max"):
    """The online ACE layer forward (Alg. 1's online loop; Eq. ace_sparse_output).

    layer      dict with x, gamma, w_router, b_router, w_gate, w_up, w_down and
               optionally ws_gate/ws_up/ws_down (an ungated, always-on shared expert).
    k          top-k.
    a_gsp, a_rcr  [N] amplification tables (the values handed to the GPU).
    skip_disable  plain top-k layer: every slot kept and ghat = g exactly.
    fusion     contribution rule (FUSIONS; "max" is ACE).
    tokens     optional iterable of token indices for which y is evaluated
               (routing and masks are always computed for every token).
    decisions  optional (topk_idx [T,k], keep [T,k]): evaluate y with these routing
               decisions instead of the oracle's own (used when a GPU decision taken
               inside the tie band differs).  Gates are then the fp64 router
               probabilities of those experts renormalised over them, and ghat is
               renormalised over the given kept slots as in Alg. 4.
    Returns dict with x_in, z, pi, topk_idx, g, keep, ghat, c, p_gsp, p_rcr, y
    (rows of y outside `tokens` are NaN).
    """
    x_in = rmsnorm(layer["x"], layer["gamma"], rms_eps)
    z, pi, idx, g = route(x_in, layer["w_router"], layer.get("b_router"), k)
    T = idx.shape[0]
    if decisions is not None:
        idx = np.asarray(decisions[0], dtype=np.int64).reshape(T, k)
        top = pi[np.arange(T)[:, None], idx]
        g = top / top.sum(axis=1, keepdims=True)
    a_gsp = f64(a_gsp)
    a_rcr = f64(a_rcr)
    keep = np.zeros((T, k), dtype=bool)
    ghat = np.zeros((T, k))
    c = np.zeros((T, k))
    p_gsp = np.zeros((T, k))
    p_rcr = np.zeros((T, k))
    for t in range(T):
        r = ace_skip(g[t], a_gsp[idx[t]], a_rcr[idx[t]], tau, m_min, eps, fusion)
        c[t], p_gsp[t], p_rcr[t] = r["c"], r["p_gsp"], r["p_rcr"]
        if skip_disable:
            keep[t] = True
            ghat[t] = g[t]
        elif decisions is None:
            keep[t] = r["keep"]
            ghat[t] = r["ghat"]
        else:
            keep[t] = np.asarray(decisions[1][t], dtype=bool)
            z_gate = g[t][keep[t]].sum() + eps
            ghat[t][keep[t]] = g[t][keep[t]] / z_gate
    d = layer["x"].shape[1]
    y = np.full((T, d), np.nan)
    for t in (range(T) if tokens is None else tokens):
        acc = np.zeros(d)
        for i in range(k):
            if keep[t, i]:
                e = idx[t, i]
                acc += ghat[t, i] * expert_ffn(x_in[t], layer["w_gate"][e], layer["w_up"][e],
                                               layer["w_down"][e])
        if layer.get("ws_gate") is not None:
            acc += expert_ffn(x_in[t], layer["ws_gate"], layer["ws_up"], layer["ws_down"])
        y[t] = acc
    return dict(x_in=x_in, z=z, pi=pi, topk_idx=idx, g=g, keep=keep, ghat=ghat, c=c,
                p_gsp=p_gsp, p_rcr=p_rcr, y=y)
