"""Pins of the CPU oracle against facts other than itself.

Each check raises AssertionError when the oracle disagrees with what the paper
or the mathematics fixes: closed forms, invariants the paper proves, brute
force on tiny inputs, and the hand-derived Alg. 4 worked example.  The checks
look up oracle functions at call time, so a mutation test can plant a mistake
in the oracle and confirm that some check catches it.
"""
from __future__ import annotations

import json
import os
from itertools import combinations

import numpy as np

import oracle
from synth import config, make_layer

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def tiny_layer(T=24, d=16, N=6, k=3, m=8, seed=0, dtype="f32", **kw):
    return make_layer(config("tiny_f32", T=T, d=d, N=N, k=k, m=m, dtype=dtype, seed=seed, **kw))


# --------------------------------------------------------------------------- router
def check_rmsnorm_closed_form():
    # x = [3, 4]: mean(x^2) = 12.5; gamma = [1, 2]
    x_in = oracle.forward.rmsnorm(np.array([[3.0, 4.0]]), np.array([1.0, 2.0]), 0.0)
    want = np.array([[3.0 / np.sqrt(12.5), 8.0 / np.sqrt(12.5)]])
    assert np.allclose(x_in, want, rtol=0, atol=1e-15), x_in
    # with eps: x = [1, 1, 1, 1], gamma = 1 -> 1/sqrt(1 + eps)
    x_in = oracle.forward.rmsnorm(np.ones((1, 4)), np.ones(4), 0.25)
    assert np.allclose(x_in, 1.0 / np.sqrt(1.25), rtol=0, atol=1e-15)


def check_topk_brute_force():
    rng = _rng(1)
    for _ in range(50):
        N = int(rng.integers(2, 12))
        k = int(rng.integers(1, N + 1))
        z = rng.integers(-3, 4, size=N).astype(float)      # many exact ties
        got = oracle.forward.topk_order(z, k)
        want = np.lexsort((np.arange(N), -z))[:k]          # by -z, then by id
        assert np.array_equal(got, want), (z, got, want)


def check_route_gates_and_translation_invariance():
    L = tiny_layer(seed=3)
    x_in = oracle.forward.rmsnorm(L["x"], L["gamma"], 1e-6)
    z, pi, idx, g = oracle.forward.route(x_in, L["w_router"], None, 3)
    assert np.allclose(pi.sum(1), 1.0, atol=1e-14)
    assert np.allclose(g.sum(1), 1.0, atol=1e-14)
    assert np.all(np.diff(g, axis=1) <= 1e-15), "gates must be in descending order"
    # gates are the selected softmax probabilities, renormalised
    for t in range(len(z)):
        e = np.exp(z[t, idx[t]] - z[t, idx[t]].max())
        assert np.allclose(g[t], e / e.sum(), atol=1e-14)
    # App. B.2: adding one vector to every router row changes no probability
    shift = _rng(4).standard_normal(L["w_router"].shape[1])
    z2, pi2, idx2, g2 = oracle.forward.route(x_in, L["w_router"] + shift[None, :], None, 3)
    assert np.allclose(pi2, pi, atol=1e-12)
    assert np.array_equal(idx2, idx)
    assert np.allclose(g2, g, atol=1e-12)


# --------------------------------------------------------------------------- Alg. 4
def check_worked_example():
    ex = json.load(open(os.path.join(GOLDEN, "alg4_worked_example.json")))
    g = np.array(ex["g"])
    for case in ex["cases"]:
        if case["tables"] == "all ones":
            ag = ar = np.ones(4)
        else:
            ag, ar = np.array(ex["a_gsp"]), np.array(ex["a_rcr"])
        r = oracle.forward.ace_skip(g, ag, ar, case["tau"], case["m_min"], ex["eps"])
        if case["tables"] != "all ones":
            assert np.allclose(r["p_gsp"], ex["p_gsp"], atol=1e-15)
            assert np.allclose(r["p_rcr"], ex["p_rcr"], atol=1e-15)
            assert np.allclose(r["c"], ex["c"], atol=1e-15)
        skipped = sorted(i for i in range(4) if not r["keep"][i])
        assert skipped == case["skipped"], (case, skipped)
        assert np.allclose(r["ghat"], case["ghat"], atol=1e-15), (case, r["ghat"])


def check_alg4_eps_closed_form():
    # the worked example's gates and tables with eps = 0.5: Z_gsp = 1.15 + 0.5, Z_rcr = 1.0 + 0.5
    g = np.array([0.4, 0.3, 0.2, 0.1])
    r = oracle.forward.ace_skip(g, np.array([1.0, 1.0, 2.0, 0.5]), np.array([1.0, 1.0, 0.5, 2.0]),
                                0.0, 1, 0.5)
    assert np.allclose(r["p_gsp"], [8 / 33, 6 / 33, 8 / 33, 1 / 33], rtol=0, atol=1e-15)
    assert np.allclose(r["p_rcr"], [4 / 15, 3 / 15, 1 / 15, 2 / 15], rtol=0, atol=1e-15)
    assert np.allclose(r["ghat"], g / 1.5, rtol=0, atol=1e-15)
    # tau = 0.14 with eps = 0.5: slot 3 has p_gsp = 1/33 and p_rcr = 2/15, both below -> skipped;
    # slot 2 has p_rcr = 1/15 but p_gsp = 8/33 -> kept
    r = oracle.forward.ace_skip(g, np.array([1.0, 1.0, 2.0, 0.5]), np.array([1.0, 1.0, 0.5, 2.0]),
                                0.14, 1, 0.5)
    assert r["keep"].tolist() == [True, True, True, False]


def _random_tokens(n, k, seed):
    rng = _rng(seed)
    for _ in range(n):
        g = np.sort(rng.dirichlet(np.ones(k)))[::-1]
        yield g, rng.uniform(0.3, 2.0, k), rng.uniform(0.3, 2.0, k), float(rng.uniform(0.0, 0.6))


def check_max_rule_is_intersection_and_safeguards():
    for g, ag, ar, tau in _random_tokens(400, 6, 5):
        for m_min in (1, 2, 4):
            r = oracle.forward.ace_skip(g, ag, ar, tau, m_min, 1e-6)
            skipped = {i for i in range(6) if not r["keep"][i]}
            inter = (r["s_gsp_set"] & r["s_rcr_set"]) - {0}
            assert skipped <= inter                       # Eq. app_safeguarded_subset
            if m_min == 1:
                assert skipped == {i for i in range(1, 6) if r["c"][i] < tau}
                assert skipped == inter
            assert r["keep"][0]                           # top-1 never skipped
            assert r["keep"].sum() >= min(m_min, 6)
            # Eq. app_skipped_mass_comparison
            alpha = lambda S: sum(g[i] for i in S)
            assert alpha(skipped) <= min(alpha(r["s_gsp_set"]), alpha(r["s_rcr_set"])) + 1e-15
            # renormalised gates
            kept = r["keep"]
            assert np.allclose(r["ghat"][kept], g[kept] / (g[kept].sum() + 1e-6), atol=1e-15)
            assert np.all(r["ghat"][~kept] == 0)


def check_alg4_special_cases():
    for g, ag, ar, tau in _random_tokens(200, 5, 6):
        eps = 1e-6
        # tau <= 0: nothing skipped, ghat = g/(1+eps)
        r = oracle.forward.ace_skip(g, ag, ar, 0.0, 1, eps)
        assert r["keep"].all() and np.allclose(r["ghat"], g / (1 + eps), atol=1e-16)
        # all-ones tables: router-score skipping, skip iff g/(1+eps) < tau
        r = oracle.forward.ace_skip(g, np.ones(5), np.ones(5), tau, 1, eps)
        want = np.array([True] + [g[i] / (1 + eps) >= tau for i in range(1, 5)])
        assert np.array_equal(r["keep"], want)
        # equal tables: single-view GSP, c = p_gsp
        r = oracle.forward.ace_skip(g, ag, ag, tau, 1, eps)
        assert np.allclose(r["c"], g * ag / ((g * ag).sum() + eps), atol=1e-16)
        # m_min = k: plain top-k
        r = oracle.forward.ace_skip(g, ag, ar, tau, 5, eps)
        assert r["keep"].all()


def check_alg4_brute_force():
    """Declarative characterisation, checked over every subset: the skip set is
    the largest subset of the skippable slots {i != top1 : c_i < tau} that
    leaves at least m_min slots active, and among those the one skipping the
    least total contribution c (distinct c values make it unique)."""
    rng = _rng(7)
    for _ in range(300):
        k = int(rng.integers(2, 6))
        g = np.sort(rng.dirichlet(np.ones(k)))[::-1]
        ag, ar = rng.uniform(0.3, 2.0, k), rng.uniform(0.3, 2.0, k)
        tau = float(rng.uniform(0.0, 0.7))
        m_min = int(rng.integers(1, k + 1))
        r = oracle.forward.ace_skip(g, ag, ar, tau, m_min, 1e-6)
        c = r["c"]
        p_g = g * ag / ((g * ag).sum() + 1e-6)
        p_r = g * ar / ((g * ar).sum() + 1e-6)
        skippable = [i for i in range(1, k) if p_g[i] < tau and p_r[i] < tau]
        best = None
        for n in range(len(skippable), -1, -1):
            if k - n < m_min:
                continue
            cands = [set(S) for S in combinations(skippable, n)]
            best = min(cands, key=lambda S: sum(c[i] for i in S))
            break
        assert {i for i in range(k) if not r["keep"][i]} == best, (g, ag, ar, tau, m_min)


def check_fusion_variants_against_the_max_rule():
    """The ablation variants (Tab. fusion_ablation, Tab. ablation; Sec. 4.1 Score)
    against the ACE rule and against each other: the single views and router-score
    skipping are the max rule with equal / all-ones tables; {max, min} = {p_GSP,
    p_RCR}, so c_min + c_max = p_GSP + p_RCR = 2 c_mean; min is the union rule."""
    F = oracle.forward
    eps = 1e-6
    for g, ag, ar, tau in _random_tokens(300, 6, 11):
        r = {f: F.ace_skip(g, ag, ar, tau, 1, eps, f) for f in F.FUSIONS}
        same_gsp = F.ace_skip(g, ag, ag, tau, 1, eps, "max")
        same_rcr = F.ace_skip(g, ar, ar, tau, 1, eps, "max")
        ones = F.ace_skip(g, np.ones(6), np.ones(6), tau, 1, eps, "max")
        assert np.array_equal(r["gsp"]["keep"], same_gsp["keep"]) and np.allclose(r["gsp"]["c"], same_gsp["c"], rtol=0, atol=0)
        assert np.array_equal(r["rcr"]["keep"], same_rcr["keep"]) and np.allclose(r["rcr"]["c"], same_rcr["c"], rtol=0, atol=0)
        assert np.array_equal(r["score"]["keep"], ones["keep"]) and np.allclose(r["score"]["c"], ones["c"], rtol=1e-15, atol=0)
        cmax, cmin, cmean = r["max"]["c"], r["min"]["c"], r["mean"]["c"]
        assert np.all(cmin <= cmean) and np.all(cmean <= cmax) and np.all(cmin <= cmax)
        assert np.allclose(cmin + cmax, 2 * cmean, rtol=1e-15, atol=1e-17)
        # with m_min = 1 the skip sets nest: max inside mean inside min
        sk = {f: {i for i in range(6) if not r[f]["keep"][i]} for f in F.FUSIONS}
        assert sk["max"] <= sk["mean"] <= sk["min"]
        # min is the union of the two views' candidate sets (top-1 excluded)
        assert sk["min"] == (r["max"]["s_gsp_set"] | r["max"]["s_rcr_set"]) - {0}
        for f in F.FUSIONS:
            assert r[f]["keep"][0]
            kept = r[f]["keep"]
            assert np.allclose(r[f]["ghat"][kept], g[kept] / (g[kept].sum() + eps), atol=1e-15)


def check_fusion_brute_force():
    """Every variant obeys the same declarative characterisation as the ACE rule
    (largest skippable subset leaving m_min active, least total c), with the
    skippable slots taken from the two views directly."""
    F = oracle.forward
    rng = _rng(13)
    for _ in range(200):
        k = int(rng.integers(2, 6))
        g = np.sort(rng.dirichlet(np.ones(k)))[::-1]
        ag, ar = rng.uniform(0.3, 2.0, k), rng.uniform(0.3, 2.0, k)
        tau = float(rng.uniform(0.0, 0.7))
        m_min = int(rng.integers(1, k + 1))
        p_g = g * ag / ((g * ag).sum() + 1e-6)
        p_r = g * ar / ((g * ar).sum() + 1e-6)
        low = {"max": lambda i: p_g[i] < tau and p_r[i] < tau,
               "min": lambda i: p_g[i] < tau or p_r[i] < tau,
               "mean": lambda i: p_g[i] + p_r[i] < 2 * tau,
               "gsp": lambda i: p_g[i] < tau,
               "rcr": lambda i: p_r[i] < tau,
               "score": lambda i: g[i] < tau * (g.sum() + 1e-6)}
        for f in F.FUSIONS:
            r = F.ace_skip(g, ag, ar, tau, m_min, 1e-6, f)
            c = r["c"]
            skippable = [i for i in range(1, k) if low[f](i)]
            best = None
            for n in range(len(skippable), -1, -1):
                if k - n < m_min:
                    continue
                best = min((set(S) for S in combinations(skippable, n)), key=lambda S: sum(c[i] for i in S))
                break
            assert {i for i in range(k) if not r["keep"][i]} == best, (f, g, ag, ar, tau, m_min)


# --------------------------------------------------------------------------- output
def check_dense_brute_force_output():
    L = tiny_layer(T=20, d=12, N=5, k=3, m=7, seed=8)
    tb = oracle.tables.build_tables(L)
    out = oracle.forward.moe_forward(L, 3, tb["a_gsp"], tb["a_rcr"], tau=0.3)
    x_in = out["x_in"]
    # every expert on every token, with matrix products over the whole batch
    F = np.stack([
        (1 / (1 + np.exp(-(x_in @ L["w_gate"][e].astype(float).T))) * (x_in @ L["w_gate"][e].astype(float).T)
         * (x_in @ L["w_up"][e].astype(float).T)) @ L["w_down"][e].astype(float).T
        for e in range(5)], axis=1)                       # [T, N, d]
    Wdense = np.zeros((20, 5))
    for t in range(20):
        for i in range(3):
            Wdense[t, out["topk_idx"][t, i]] += out["ghat"][t, i]
    y = np.einsum("tn,tnd->td", Wdense, F)
    assert np.allclose(out["y"], y, rtol=1e-12, atol=1e-14)
    assert (~out["keep"]).any() and out["keep"][:, 0].all()


def check_dense_special_cases():
    # N = 1, k = 1: a dense SwiGLU FFN on the normalised input
    L = tiny_layer(T=10, d=8, N=1, k=1, m=6, seed=9)
    out = oracle.forward.moe_forward(L, 1, np.ones(1, np.float32), np.ones(1, np.float32), tau=0.5,
                                     eps=0.0)
    x = L["x"].astype(float)
    x_in = x / np.sqrt((x ** 2).mean(1, keepdims=True) + 1e-6) * L["gamma"]
    a = x_in @ L["w_gate"][0].astype(float).T
    want = (a / (1 + np.exp(-a)) * (x_in @ L["w_up"][0].astype(float).T)) @ L["w_down"][0].astype(float).T
    assert np.allclose(out["y"], want, rtol=1e-12, atol=1e-14)
    # k = N, tau = 0, eps = 0: dense softmax-weighted mixture of every expert
    L = tiny_layer(T=6, d=8, N=4, k=4, m=5, seed=10)
    out = oracle.forward.moe_forward(L, 4, np.ones(4, np.float32), np.ones(4, np.float32), tau=0.0,
                                     eps=0.0)
    x_in = out["x_in"]
    pi = np.exp(x_in @ L["w_router"].astype(float).T)
    pi /= pi.sum(1, keepdims=True)
    y = np.zeros_like(x_in)
    for e in range(4):
        a = x_in @ L["w_gate"][e].astype(float).T
        fe = (a / (1 + np.exp(-a)) * (x_in @ L["w_up"][e].astype(float).T)) @ L["w_down"][e].astype(float).T
        y += pi[:, e:e + 1] * fe
    assert np.allclose(out["y"], y, rtol=1e-12, atol=1e-14)


def check_no_skip_and_perturbation_identity():
    L = tiny_layer(T=16, d=12, N=6, k=4, m=7, seed=11)
    tb = oracle.tables.build_tables(L)
    plain = oracle.forward.moe_forward(L, 4, tb["a_gsp"], tb["a_rcr"], tau=0.3, skip_disable=True)
    # tau = 0 keeps every slot; the eps of the final renormalisation scales y by 1/(1+eps)
    nos = oracle.forward.moe_forward(L, 4, tb["a_gsp"], tb["a_rcr"], tau=0.0, eps=1e-6)
    assert np.allclose(nos["y"], plain["y"] / (1 + 1e-6), rtol=1e-13, atol=1e-15)
    # with eps = 0: ||y - y_hat|| = alpha ||mu_S - mu_I|| <= 2 alpha F_max (App. B.4)
    ace = oracle.forward.moe_forward(L, 4, tb["a_gsp"], tb["a_rcr"], tau=0.3, eps=0.0)
    assert (~ace["keep"]).any()
    for t in range(16):
        keep = ace["keep"][t]
        g = plain["g"][t]
        fs = np.stack([oracle.forward.expert_ffn(ace["x_in"][t], L["w_gate"][e], L["w_up"][e],
                                                 L["w_down"][e]) for e in plain["topk_idx"][t]])
        alpha = g[~keep].sum()
        lhs = np.linalg.norm(plain["y"][t] - ace["y"][t])
        if alpha == 0:
            assert lhs < 1e-14
            continue
        mu_i = (g[keep, None] * fs[keep]).sum(0) / (1 - alpha)
        mu_s = (g[~keep, None] * fs[~keep]).sum(0) / alpha
        assert abs(lhs - alpha * np.linalg.norm(mu_s - mu_i)) < 1e-12
        assert lhs <= 2 * alpha * np.linalg.norm(fs, axis=1).max() + 1e-14


def check_swiglu_bound():
    # Eq. swiglu_upper_bound: ||f(x)|| <= ||x_bar||^2 ||Gamma W_g||_2 ||Gamma W_u||_2 ||W_d||_2
    rng = _rng(12)
    for _ in range(50):
        d, m = 9, 7
        gam = 1 + 0.1 * rng.standard_normal(d)
        wg, wu, wd = rng.standard_normal((m, d)), rng.standard_normal((m, d)), rng.standard_normal((d, m))
        xb = rng.standard_normal(d)
        f = oracle.forward.expert_ffn(xb * gam, wg, wu, wd)
        bound = (np.linalg.norm(xb) ** 2 * np.linalg.norm(wg * gam, 2) * np.linalg.norm(wu * gam, 2)
                 * np.linalg.norm(wd, 2))
        assert np.linalg.norm(f) <= bound * (1 + 1e-12)


# --------------------------------------------------------------------------- GSP
def check_gsp_scaled_copies():
    rng = _rng(13)
    d, m, N = 10, 6, 5
    gam = 1 + 0.1 * rng.standard_normal(d)
    base = dict(g=rng.standard_normal((m, d)), u=rng.standard_normal((m, d)), d=rng.standard_normal((d, m)))
    c = rng.uniform(0.2, 3.0, N)
    for which in ("g", "u", "d", "gu"):
        wg = np.stack([base["g"] * (c[e] if "g" in which else 1) for e in range(N)])
        wu = np.stack([base["u"] * (c[e] if "u" in which else 1) for e in range(N)])
        wd = np.stack([base["d"] * (c[e] if which == "d" else 1) for e in range(N)])
        A = oracle.tables.gsp_table(gam, wg, wu, wd, eps=0.0)
        want = c ** 2 if which == "gu" else c
        assert np.allclose(A, want / want.mean(), rtol=1e-12), (which, A, want / want.mean())


def check_gsp_properties():
    rng = _rng(14)
    d, m, N = 8, 5, 6
    gam = 1 + 0.1 * rng.standard_normal(d)
    wg, wu, wd = rng.standard_normal((N, m, d)), rng.standard_normal((N, m, d)), rng.standard_normal((N, d, m))
    eps = 1e-3
    A = oracle.tables.gsp_table(gam, wg, wu, wd, eps)
    raw = np.array([oracle.tables.gsp_raw(gam, wg[e], wu[e], wd[e]) for e in range(N)])
    mu = raw.mean()
    assert np.isclose(A.mean(), mu / (mu + eps), rtol=1e-13)
    # permuting experts permutes the table
    p = rng.permutation(N)
    assert np.allclose(oracle.tables.gsp_table(gam, wg[p], wu[p], wd[p], eps), A[p], rtol=1e-13)
    # Frobenius norm of W_d G via the trace identity ||W_d G||^2 = <W_d^T W_d, G G^T>
    for e in range(N):
        G, U = wg[e] * gam, wu[e] * gam
        a_up = np.sqrt(np.sum(U * U)) * np.sqrt(np.sum((wd[e].T @ wd[e]) * (G @ G.T)))
        a_gate = np.sqrt(np.sum(G * G)) * np.sqrt(np.sum((wd[e].T @ wd[e]) * (U @ U.T)))
        assert np.isclose(raw[e], np.sqrt(a_up * a_gate), rtol=1e-12)
    # d = m = 1: a~ = gamma^2 |w_g w_u w_d|
    for _ in range(10):
        g1, wg1, wu1, wd1 = rng.standard_normal(4)
        r = oracle.tables.gsp_raw(np.array([g1]), np.array([[wg1]]), np.array([[wu1]]), np.array([[wd1]]))
        assert np.isclose(r, g1 * g1 * abs(wg1 * wu1 * wd1), rtol=1e-13)


# --------------------------------------------------------------------------- RCR
def check_rcr_properties():
    rng = _rng(15)
    d, m, N = 9, 6, 5
    wr = rng.standard_normal((N, d))
    wg, wu, wd = rng.standard_normal((N, m, d)), rng.standard_normal((N, m, d)), rng.standard_normal((N, d, m))
    eps = 1e-6
    A = oracle.tables.rcr_table(wr, wg, wu, wd, eps)
    # App. B.2: a shared translation of the router rows changes nothing
    A2 = oracle.tables.rcr_table(wr + rng.standard_normal(d)[None, :], wg, wu, wd, eps)
    assert np.allclose(A2, A, rtol=1e-10)
    # scaling every router row by s > 0 leaves the prototypes unchanged (up to eps)
    A3 = oracle.tables.rcr_table(3.7 * wr, wg, wu, wd, eps)
    assert np.allclose(A3, A, rtol=1e-5)
    # ||q_e|| = sqrt(d) r_e / (r_e + eps), with r_e the RMS of the centred row
    q = oracle.tables.rcr_prototypes(wr, eps=0.1)
    wt = wr - wr.mean(0)
    r = np.sqrt((wt ** 2).mean(1))
    assert np.allclose(np.linalg.norm(q, axis=1), np.sqrt(d) * r / (r + 0.1), rtol=1e-13)
    # prototype direction is the centred router row
    cos = np.sum(q * wt, 1) / np.linalg.norm(q, axis=1) / np.linalg.norm(wt, axis=1)
    assert np.allclose(cos, 1.0, atol=1e-13)
    # a~ is linear in W_down: scaling expert 2's down matrix by 2.5 scales its raw value by 2.5
    qq = oracle.tables.rcr_prototypes(wr, eps)
    r0 = oracle.tables.rcr_raw(qq[2], wg[2], wu[2], wd[2], eps)
    r1 = oracle.tables.rcr_raw(qq[2], wg[2], wu[2], 2.5 * wd[2], eps)
    assert np.isclose(r1, 2.5 * r0, rtol=1e-13)
    # d = m = 1: q = w~/(|w~| + eps), a~ = |w_d silu(w_g q) w_u q| / (|q| + eps)
    w = rng.standard_normal((3, 1))
    g1, u1, dd = rng.standard_normal((3, 1, 1)), rng.standard_normal((3, 1, 1)), rng.standard_normal((3, 1, 1))
    A1 = oracle.tables.rcr_table(w, g1, u1, dd, eps=0.0)
    wt = w[:, 0] - w[:, 0].mean()
    qv = wt / np.abs(wt)
    a = g1[:, 0, 0] * qv
    raw = np.abs(dd[:, 0, 0] * (a / (1 + np.exp(-a))) * u1[:, 0, 0] * qv) / np.abs(qv)
    assert np.allclose(A1, raw / raw.mean(), rtol=1e-12)


# --------------------------------------------------------------------------- tau mapping
def check_tau_mapping():
    # hand example: 10 slots, k = 2, candidates are slot 1 of each of 5 tokens
    c = np.array([[0.9, 0.10], [0.8, 0.30], [0.7, 0.20], [0.6, 0.50], [0.95, 0.40]])
    n_all = c.size
    cand = oracle.tau.candidate_mask(c, 1)
    assert cand[:, 0].sum() == 0 and cand[:, 1].all()
    pool = c[cand]
    assert oracle.tau.tau_for_budget(pool, n_all, 0.0) == 0.0
    assert np.isclose(oracle.tau.tau_for_budget(pool, n_all, 0.2), 0.25)   # m_q = 2: between 0.2 and 0.3
    assert np.isclose(oracle.tau.tau_for_budget(pool, n_all, 0.1), 0.15)   # m_q = 1
    assert oracle.tau.tau_for_budget(pool, n_all, 0.5) == np.inf           # m_q = 5 = N_cand
    assert oracle.tau.tau_for_budget(pool, n_all, 0.9) == np.inf           # clipped
    # round half to even: q N_all = 2.5 -> 2
    assert np.isclose(oracle.tau.tau_for_budget(pool, n_all, 0.25), 0.25)
    # ties at the boundary: scores [1, 2, 2, 2, 3]; m_q = 2 -> below (count 1) vs above (count 4)
    s = np.array([1.0, 2.0, 2.0, 2.0, 3.0])
    assert oracle.tau.tau_for_budget(s, 10, 0.2) == 2.0                     # realises #{c<2} = 1
    assert np.isclose(oracle.tau.tau_for_budget(s, 10, 0.3), 2.5)          # m_q=3: |1-3|=2 > |4-3|=1
    # m_min = 2 protects the highest-c non-top-1 slot (ties -> lower slot)
    c3 = np.array([[0.5, 0.2, 0.3], [0.6, 0.1, 0.1]])
    cm = oracle.tau.candidate_mask(c3, 2)
    assert cm.tolist() == [[False, True, False], [False, False, True]]


def check_tau_realises_budget_brute_force():
    rng = _rng(16)
    for trial in range(40):
        T, k = int(rng.integers(3, 9)), int(rng.integers(2, 5))
        L = tiny_layer(T=T, d=8, N=6, k=k, m=5, seed=100 + trial)
        tb = oracle.tables.build_tables(L)
        m_min = int(rng.integers(1, k + 1))
        base = oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=0.0, m_min=m_min,
                                          tokens=[])
        cand = oracle.tau.candidate_mask(base["c"], m_min)
        pool = base["c"][cand]
        n_all = base["c"].size
        prev = -1
        for q in (0.0, 0.1, 0.25, 0.4, 0.5, 0.7, 1.0):
            tau = oracle.tau.tau_for_budget(pool, n_all, q)
            out = oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=tau, m_min=m_min,
                                             tokens=[])
            realised = int((~out["keep"]).sum())
            m_q = int(np.clip(np.rint(q * n_all), 0, pool.size))
            # brute force over every threshold that separates the sorted scores
            vals = np.unique(pool)
            options = [0.0] + [float(v) for v in vals] + [np.inf]
            counts = [int((pool < t).sum()) for t in options]
            best = min(abs(cnt - m_q) for cnt in counts)
            assert abs(realised - m_q) == best, (q, realised, m_q, best)
            assert realised == int((pool < tau).sum())
            assert realised >= prev                           # monotone in q
            prev = realised


def check_tau_tiny_config_clip_branch():
    L = make_layer(config("tiny_f32"))
    tb = oracle.tables.build_tables(L)
    base = oracle.forward.moe_forward(L, 2, tb["a_gsp"], tb["a_rcr"], tau=0.0, tokens=[])
    taus = oracle.tau.tau_table([base["c"]], 1, [0.5])
    assert taus[0.5] == np.inf
    out = oracle.forward.moe_forward(L, 2, tb["a_gsp"], tb["a_rcr"], tau=taus[0.5], tokens=[])
    assert out["keep"][:, 0].all() and not out["keep"][:, 1].any()
    assert oracle.tau.realised_skip_ratio(out["keep"]) == 0.5


# --------------------------------------------------------------------------- plan
def check_plan():
    idx = np.array([[2, 0], [0, 1], [2, 1], [1, 2]])
    keep = np.array([[True, True], [True, False], [True, True], [True, False]])
    p = oracle.plan.dispatch_plan(idx, keep, 3)
    # expert 0: tokens 0, 1; expert 1: tokens 2, 3; expert 2: tokens 0, 2
    assert p["counts"].tolist() == [2, 2, 2]
    assert p["offsets"].tolist() == [0, 2, 4, 6]
    assert p["perm"].tolist() == [0, 1, 2, 3, 0, 2]
    assert p["slot_row"].tolist() == [[4, 0], [1, -1], [5, 2], [3, -1]]


# --------------------------------------------------------------------------- tie accounting
# Hand-built tokens for each decision margin the parity tests excuse (decisions within
# 1e-6 of a margin count as ties): the top-k boundary and the in-top-k slot order (Sec. 3.1,
# ties to the lower id), the strict c < tau test of a non-top-1 slot (Alg. 4, top-1
# kept) and, with m_min > 1, the restore order by descending c (Alg. 4).  Logits and
# contributions are written out here with plain numpy, not taken from the oracle.
_TB = 1e-6  # the tie band


def _tok(z, idx, a=None, eps=1e-6):
    """pi, gates and contributions c of one hand-built token whose experts `idx`
    (slot order) are routed; a = the per-expert table used for both views
    (so p_GSP = p_RCR = c), all ones by default."""
    z = np.asarray(z, float)
    e = np.exp(z - z.max())
    pi = e / e.sum()
    g = pi[idx] / pi[idx].sum()
    a = np.ones(z.size) if a is None else np.asarray(a, float)
    s = g * a[idx]
    return pi, g, s / (s.sum() + eps)


def check_ties_margins_hand_tokens():
    T = oracle.ties
    inf = np.inf
    # (a) k-th and (k+1)-th logits 4e-7 apart: the top-k set is ambiguous
    m = T.token_margins([3.0, 1.0 + 4e-7, 1.0, 0.0, -1.0], [0, 1], [0.7, 0.3], inf, 1)
    assert abs(m["boundary"] - 4e-7) < 1e-12 and abs(m["order"] - (2.0 - 4e-7)) < 1e-12, m
    assert T.is_tied(m, _TB)
    # the same token one logit further: nothing tied (boundary is z_(k) - z_(k+1), not z_(k+1) - z_(k+2))
    m = T.token_margins([3.0, 1.0 + 4e-7, 1.0, 0.0, -1.0], [0, 1, 2], [0.6, 0.3, 0.1], inf, 1)
    assert abs(m["boundary"] - 1.0) < 1e-12 and abs(m["order"] - 4e-7) < 1e-12, m
    assert T.is_tied(m, _TB)                               # via the order of slots 1 and 2
    m = T.token_margins([3.0, 1.0 + 4e-7, 1.0 - 1e-3, 0.0, 0.0 - 2e-7], [0, 1, 2], [0.6, 0.3, 0.1], inf, 1)
    assert abs(m["boundary"] - (1.0 - 1e-3)) < 1e-12 and not T.is_tied(m, _TB), m
    # (b) order: the margin is taken along the slot order (descending logits), whatever the ids
    m = T.token_margins([0.0, 3.0, 1.0, 2.0, -1.0], [1, 3, 2], [0.6, 0.3, 0.1], inf, 1)
    assert m["order"] == 1.0 and m["boundary"] == 1.0 and not T.is_tied(m, _TB), m
    m = T.token_margins([1.0 + 3e-7, 1.0, -1.0, -2.0], [0, 1], [0.5, 0.5], inf, 1)
    assert abs(m["order"] - 3e-7) < 1e-12 and T.is_tied(m, _TB), m
    # (c) |c - tau| of a non-top-1 slot
    m = T.token_margins([3.0, 2.0, 1.0, 0.0], [0, 1, 2], [0.6, 0.3000004, 0.1], 0.3, 1)
    assert abs(m["tau"] - 4e-7) < 1e-12 and T.is_tied(m, _TB), m
    # (d) the top-1 slot is never a candidate, so its distance to tau is no margin
    m = T.token_margins([3.0, 2.0, 1.0, 0.0], [0, 1, 2], [0.3000004, 0.2, 0.1], 0.3, 1)
    assert abs(m["tau"] - 0.1) < 1e-12 and not T.is_tied(m, _TB), m
    # tau = +inf (the clip branch) has no tau margin
    assert T.token_margins([3.0, 2.0, 1.0], [0, 1], [0.6, 0.4], inf, 1)["tau"] == inf
    # (e) restore order: only with m_min > 1, over the non-top-1 contributions
    c = [0.5, 0.2000003, 0.2, 0.05]
    m1 = T.token_margins([4.0, 3.0, 2.0, 1.0, 0.0], [0, 1, 2, 3], c, 0.9, 1)
    m2 = T.token_margins([4.0, 3.0, 2.0, 1.0, 0.0], [0, 1, 2, 3], c, 0.9, 2)
    assert m1["restore"] == inf and not T.is_tied(m1, _TB), m1
    assert abs(m2["restore"] - 3e-7) < 1e-12 and T.is_tied(m2, _TB), m2
    # top-1's c is no restore candidate either
    m = T.token_margins([4.0, 3.0, 2.0, 1.0, 0.0], [0, 1, 2, 3], [0.2000001, 0.2, 0.1, 0.05], 0.9, 2)
    assert abs(m["restore"] - 0.05) < 1e-12 and not T.is_tied(m, _TB), m
    # the band is strict: a margin of exactly the band is not a tie
    assert not T.is_tied(dict(boundary=_TB, order=1.0, tau=1.0, restore=np.inf), _TB)
    assert T.is_tied(dict(boundary=np.nextafter(_TB, 0.0), order=1.0, tau=1.0, restore=np.inf), _TB)


def check_ties_admissible_hand_tokens():
    T = oracle.ties
    eps = 1e-6
    ones = np.ones(6)
    z = [2.0, 1.0, 0.5, -1.0, -2.0, -3.0]
    idx = [0, 1, 2]
    pi, g, c = _tok(z, idx)

    def adm(keep, tau, gidx=idx, zz=z, p=pi, a=ones, m_min=1, band=_TB):
        return T.admissible_token(zz, p, gidx, keep, a, a, tau, m_min, eps, band)[0]

    # slot 2's c within the band of tau: either decision is admissible
    tau = c[2] + 5e-7
    assert adm([1, 1, 0], tau) and adm([1, 1, 1], tau)
    assert not adm([1, 0, 1], tau), "slot 1 (c far above tau) skipped"
    assert not adm([0, 1, 1], tau), "top-1 skipped"
    # c clearly below tau: the slot must be skipped
    tau = c[2] + 5e-6
    assert adm([1, 1, 0], tau) and not adm([1, 1, 1], tau)
    # c clearly above tau: the slot must be kept
    tau = c[2] - 5e-6
    assert adm([1, 1, 1], tau) and not adm([1, 1, 0], tau)
    # exactly one band below tau is outside the (strict) band: a clear skip (a band of
    # 2^-20, so that tau - c is exactly the band in fp64)
    b2 = 2.0 ** -20
    tau = c[2] + b2
    assert tau - c[2] == b2
    assert adm([1, 1, 0], tau, band=b2) and not adm([1, 1, 1], tau, band=b2)
    # top-k set: expert 3 within the band of expert 2 may replace it, not when clearly smaller
    for gap, ok in ((4e-7, True), (4e-6, False)):
        zb = [2.0, 1.0, 0.5 + gap, 0.5, -2.0, -3.0]
        pb, _, cb = _tok(zb, [0, 1, 3])
        assert adm([1, 1, 1], 0.0, gidx=[0, 1, 3], zz=zb, p=pb) == ok, gap
    # slot order: two near-equal logits may come in either order, not clearly inverted ones
    for gap, ok in ((4e-7, True), (4e-6, False)):
        zo = [2.0 + gap, 2.0, 0.5, -1.0, -2.0, -3.0]
        po, _, _ = _tok(zo, [1, 0, 2])
        assert adm([1, 1, 1], 0.0, gidx=[1, 0, 2], zz=zo, p=po) == ok, gap
    # m_min = 2 restore: slots 1 and 2 have near-equal c (tables offset the gates), all three
    # non-top-1 slots are below tau, so exactly one is restored, the one with the largest c
    z4 = [3.0, 2.0, 1.5, 1.0, -1.0, -2.0]
    i4 = [0, 1, 2, 3]
    e4 = np.exp(np.asarray(z4) - 3.0)
    g4 = e4[i4] / e4[i4].sum()
    for delta, tie in ((1e-6, True), (1e-3, False)):
        a4 = np.ones(6)
        a4[2] = (g4[1] / g4[2]) * (1.0 - delta)            # s_2 = s_1 (1 - delta)
        p4, _, c4 = _tok(z4, i4, a4)
        assert c4[1] > c4[2] > c4[3] and (abs(c4[1] - c4[2]) < _TB) == tie, (c4, delta)
        tau4 = c4[1] + 0.05
        assert adm([1, 1, 0, 0], tau4, gidx=i4, zz=z4, p=p4, a=a4, m_min=2)
        assert adm([1, 0, 1, 0], tau4, gidx=i4, zz=z4, p=p4, a=a4, m_min=2) == tie
        assert not adm([1, 0, 0, 1], tau4, gidx=i4, zz=z4, p=p4, a=a4, m_min=2), "restored the lowest c"
        assert not adm([1, 1, 1, 0], tau4, gidx=i4, zz=z4, p=p4, a=a4, m_min=2), "restored one too many"
        assert not adm([1, 0, 0, 0], tau4, gidx=i4, zz=z4, p=p4, a=a4, m_min=2), "m_min not met"


def check_ties_compare_decisions():
    """Token 0 clear and equal; token 1 clear but different (a mismatch); token 2
    tied (c within the band) and differing admissibly; token 3 tied and differing
    inadmissibly (a clearly kept slot skipped)."""
    T = oracle.ties
    eps = 1e-6
    ones = np.ones(6)
    z0 = [2.0, 1.0, 0.5, -1.0, -2.0, -3.0]
    idx = [0, 1, 2]
    _, _, c0 = _tok(z0, idx)
    tau = c0[2] + 5e-7                       # tokens 2 and 3: slot 2 within the band of tau
    z1 = [2.0, 1.0, 0.0, -1.0, -2.0, -3.0]  # tokens 0 and 1: slot 2's c far below tau
    _, _, c1 = _tok(z1, idx)
    assert abs(c1[2] - tau) > 1e-3
    zs = np.array([z1, z1, z0, z0])
    pis = np.stack([_tok(zz, idx)[0] for zz in zs])
    cs = np.stack([c1, c1, c0, c0])
    okeep = np.array([[1, 1, 0], [1, 1, 0], [1, 1, 0], [1, 1, 0]], bool)
    oidx = np.array([idx] * 4)
    gkeep = np.array([[1, 1, 0], [1, 1, 1], [1, 1, 1], [1, 0, 0]], bool)
    # token 1: c1[2] is clearly below tau, so the oracle skips it; keeping it is a mismatch
    assert c1[2] < tau
    rep = T.compare_decisions(zs, pis, oidx, okeep, cs, oidx.copy(), gkeep, ones, ones, tau, 1, eps)
    assert rep["n_tokens"] == 4
    assert rep["tied"] == [2, 3], rep
    assert rep["mismatch_untied"] == [1], rep
    assert rep["differing_tied"] == [2, 3], rep
    assert rep["inadmissible"] == [3], rep
    # identical decisions everywhere: tied tokens are still counted, nothing else reported
    rep = T.compare_decisions(zs, pis, oidx, okeep, cs, oidx.copy(), okeep.copy(), ones, ones, tau, 1, eps)
    assert rep["tied"] == [2, 3] and not rep["mismatch_untied"] and not rep["differing_tied"]
    assert not rep["inadmissible"]


ALL_CHECKS = [v for k, v in sorted(globals().items()) if k.startswith("check_")]
