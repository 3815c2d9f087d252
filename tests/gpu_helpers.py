"""Shared helpers of the GPU parity tests: move seeded inputs to the device, run
the HIP path through the C ABI, and compare with the CPU oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2609_05228_amd as ace

DEV = "cuda:0"
TDT = {"bf16": torch.bfloat16, "f32": torch.float32}
BAND = oracle.ties.BAND


def device_layer(L: dict, dev: str = DEV) -> dict:
    """Device copies of a synth layer (values are exact in the storage dtype)."""
    dt = TDT[L["cfg"].dtype]
    out = {}
    for key in ("x", "gamma", "w_router", "w_gate", "w_up", "w_down", "ws_gate", "ws_up", "ws_down"):
        v = L.get(key)
        out[key] = None if v is None else torch.from_numpy(v).to(dev).to(dt).contiguous()
    b = L.get("b_router")
    out["b_router"] = None if b is None else torch.from_numpy(b).to(dev)
    return out


def run_gpu(D: dict, a_gsp, a_rcr, k: int, tau: float, x=None, **kw) -> dict:
    """Run the HIP layer; return numpy copies of every output."""
    ag = torch.as_tensor(np.asarray(a_gsp, np.float32)).to(DEV)
    ar = torch.as_tensor(np.asarray(a_rcr, np.float32)).to(DEV)
    o = ace.moe_forward(D["x"] if x is None else x, D, ag, ar, k=k, tau=tau, want_plan=True, **kw)
    torch.cuda.synchronize()
    res = {}
    for key, v in o.items():
        res[key] = v.float().cpu().numpy() if v.dtype == torch.bfloat16 else v.cpu().numpy()
    return res


def check_decisions(orc: dict, gpu: dict, a_gsp, a_rcr, tau: float, m_min: int, eps: float = 1e-6,
                    fusion: str = "max"):
    """Bit-exact routing and masks, except admissible decisions of tied tokens."""
    rep = oracle.ties.compare_decisions(orc["z"], orc["pi"], orc["topk_idx"], orc["keep"], orc["c"],
                                        gpu["topk_idx"], gpu["keep"].astype(bool),
                                        np.asarray(a_gsp, np.float64), np.asarray(a_rcr, np.float64),
                                        tau, m_min, eps, fusion=fusion)
    assert not rep["mismatch_untied"], f"untied tokens differ: {rep['mismatch_untied'][:10]}"
    assert not rep["inadmissible"], f"tied tokens with inadmissible GPU decisions: {rep['inadmissible']}"
    return rep


def check_plan(gpu: dict, N: int):
    """The GPU plan equals the plan the oracle derives from the GPU's decisions."""
    p = oracle.plan.dispatch_plan(gpu["topk_idx"], gpu["keep"].astype(bool), N)
    n = int(p["offsets"][-1])
    assert np.array_equal(gpu["counts"], p["counts"])
    assert np.array_equal(gpu["offsets"], p["offsets"])
    assert np.array_equal(gpu["perm"][:n], p["perm"])


def rel_l2(a, b) -> float:
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# worst single-token relative L2 error allowed in bf16 (the aggregate bar is 1e-2): a
# token's output carries the bf16 roundings of its H row, its Y rows and y itself
# (each 2^-9 relative), so one token three times the aggregate bar is a kernel error
BF16_WORST_TOKEN = 3e-2


def check_y(y_gpu, y_ref, dtype: str, rows=None):
    """Output tolerances: fp32 rel-L2 and max-abs 1e-5; bf16 rel-L2 1e-2 over the
    checked rows and at most BF16_WORST_TOKEN on every single token."""
    if rows is not None:
        y_gpu, y_ref = y_gpu[rows], y_ref[rows]
    r = rel_l2(y_gpu, y_ref)
    per_tok = [rel_l2(y_gpu[i], y_ref[i]) for i in range(len(y_ref))] if len(y_ref) else [0.0]
    if dtype == "f32":
        assert r <= 1e-5, f"fp32 rel L2 {r}"
        assert np.max(np.abs(y_gpu - y_ref)) <= 1e-5 * np.max(np.abs(y_ref)), "fp32 max abs"
    else:
        assert r <= 1e-2, f"bf16 rel L2 {r} (worst token {max(per_tok)})"
        worst = int(np.argmax(per_tok))
        assert per_tok[worst] <= BF16_WORST_TOKEN, f"bf16 token {worst} of the checked rows: rel L2 {per_tok[worst]}"
    return r, max(per_tok)


def with_f64_weights(L: dict) -> dict:
    """The same layer with its expert weights widened to fp64 once (the oracle then
    skips the per-call conversion; the values are unchanged)."""
    out = dict(L)
    for key in ("w_gate", "w_up", "w_down", "ws_gate", "ws_up", "ws_down"):
        if out.get(key) is not None:
            out[key] = np.asarray(out[key], dtype=np.float64)
    return out


def hot_expert_tokens(topk_idx, keep, n_experts: int = 1, first_rows: int | None = None):
    """Tokens with a kept slot on the n_experts experts with the most kept rows (each
    expert's rows are its tokens in ascending order, so these tokens cover every row
    block of its M tiles); with first_rows, only the first and last that many rows of each."""
    idx = np.asarray(topk_idx)
    keep = np.asarray(keep, bool)
    counts = np.bincount(idx[keep], minlength=int(idx.max()) + 1)
    toks = set()
    for e in np.argsort(-counts, kind="stable")[:n_experts]:
        rows = np.nonzero((idx == e) & keep)[0]           # token ids in ascending order
        if first_rows is not None and rows.size > 2 * first_rows:
            rows = np.concatenate([rows[:first_rows], rows[-first_rows:]])
        toks.update(int(t) for t in rows)
    return sorted(toks)


def full_check(L: dict, D: dict, a_gsp, a_rcr, tau: float, m_min: int = 1, tokens=None,
               skip_disable: bool = False, eps: float = 1e-6, fusion: str = "max", hot=None):
    """Run GPU and oracle on the same inputs and check decisions, plan, gates and y.
    hot = (n_experts, first_rows or None): also check y on every token routed to the
    n_experts experts with the most kept rows (see hot_expert_tokens)."""
    cfg = L["cfg"]
    gpu = run_gpu(D, a_gsp, a_rcr, cfg.k, tau, m_min=m_min, skip_disable=skip_disable,
                  write_scores=True, eps=eps, fusion=fusion)
    orc = oracle.forward.moe_forward(L, cfg.k, a_gsp, a_rcr, float(np.float32(tau)), m_min=m_min, eps=eps,
                                     skip_disable=skip_disable, tokens=[], fusion=fusion)
    rep = check_decisions(orc, gpu, a_gsp, a_rcr, float(np.float32(tau)), m_min, eps, fusion)
    check_plan(gpu, cfg.N)
    same = [t for t in range(cfg.T) if t not in set(rep["differing_tied"])]
    # gates and scores where decisions agree
    assert np.allclose(gpu["gates"][same], orc["ghat"][same], rtol=2e-6, atol=2e-7), "gates"
    assert np.allclose(gpu["scores"][same], orc["c"][same], rtol=2e-6, atol=2e-7), "scores"
    toks = list(range(cfg.T)) if tokens is None else list(tokens)
    if hot is not None and tokens is not None:
        toks = sorted(set(toks) | set(hot_expert_tokens(gpu["topk_idx"], gpu["keep"], *hot)))
    ref = oracle.forward.moe_forward(L, cfg.k, a_gsp, a_rcr, float(np.float32(tau)), m_min=m_min, eps=eps,
                                     skip_disable=skip_disable, tokens=toks,
                                     decisions=(gpu["topk_idx"], gpu["keep"].astype(bool)))
    r, worst = check_y(gpu["y"], ref["y"], cfg.dtype, rows=toks)
    return dict(gpu=gpu, oracle=orc, ties=rep, rel_l2=r, worst_token=worst, n_checked=len(toks))
