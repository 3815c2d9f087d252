"""Batches of one token.  Their router picks the top-k by rank (each expert's
(logit, id) key counted against every other key) where larger batches sort each
lane's candidates and run arg-max rounds over 16 lanes (Sec. 3.1 top-k, then
Alg. 4 on the chosen slots).  For every router tile count (N = 8 .. 256), in
bf16 and fp32: decisions, gates, scores, plan and output of the one token
against the oracle, and its routing outputs bit-identical to the same token's
in a two-token batch (the sorting path), also with exactly tied logits
(duplicated router rows: the lower expert id comes first)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import DEV, device_layer, full_check, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # (N, k, m_min, dtype)
    (8, 2, 1, "bf16"),
    (16, 1, 1, "f32"),
    (30, 4, 2, "bf16"),
    (64, 8, 1, "f32"),
    (128, 8, 1, "bf16"),
    (128, 8, 3, "f32"),
    (200, 6, 1, "bf16"),
    (256, 8, 2, "bf16"),
]


def _layer(N, k, dtype, tie):
    L = synth.make_layer(synth.config("prefill_4096", T=2, d=128, N=N, k=k, m=64, dtype=dtype, seed=90 + N))
    if tie:
        # experts 3 and 5 get twice the router row of token 0's top expert (an
        # exact scaling), so the pair leads its top-k with exactly equal logits
        tb = oracle.tables.build_tables(L)
        top = int(oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=0.0, tokens=[])["topk_idx"][0, 0])
        w = np.array(L["w_router"], copy=True)
        w[3] = w[top] * 2
        w[5] = w[3]
        L = dict(L, w_router=w)
    return L


def _one(L):
    return dict(L, x=L["x"][:1], cfg=L["cfg"].with_(T=1))


@pytest.mark.parametrize("tie", [False, True], ids=["distinct", "tied"])
@pytest.mark.parametrize("N,k,m_min,dtype", CASES, ids=[f"N{n}_k{k}_mmin{mm}_{dt}" for n, k, mm, dt in CASES])
def test_one_token(N, k, m_min, dtype, tie):
    L = _layer(N, k, dtype, tie)
    tb = oracle.tables.build_tables(L)
    base = oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=0.0, m_min=m_min, tokens=[])
    tau = float(oracle.tau.tau_table([base["c"]], m_min, [0.5])[0.5])
    if tie:
        lead = [3, 5][:k]
        top = base["topk_idx"][0]
        assert list(top[:2]) == lead, top  # the oracle orders the tied pair by id too
    D = device_layer(L)
    # the one token against the oracle
    r = full_check(_one(L), dict(D, x=D["x"][:1]), tb["a_gsp"], tb["a_rcr"], tau, m_min=m_min)
    # ... and against the same token in a two-token batch
    one = run_gpu(D, tb["a_gsp"], tb["a_rcr"], k, tau, x=D["x"][:1], m_min=m_min, write_scores=True)
    two = run_gpu(D, tb["a_gsp"], tb["a_rcr"], k, tau, x=D["x"][:2], m_min=m_min, write_scores=True)
    for key in ("topk_idx", "keep", "gates", "scores"):
        assert np.array_equal(one[key][0], two[key][0]), key
    if tie:
        assert list(one["topk_idx"][0][:2]) == lead
    print(f"[one token N={N} k={k} m_min={m_min} {dtype} tie={tie}] kept={int(one['keep'].sum())} "
          f"rel_l2={r['rel_l2']:.2e}", flush=True)
