"""GPU threshold mapping (App. C.1, `ace_tau_map`) against the oracle's mapping
on the same fp32 scores: tau (fp32), m_q and N_cand are bit-exact, including
boundary ties, the clip branches, m_min > 1 and several layers in one pass."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_05228_amd as ace
import synth
from gpu_helpers import DEV, device_layer, run_gpu

pytestmark = pytest.mark.gpu

QS = [0.0, 0.1, 0.25, 0.5, 0.6, 0.875, 1.0]


def _oracle(c_list, m_min, qs):
    """Oracle taus (rounded once to fp32), m_q and N_cand for the given score arrays."""
    c_list = [np.asarray(c, np.float64) for c in c_list]
    taus = oracle.tau.tau_table(c_list, m_min, qs)
    n_all = sum(c.size for c in c_list)
    n_cand = int(sum(oracle.tau.candidate_mask(c, m_min).sum() for c in c_list))
    m_q = [int(np.clip(np.rint(q * n_all), 0, n_cand)) for q in qs]
    return np.array([np.float32(taus[q]) for q in qs], np.float32), m_q, n_cand


def _gpu(scores_np, m_min, qs):
    s = torch.from_numpy(np.ascontiguousarray(scores_np, np.float32)).to(DEV)
    r = ace.tau_map(s, qs, m_min)
    torch.cuda.synchronize()
    return r["tau"].cpu().numpy(), r["m_q"].cpu().tolist(), int(r["n_cand"].item())


def _check(c_list, m_min, qs, name):
    want_tau, want_m, want_nc = _oracle(c_list, m_min, qs)
    got_tau, got_m, got_nc = _gpu(np.concatenate([np.asarray(c, np.float32) for c in c_list]), m_min, qs)
    print(f"[tau {name}] n_cand={got_nc} tau={got_tau.tolist()}", flush=True)
    assert got_nc == want_nc
    assert got_m == want_m
    assert np.array_equal(got_tau.view(np.uint32), want_tau.view(np.uint32)), (got_tau, want_tau)
    return got_tau


@pytest.fixture(scope="module")
def small_scores():
    """Scores of a GPU score pass over a small bf16 layer."""
    L = synth.make_layer(synth.config("prefill_4096", T=700, d=256, N=64, k=8, m=128, seed=31))
    tb = oracle.tables.build_tables(L)
    g = run_gpu(device_layer(L), tb["a_gsp"], tb["a_rcr"], 8, 0.0, write_scores=True)
    return L, tb, g["scores"]


@pytest.mark.parametrize("m_min", [1, 2, 3, 8])
def test_tau_from_layer_scores(small_scores, m_min):
    _, _, sc = small_scores
    _check([sc], m_min, QS, f"layer m_min={m_min}")


def test_tau_realises_budget(small_scores):
    """Running the layer with the GPU tau skips exactly m_q slots (no boundary tie here)."""
    L, tb, sc = small_scores
    got_tau, got_m, _ = _gpu(sc, 1, [0.5])
    g = run_gpu(device_layer(L), tb["a_gsp"], tb["a_rcr"], 8, float(got_tau[0]))
    assert int((g["keep"] == 0).sum()) == got_m[0]


def test_tau_several_layers():
    rng = np.random.default_rng(5)
    c1 = rng.dirichlet(np.ones(8), size=3000)
    c2 = rng.dirichlet(np.ones(8) * 0.5, size=2000)
    _check([c1.astype(np.float32), c2.astype(np.float32)], 1, QS, "two layers")


@pytest.mark.parametrize("m_min", [1, 2])
def test_tau_boundary_ties(m_min):
    """Scores from a small set of values: every boundary is a tie."""
    rng = np.random.default_rng(9 + m_min)
    vals = np.array([0.0, 0.01, 0.02, 0.05, 0.1, 0.2, 0.5], np.float32)
    c = vals[rng.integers(0, vals.size, size=(4000, 8))]
    qs = [0.05, 0.1, 0.2, 0.3, 0.4, 0.5, 0.7, 0.9]
    _check([c], m_min, qs, f"ties m_min={m_min}")


def test_tau_edge_cases():
    rng = np.random.default_rng(3)
    c = rng.random((50, 4)).astype(np.float32)
    tau, m, nc = _gpu(c, 4, [0.0, 0.5, 1.0])           # m_min = k: no candidates
    assert nc == 0 and m == [0, 0, 0] and np.all(tau == 0)
    tau, m, nc = _gpu(np.zeros((0, 8), np.float32), 1, [0.0, 0.5])
    assert nc == 0 and np.all(tau == 0)
    tau, m, nc = _gpu(c, 1, [1.0])                      # clip to N_cand: +inf
    assert nc == 150 and m == [150] and np.isinf(tau[0])
    _check([c], 1, [0.0, 0.3, 1.0], "edges")
    _check([rng.random((1, 2)).astype(np.float32)], 1, [0.0, 0.25, 0.5, 1.0], "one row")


def test_tau_large_pass():
    """A pass the size of a 48-layer, 8192-token model (3.1M slots)."""
    rng = np.random.default_rng(17)
    c = rng.dirichlet(np.ones(8), size=48 * 8192).astype(np.float32)
    _check([c], 1, [0.1, 0.25, 0.5, 0.6], "48x8192")


def test_tau_rejects_bad_arguments():
    s = torch.zeros((4, 8), dtype=torch.float32, device=DEV)
    for qs, m_min in (([1.5], 1), ([-0.1], 1), ([float("nan")], 1), ([0.5] * 9, 1), ([0.5], 0), ([0.5], 9)):
        with pytest.raises(ace.AceError):
            ace.tau_map(s, qs, m_min)
