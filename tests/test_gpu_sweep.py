"""GPU parity over a seeded sweep of layer configurations.

Each case draws a shape (tokens, hidden, experts, top-k, intermediate), dtype,
m_min, skip budget, contribution rule, optional shared expert, optional Zipf
router bias and optional plain top-k mode from a fixed seed, maps the budget to
a threshold with the oracle (App. C.1), and checks the HIP layer against the
fp64 oracle exactly as the named parity tests do: routing, masks and the plan
bit-exact (tied tokens admissible), gates and scores to 2e-6, outputs to the
dtype's tolerance.  Shapes stay within what the oracle finishes in seconds."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import device_layer, full_check

pytestmark = pytest.mark.gpu


def _cases(n=40, seed=2609):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if i % 5 == 4 else "bf16"
        d = int(rng.choice([128, 256, 384, 512, 768, 1024]))
        N = int(rng.integers(2, 97))
        k = 1 if i % 11 == 10 else int(rng.integers(2, min(8, N) + 1))
        m = 64 * int(rng.integers(1, 9))
        T = int(rng.choice([1, 2, 7, 16, 17, 33, 64, 65, 100, 257, 600]))
        m_min = 1 if rng.random() < 0.6 else int(rng.integers(1, k + 1))
        q = 0.0 if i % 13 == 0 else float(rng.choice([0.15, 0.3, 0.5, 0.6, 0.75]))
        fusion = str(rng.choice(["max", "max", "max", "min", "mean", "gsp", "rcr", "score"]))
        m_shared = 64 * int(rng.integers(1, 5)) if i % 4 == 1 else 0
        zipf = 1.1 if i % 3 == 2 else 0.0
        skip_disable = i % 7 == 6
        out.append(dict(i=i, dtype=dtype, T=T, d=d, N=N, k=k, m=m, m_min=m_min, q=q, fusion=fusion,
                        m_shared=m_shared, zipf=zipf, skip_disable=skip_disable, seed=300 + i))
    return out


CASES = _cases()


def _id(c):
    return ("{i}_{dtype}_T{T}_d{d}_N{N}_k{k}_m{m}_mmin{m_min}_q{q}_{fusion}_ms{m_shared}_z{zipf}"
            "{sd}").format(sd="_topk" if c["skip_disable"] else "", **c)


@pytest.mark.parametrize("c", CASES, ids=_id)
def test_sweep(c):
    cfg = synth.config("prefill_4096", T=c["T"], d=c["d"], N=c["N"], k=c["k"], m=c["m"], dtype=c["dtype"],
                       n_shared=1 if c["m_shared"] else 0, m_shared=c["m_shared"], zipf_s=c["zipf"],
                       seed=c["seed"])
    L = synth.make_layer(cfg)
    tb = oracle.tables.build_tables(L)
    base = oracle.forward.moe_forward(L, cfg.k, tb["a_gsp"], tb["a_rcr"], tau=0.0, m_min=c["m_min"], tokens=[],
                                      fusion=c["fusion"])
    tau = float(np.float32(oracle.tau.tau_table([base["c"]], c["m_min"], [c["q"]])[c["q"]]))
    r = full_check(L, device_layer(L), tb["a_gsp"], tb["a_rcr"], tau, m_min=c["m_min"],
                   skip_disable=c["skip_disable"], fusion=c["fusion"])
    keep = r["gpu"]["keep"].astype(bool)
    assert keep[:, 0].all(), "top-1 skipped"
    assert (keep.sum(axis=1) >= c["m_min"]).all(), "fewer than m_min slots kept"
    if c["skip_disable"]:
        assert keep.all()
    print(f"[{_id(c)}] tau={tau:.4g} skip={1 - keep.mean():.3f} rel_l2={r['rel_l2']:.2e} "
          f"tied={len(r['ties']['tied'])}", flush=True)
