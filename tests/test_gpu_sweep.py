"""GPU parity over a seeded sweep of layer configurations.

Each case draws a shape (tokens, hidden, experts, top-k, intermediate), dtype,
m_min, skip budget, contribution rule, optional shared expert, optional Zipf
router bias and optional plain top-k mode from a fixed seed, maps the budget to
a threshold with the oracle (App. C.1), and checks the HIP layer against the
fp64 oracle exactly as the named parity tests do: routing, masks and the plan
bit-exact (tied tokens admissible), gates and scores to 2e-6, outputs to the
dtype's tolerance (every token up to 300 tokens, every seventh and the last
beyond).  Shapes stay within what the oracle finishes in seconds."""
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


def _cases_wide(n=60, seed=77):
    """Wider ranges: up to 256 experts (every router tile count), single tokens, hidden
    sizes up to 2048 for small batches, batches past 256 tokens (outputs then on a
    token sample), shared experts of the routed experts' own width (extra M tiles of
    the routed launches) and stronger Zipf skews."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if rng.random() < 0.2 else "bf16"
        N = int(rng.choice([int(rng.integers(1, 40)), int(rng.integers(40, 129)), int(rng.integers(129, 257))]))
        k = int(rng.integers(1, min(8, N) + 1))
        T = int(rng.choice([1, 1, 2, 3, 5, 8, 15, 16, 31, 48, 63, 64, 65, 130, 255, 256, 257, 511, 700, 1100]))
        d = int(rng.choice([128, 256, 384, 640, 1024, 2048])) if T <= 64 else int(rng.choice([128, 256, 384, 512]))
        m = 64 * int(rng.integers(1, 13)) if T <= 256 else 64 * int(rng.integers(1, 7))
        m_min = 1 if rng.random() < 0.6 else int(rng.integers(1, k + 1))
        q = float(rng.choice([0.0, 0.2, 0.4, 0.5, 0.7, 0.9]))
        fusion = str(rng.choice(["max"] * 5 + ["min", "mean", "gsp", "rcr", "score"]))
        m_shared = 64 * int(rng.integers(1, 9)) if rng.random() < 0.3 else 0
        if m_shared and rng.random() < 0.4:
            m_shared = m
        zipf = float(rng.choice([0.0, 0.0, 0.8, 1.1, 1.5]))
        skip_disable = bool(rng.random() < 0.1)
        out.append(dict(i=100 + i, dtype=dtype, T=T, d=d, N=N, k=k, m=m, m_min=m_min, q=q, fusion=fusion,
                        m_shared=m_shared, zipf=zipf, skip_disable=skip_disable, seed=5000 + i))
    return out


CASES = _cases() + _cases_wide()


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
    toks = None if c["T"] <= 300 else sorted(set(range(0, c["T"], 7)) | {c["T"] - 1})
    r = full_check(L, device_layer(L), tb["a_gsp"], tb["a_rcr"], tau, m_min=c["m_min"],
                   skip_disable=c["skip_disable"], fusion=c["fusion"], tokens=toks)
    keep = r["gpu"]["keep"].astype(bool)
    assert keep[:, 0].all(), "top-1 skipped"
    assert (keep.sum(axis=1) >= c["m_min"]).all(), "fewer than m_min slots kept"
    if c["skip_disable"]:
        assert keep.all()
    print(f"[{_id(c)}] tau={tau:.4g} skip={1 - keep.mean():.3f} rel_l2={r['rel_l2']:.2e} "
          f"tied={len(r['ties']['tied'])}", flush=True)
