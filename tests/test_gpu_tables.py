"""GPU table builder (`ace_build_tables`, Alg. 2 GSP and Alg. 3 RCR in fp64) against
the oracle's fp64 tables on the same weights: fp64 values within 1e-10 relative
(summation order only), the fp32 tables handed to the layer within one ulp."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_05228_amd as ace
import synth
from gpu_helpers import device_layer

import os, sys  # noqa: E401
sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))

pytestmark = pytest.mark.gpu


def _ulps(a, b):
    ia = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    ib = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(ia - ib)


def _gpu_tables(L):
    D = device_layer(L)
    r = ace.build_tables(D, want_f64=True)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in r.items()}


def _compare(g, want64, name):
    for key in ("a_gsp", "a_rcr"):
        rel = np.max(np.abs(g[key + "64"] - want64[key]) / np.abs(want64[key]))
        ul = _ulps(g[key], want64[key].astype(np.float32))
        print(f"[tables {name}] {key}: max rel {rel:.2e}, fp32 ulps max {ul.max()} ({(ul > 0).sum()} differ)",
              flush=True)
        assert rel < 1e-10, (key, rel)
        assert ul.max() <= 1, (key, ul.max())


@pytest.mark.parametrize("shape", [
    ("tiny_f32", {}),
    ("tiny_f32", dict(T=8, d=128, N=12, k=3, m=64, seed=3)),
    ("prefill_4096", dict(T=8, d=256, N=16, k=4, m=192, seed=7)),
    ("prefill_4096", dict(T=8, d=128, N=40, k=6, m=320, seed=7)),
    ("zipf_256", dict(T=8, d=256, N=32, k=4, m=128, m_shared=192)),
], ids=lambda s: f"{s[0]}_{s[1]}")
def test_tables_small(shape):
    name, kw = shape
    L = synth.make_layer(synth.config(name, **kw))
    tb = oracle.tables.build_tables(L)
    _compare(_gpu_tables(L), {"a_gsp": tb["a_gsp64"], "a_rcr": tb["a_rcr64"]}, f"{name} {kw}")


@pytest.mark.parametrize("name", ["prefill_4096", "zipf_256"])
def test_tables_full_size(name):
    """Against the stored oracle tables of the full-size workloads (fp32, from fp64)."""
    import make_tables
    gold = make_tables.load(name)
    L = synth.make_layer(synth.config(name, T=16))
    g = _gpu_tables(L)
    for key in ("a_gsp", "a_rcr"):
        ul = _ulps(g[key], np.array(gold[key], np.float32))
        print(f"[tables {name}] {key}: fp32 ulps max {ul.max()} ({(ul > 0).sum()} of {ul.size} differ)", flush=True)
        assert ul.max() <= 1


def test_tables_deterministic():
    L = synth.make_layer(synth.config("prefill_4096", T=8, d=256, N=16, k=4, m=192, seed=2))
    a, b = _gpu_tables(L), _gpu_tables(L)
    for key in a:
        assert np.array_equal(a[key], b[key])
