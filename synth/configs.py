"""Workload shapes for the ACE MoE layer.

The shapes stand in for the MoE layers of the models the paper evaluates
(30B-total / 3B-active class: hidden 2048, 128 experts, top-8, expert
intermediate 768).  The paper's own models and benchmarks are not used.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int            # tokens
    d: int            # hidden size
    N: int            # routed experts
    k: int            # top-k
    m: int            # expert intermediate size
    dtype: str = "bf16"   # "bf16" or "f32": x, gamma and every weight
    n_shared: int = 0     # 0 or 1 always-on shared expert
    m_shared: int = 0     # its intermediate size
    zipf_s: float = 0.0   # >0: per-expert router bias -s*ln(rank)
    seed: int = 0
    x_std: float = 1.0
    gamma_std: float = 0.1    # gamma ~ 1 + N(0, gamma_std)
    w_std: float = 0.02       # router and expert weights ~ N(0, w_std)

    def with_(self, **kw) -> "LayerConfig":
        return replace(self, **kw)


CONFIGS = {
    # tiny fp32 layer: parity in fp32, oracle well under a second
    "tiny_f32": LayerConfig("tiny_f32", T=64, d=256, N=8, k=2, m=512, dtype="f32"),
    # 30B-A3B-shaped layer, 4096-token prefill
    "prefill_4096": LayerConfig("prefill_4096", T=4096, d=2048, N=128, k=8, m=768),
    # the same layer in decode (T is the decode batch: 1, 8, 32 or 64)
    "decode": LayerConfig("decode", T=32, d=2048, N=128, k=8, m=768),
    # wider pool with one shared expert and Zipf-skewed expert popularity
    "zipf_256": LayerConfig("zipf_256", T=8192, d=2048, N=256, k=8, m=512,
                            n_shared=1, m_shared=512, zipf_s=1.1),
    # one layer of the 48-layer stack (layer l is make_layer(cfg, layer=l)); 8192-token prefill
    "stack_48": LayerConfig("stack_48", T=8192, d=2048, N=128, k=8, m=768),
}

STACK_LAYERS = 48


def config(name: str, **overrides) -> LayerConfig:
    return CONFIGS[name].with_(**overrides)
