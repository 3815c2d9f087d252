"""Seeded generators for the ACE MoE layer inputs.

Every tensor is cut into blocks along its first axis (one expert of a weight
stack, or 256 rows of a matrix), and block c comes from its own stream
``PCG64(SeedSequence([seed, layer, tensor_id, c]))``, so blocks can be drawn in
parallel.  Values are drawn in fp64, scaled, then rounded to the storage dtype
(fp32, or fp32 then bf16 with round-to-nearest-even).  The arrays returned are float32 arrays whose values
are exactly representable in the storage dtype, so the GPU and the oracle see
the same numbers.

Tensor ids: x=0, gamma=1, router=2, gate=3, up=4, down=5, Zipf permutation=6,
shared gate/up/down=7/8/9, decode step s = 100+s.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import LayerConfig

TID_X, TID_GAMMA, TID_ROUTER, TID_GATE, TID_UP, TID_DOWN = 0, 1, 2, 3, 4, 5
TID_ZIPF, TID_SGATE, TID_SUP, TID_SDOWN = 6, 7, 8, 9
TID_DECODE0 = 100


def rng_for(seed: int, layer: int, tensor_id: int, block: int | None = None) -> np.random.Generator:
    key = [seed, layer, tensor_id] if block is None else [seed, layer, tensor_id, block]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the bits as uint16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(a)
    if nan.any():
        rounded = np.where(nan, (u >> 16) | 0x40, rounded)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _to_dtype(a64: np.ndarray, dtype: str) -> np.ndarray:
    a32 = a64.astype(np.float32)
    if dtype == "f32":
        return a32
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(a32))
    raise ValueError(f"unknown dtype {dtype!r}")


def _normal(cfg: LayerConfig, layer: int, tid: int, shape, std: float, mean: float = 0.0) -> np.ndarray:
    """N(mean, std) draws of `shape`, block by block along axis 0 (see module doc)."""
    shape = tuple(shape)
    out = np.empty(shape, dtype=np.float32)
    rows = shape[0]
    step = 1 if len(shape) == 3 else 256
    blocks = [(c, r0, min(rows, r0 + step)) for c, r0 in enumerate(range(0, rows, step))]

    def fill(blk):
        c, r0, r1 = blk
        g = rng_for(cfg.seed, layer, tid, c)
        out[r0:r1] = _to_dtype(mean + std * g.standard_normal((r1 - r0,) + shape[1:]), cfg.dtype)

    if len(blocks) == 1:
        fill(blocks[0])
    else:
        with ThreadPoolExecutor(max_workers=_workers()) as ex:
            list(ex.map(fill, blocks))
    return out


def make_layer(cfg: LayerConfig, layer: int = 0) -> dict:
    """All inputs of one MoE layer (activations, RMSNorm gamma, router, experts)."""
    T, d, N, m = cfg.T, cfg.d, cfg.N, cfg.m
    out = {
        "cfg": cfg,
        "x": _normal(cfg, layer, TID_X, (T, d), cfg.x_std),
        "gamma": _normal(cfg, layer, TID_GAMMA, (d,), cfg.gamma_std, mean=1.0),
        "w_router": _normal(cfg, layer, TID_ROUTER, (N, d), cfg.w_std),
        "w_gate": _normal(cfg, layer, TID_GATE, (N, m, d), cfg.w_std),
        "w_up": _normal(cfg, layer, TID_UP, (N, m, d), cfg.w_std),
        "w_down": _normal(cfg, layer, TID_DOWN, (N, d, m), cfg.w_std),
        "b_router": None,
        "ws_gate": None, "ws_up": None, "ws_down": None,
    }
    if cfg.zipf_s > 0:
        # expert popularity ~ rank^-s: a logit bias of -s*ln(rank), ranks a seeded permutation
        ranks = rng_for(cfg.seed, layer, TID_ZIPF).permutation(N) + 1
        out["b_router"] = (-cfg.zipf_s * np.log(ranks.astype(np.float64))).astype(np.float32)
    if cfg.n_shared:
        ms = cfg.m_shared
        out["ws_gate"] = _normal(cfg, layer, TID_SGATE, (ms, d), cfg.w_std)
        out["ws_up"] = _normal(cfg, layer, TID_SUP, (ms, d), cfg.w_std)
        out["ws_down"] = _normal(cfg, layer, TID_SDOWN, (d, ms), cfg.w_std)
    return out


def decode_inputs(cfg: LayerConfig, batch: int, step: int, layer: int = 0) -> np.ndarray:
    """Fresh N(0,1) decode-step activations [batch, d] for step `step`."""
    return _normal(cfg.with_(T=batch), layer, TID_DECODE0 + step, (batch, cfg.d), cfg.x_std)
