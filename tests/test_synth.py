"""The seeded input generators: determinism and bf16 rounding (no GPU)."""
import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -1e-40], np.float32)])
    ours = synth.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(synth.f32_to_bf16_bits(back), ours)


def test_layer_is_deterministic_and_representable():
    c = synth.config("prefill_4096", T=33, d=128, N=8, k=2, m=64)
    a, b = synth.make_layer(c), synth.make_layer(c)
    for key in ("x", "gamma", "w_router", "w_gate", "w_up", "w_down"):
        assert np.array_equal(a[key], b[key])
        v = a[key]
        assert np.array_equal(synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(v)), v)
    assert abs(a["x"].std() - 1.0) < 0.05
    assert abs(a["w_gate"].std() - 0.02) < 0.001
    assert abs(a["gamma"].mean() - 1.0) < 0.05
    c2 = c.with_(seed=1)
    assert not np.array_equal(synth.make_layer(c2)["x"], a["x"])


def test_zipf_bias_and_shared_expert():
    c = synth.config("zipf_256", T=8, d=64, N=16, m=32, m_shared=32)
    L = synth.make_layer(c)
    ranks = np.rint(np.exp(-L["b_router"].astype(np.float64) / 1.1)).astype(int)
    assert sorted(ranks.tolist()) == list(range(1, 17))
    assert L["ws_gate"].shape == (32, 64) and L["ws_down"].shape == (64, 32)


def test_decode_steps_differ():
    c = synth.config("decode", d=64)
    a, b = synth.decode_inputs(c, 4, 0), synth.decode_inputs(c, 4, 1)
    assert a.shape == (4, 64) and not np.array_equal(a, b)
