"""The router's exact hi/lo split, checked on the CPU.

The bf16 router computes z_e = rstd * sum_k (x_k gamma_k) w_{e,k} + b_e (the RMS
scale of Sec. 3.1's x = x_bar Gamma factored out of App. B.2's logit).  It forms
each product p = x_k gamma_k in fp32, cuts p into a bf16 high half (p with its low
16 bits cleared) and the fp32 remainder lo = p - hi, and feeds both halves to the
bf16 matrix cores against the bf16 router rows.  That is an fp32 GEMM on the
exact products only if
  1. p is exact in fp32 (two 8-bit significands give at most 16 bits),
  2. lo is exact in fp32 and has no bits below the bf16 mantissa (its low 16
     bits are zero), so that hi and lo are both bf16 values and hi + lo = p,
  3. each half times a bf16 router weight is exact in fp32.
These tests check the three facts over every bf16 x with an exponent in [-60, 60]
(and zero), against many gamma values, in numpy fp32 / fp64 arithmetic.  The
domain is every product of magnitude at least 2^-110: below that the remainder
would be an fp32 subnormal, which no layer input of RMSNorm scale comes near.
"""
import numpy as np

from synth.gen import bf16_bits_to_f32, f32_to_bf16_bits


def _split(p32):
    """The kernel's split: hi = p with its low 16 bits cleared, lo = p - hi in fp32."""
    hi = (p32.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
    lo = (p32 - hi).astype(np.float32)
    return hi, lo


def _all_bf16(min_exp=-60, max_exp=60):
    """Every finite bf16 value whose unbiased exponent lies in [min_exp, max_exp], and zero."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = bf16_bits_to_f32(bits)
    e = ((bits.astype(np.uint32) >> 7) & 0xFF).astype(np.int64) - 127
    ok = np.isfinite(v) & (((e >= min_exp) & (e <= max_exp)) | (v == 0))
    return v[ok]


def _check(x, g):
    x64, g64 = x.astype(np.float64), g.astype(np.float64)
    p32 = (x * g).astype(np.float32)
    assert np.array_equal(p32.astype(np.float64), x64 * g64), "x * gamma not exact in fp32"
    hi, lo = _split(p32)
    assert not np.any(lo.view(np.uint32) & np.uint32(0xFFFF)), "remainder has bits below bf16"
    assert np.array_equal(hi.astype(np.float64) + lo.astype(np.float64), p32.astype(np.float64))
    # the remainder is at most the weight of bf16's last mantissa bit of p
    assert np.all(np.abs(lo.astype(np.float64)) < np.abs(p32.astype(np.float64)) * 2.0 ** -7 + 1e-300)
    return hi, lo


def test_split_is_exact_for_every_bf16_input():
    x = _all_bf16()
    rng = np.random.default_rng(0)
    # gamma as the layers draw it (1 + N(0, 0.1), rounded to bf16) and bf16 values of any
    # magnitude the layer could hold
    gam = np.concatenate([1.0 + 0.1 * rng.standard_normal(96), rng.standard_normal(32) * 10.0 ** rng.uniform(-6, 6, 32)])
    gam = bf16_bits_to_f32(f32_to_bf16_bits(gam.astype(np.float32)))
    for gv in gam:
        _check(x, np.full_like(x, gv))


def test_split_halves_times_router_weights_are_exact():
    rng = np.random.default_rng(1)
    n = 1 << 20
    x = bf16_bits_to_f32(f32_to_bf16_bits(rng.standard_normal(n).astype(np.float32)))
    g = bf16_bits_to_f32(f32_to_bf16_bits((1.0 + 0.1 * rng.standard_normal(n)).astype(np.float32)))
    w = bf16_bits_to_f32(f32_to_bf16_bits((0.02 * rng.standard_normal(n)).astype(np.float32)))
    hi, lo = _check(x, g)
    for half in (hi, lo):
        prod32 = (half * w).astype(np.float32)
        assert np.array_equal(prod32.astype(np.float64), half.astype(np.float64) * w.astype(np.float64))
    # so the two products sum to the exact fp64 product of the three bf16 factors
    exact = x.astype(np.float64) * g.astype(np.float64) * w.astype(np.float64)
    assert np.array_equal((hi * w).astype(np.float64) + (lo * w).astype(np.float64), exact)


def test_split_of_a_rounded_product_would_not_be_exact():
    """Control: the exactness needs bf16 inputs.  An fp32 x (24-bit significand) times
    gamma has bits the two bf16 halves cannot hold, which is why fp32 layers take the
    fp32 matrix-core path instead."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal(4096).astype(np.float32)
    g = np.full_like(x, np.float32(1.1))
    p32 = (x * g).astype(np.float32)
    hi, lo = _split(p32)
    assert np.any(lo.view(np.uint32) & np.uint32(0xFFFF))
