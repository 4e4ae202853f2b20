"""Pins of the oracle's GELU (the bf16 activation between the MLP's up and
down projections, App. D) and of the chain from the up projection's output
into the down projection's STATIC quantizer.

erf follows Abramowitz & Stegun 7.1.28 in fp32; the pins hold it against the
fp64 error function of the Python standard library (something other than the
oracle itself), the closed forms of GELU, and the quantizer's identity case."""
import math

import numpy as np

from oracle import sq_oracle as O

# 7.1.28 guarantees |error| <= 3e-7; the fp32 chain (Horner, four squarings,
# a division) adds rounding, amplified 16x by the power: measured 1.8e-6.
ERF_BOUND = 2.5e-6


def all_finite_bf16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = O.bf16_bits_to_f32(bits)
    ok = np.isfinite(x)
    return bits[ok], x[ok]


def test_erf_matches_the_error_function():
    z = np.linspace(0.0, 6.0, 20001).astype(np.float32)
    e = O.erf_as(z).astype(np.float64)
    ref = np.array([math.erf(float(v)) for v in z])
    assert np.max(np.abs(e - ref)) <= ERF_BOUND
    assert O.erf_as(np.float32([0.0]))[0] == 0.0
    assert O.erf_as(np.float32([1e30, np.inf]))[0] == 1.0  # 1 / inf = 0


def test_gelu_matches_x_phi_x_on_every_bf16_value():
    """|GELU_oracle(x) - x Phi(x)| <= |x|/2 * ERF_BOUND + 3 fp32 roundings of the
    result, with x Phi(x) = x erfc(-x / sqrt 2) / 2 in fp64 (accurate for
    negative x as well)."""
    _, x = all_finite_bf16()
    g = O.gelu_f32(x).astype(np.float64)
    xx = x.astype(np.float64)
    ref = np.array([0.5 * v * math.erfc(-v / math.sqrt(2.0)) for v in xx])
    bound = 0.5 * np.abs(xx) * ERF_BOUND + 3 * np.abs(ref) * 2.0**-24 + 2.0**-149
    assert np.all(np.isfinite(g))
    assert np.all(np.abs(g - ref) <= bound)


def test_gelu_closed_forms():
    x = np.float32([0.0, -0.0, 6.0, 100.0, 3e38, -10.0, -100.0])
    g = O.gelu_f32(x)
    assert g[0] == 0.0 and not np.signbit(g[0])
    assert g[1] == 0.0 and np.signbit(g[1])
    assert np.array_equal(g[2:5], x[2:5])  # Phi(x) = 1 in fp32: GELU(x) = x exactly, no overflow
    assert np.all(g[5:] == 0.0)            # Phi(x) = 0 in fp32
    # GELU(x) - GELU(-x) = x
    _, xs = all_finite_bf16()
    xs = xs[(xs > 0) & (xs < 1e30)]
    d = O.gelu_f32(xs).astype(np.float64) - O.gelu_f32(-xs).astype(np.float64)
    assert np.all(np.abs(d - xs) <= 4 * xs.astype(np.float64) * 2.0**-24 + 2.0**-149)


def test_gelu_bf16_rounds_the_fp32_value():
    bits, x = all_finite_bf16()
    assert np.array_equal(O.gelu_bf16(bits), O.f32_to_bf16_bits(O.gelu_f32(x)))


def test_mlp_chain_identity_case():
    """STATIC thresholds c = 127 with unit gains and D = I (Delta = 1): integer
    up outputs h >= 6 pass GELU unchanged (Phi(h) = 1 in fp32) and come back as
    their own codes; h <= -10 gives GELU 0 and code 0; r = 1."""
    h = np.concatenate([np.arange(6, 128), -np.arange(10, 128)]).astype(np.float32)
    y = np.tile(h, (3, 1))
    t2s = np.array([0, 1, 2], np.int32)
    gamma = np.ones((2, 3), np.float32)
    clip = np.full(2, 127.0, np.float32)
    hb, g, qa = O.mlp_chain_codes(y, t2s, gamma, 1, None, clip)
    want = np.where(h > 0, h, 0).astype(np.int64)
    assert np.array_equal(qa["codes"].astype(np.int64), np.tile(want, (3, 1)))
    assert np.array_equal(qa["scale"], np.ones(3, np.float32))
    # a gain of 2 on stream 1 doubles its codes (saturating at 127)
    gamma[1, 1] = 2.0
    _, _, qa2 = O.mlp_chain_codes(y, t2s, gamma, 1, None, clip)
    assert np.array_equal(qa2["codes"][1].astype(np.int64), np.minimum(2 * want, 127))
    assert qa2["scale"][1] == np.float32(0.5)


def test_mlp_chain_identity_case_4bit():
    """The same with the 4-bit quantizer: c = 7 (Delta = fp16(1) = 1), unit
    gains, D = I: integer up outputs 6 and 7 come back as their own codes,
    larger ones clip to 7, h <= -10 gives code 0; every group step is fp16 1.
    A gain of 0.5 halves the codes (rounding to even)."""
    h = np.concatenate([np.arange(6, 70), -np.arange(10, 74)]).astype(np.float32)  # 128 = two 64-groups
    y = np.tile(h, (3, 1))
    t2s = np.array([0, 1, 2], np.int32)
    gamma = np.ones((2, 3), np.float32)
    clip = np.full(2, 7.0, np.float32)
    _, _, qa = O.mlp_chain_codes(y, t2s, gamma, 1, None, clip, act_bits=4)
    want = np.where(h > 0, np.minimum(h, 7), 0).astype(np.int64)
    assert np.array_equal(qa["codes"].astype(np.int64), np.tile(want, (3, 1)))
    assert np.array_equal(qa["scale"], np.full((3, 2), 0x3C00, np.uint16))
    gamma[1, 2] = 0.5
    _, _, qa2 = O.mlp_chain_codes(y, t2s, gamma, 1, None, clip, act_bits=4)
    half = np.where(h > 0, np.minimum(np.rint(h * 0.5), 7), 0).astype(np.int64)
    assert np.array_equal(qa2["codes"][2].astype(np.int64), half)
