"""Pins of the oracle's number formats and int4 packing against library
routines and hand-derived values (CPU only)."""
import numpy as np
import pytest
import torch

from oracle import sq_oracle as O


def test_bf16_rne_hand_cases():
    # 1 + 2^-8 lies exactly between 1 and 1 + 2^-7: ties to the even mantissa (1.0).
    # 1 + 3*2^-8 lies between 1 + 2^-7 (odd) and 1 + 2^-6 (even): goes up.
    # 1 + 2^-8 + 2^-20 is above the tie: rounds up to 1 + 2^-7.
    x = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-8 + 2**-20, -2.0, 0.0], dtype=np.float32)
    want = np.array([0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC000, 0x0000], dtype=np.uint16)
    assert np.array_equal(O.f32_to_bf16_bits(x), want)


def test_bf16_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
        (rng.integers(0, 2**31 - 2**23, 20000, dtype=np.int64) & ~0xFFFF | 0x8000).astype(np.uint32).view(np.float32),
    ]).astype(np.float32)
    x = x[np.isfinite(x)]
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.f32_to_bf16_bits(x), ref)
    assert np.array_equal(O.bf16_bits_to_f32(ref), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_f16_hand_cases_and_torch():
    x = np.array([65504.0, 65520.0, 2.0**-24, 2.0**-25, 3 * 2.0**-26, 1.0 / 3.0], dtype=np.float32)
    want = np.array([0x7BFF, 0x7C00, 0x0001, 0x0000, 0x0001, 0x3555], dtype=np.uint16)
    assert np.array_equal(O.f32_to_f16_bits(x), want)
    rng = np.random.default_rng(2)
    y = (rng.standard_normal(50000) * 10.0 ** rng.integers(-9, 5, 50000)).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.f32_to_f16_bits(y), ref)


def test_int4_pack_fixture():
    # Byte 4g+b = code(8g+b) in the low nibble | code(8g+b+4) in the high nibble.
    codes = np.array([[0, 1, 2, 3, 4, 5, 6, 7],
                      [-1, -1, -1, -1, -1, -1, -1, -1],
                      [-8, 7, -7, 1, 0, -1, 3, -3]], dtype=np.int8)
    want = np.array([[0x40, 0x51, 0x62, 0x73],
                     [0xFF, 0xFF, 0xFF, 0xFF],
                     [0x08, 0xF7, 0x39, 0xD1]], dtype=np.uint8)
    assert np.array_equal(O.pack_int4(codes), want)
    assert np.array_equal(O.unpack_int4(want), codes)


@pytest.mark.parametrize("K", [8, 64, 136])
def test_int4_roundtrip(K):
    rng = np.random.default_rng(K)
    codes = rng.integers(-8, 8, size=(7, K)).astype(np.int8)
    assert np.array_equal(O.unpack_int4(O.pack_int4(codes)), codes)
