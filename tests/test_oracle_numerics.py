"""Pins of the oracle's bf16 conversion (round-to-nearest-even)."""
import numpy as np
import pytest

from oracle.numerics import f32_to_bf16_bits, bf16_bits_to_f32

pytestmark = pytest.mark.cpu


def _f(u32):
    return np.array([u32], dtype=np.uint32).view(np.float32)


@pytest.mark.parametrize("u32,expect", [
    (0x3F800000, 0x3F80),      # 1.0
    (0x3F808000, 0x3F80),      # 1 + 2^-8: exact tie, lower neighbour even
    (0x3F818000, 0x3F82),      # tie, upper neighbour even
    (0x3F808001, 0x3F81),      # just above the tie
    (0x3F807FFF, 0x3F80),      # just below the tie
    (0x3FFFFFFF, 0x4000),      # carry into the exponent
    (0x7F7FFFFF, 0x7F80),      # largest float rounds to +inf
    (0x80000000, 0x8000),      # -0 keeps its sign
    (0x00000001, 0x0000),      # smallest subnormal rounds to 0
    (0xFF800000, 0xFF80),      # -inf
])
def test_rne_hand_cases(u32, expect):
    assert int(f32_to_bf16_bits(_f(u32))[0]) == expect


def test_nan_stays_nan():
    r = f32_to_bf16_bits(_f(0x7F800001))
    assert np.isnan(bf16_bits_to_f32(r))[0]


def test_matches_torch_conversion():
    import torch
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(100000) * np.exp(rng.uniform(-30, 30, 100000))).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(a), ref)


def test_roundtrip_exact():
    u = np.arange(0, 1 << 16, dtype=np.uint16)
    f = bf16_bits_to_f32(u)
    ok = ~np.isnan(f)
    assert np.array_equal(f32_to_bf16_bits(f)[ok], u[ok])
