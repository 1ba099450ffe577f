"""Pins for bf16 rounding (oracle.numerics) against the format and a library conversion."""
import numpy as np
import torch

from oracle.numerics import as_float64, bf16_bits_to_float, round_bf16


def test_round_bf16_ties_to_even_hand_values():
    # spacing of bf16 in [1, 2) is 2**-7
    assert round_bf16(1.0 + 2.0**-8) == 1.0  # tie between 1 and 1+2^-7 -> even (1.0)
    assert round_bf16(1.0 + 3 * 2.0**-8) == 1.0 + 2.0**-6  # tie between 1+2^-7 (odd) and 1+2^-6 (even)
    assert round_bf16(1.0 + 2.0**-8 + 2.0**-20) == 1.0 + 2.0**-7  # just above the tie rounds up
    assert round_bf16(-(1.0 + 2.0**-8)) == -1.0
    assert round_bf16(0.0) == 0.0
    assert round_bf16(3.0) == 3.0
    assert round_bf16(255.5) == 256.0  # spacing 1 in [128, 256): 255.5 ties to even 256
    assert round_bf16(2.0**-126 * 1.5) == 2.0**-126 * 1.5  # smallest binade keeps 8 bits


def test_round_bf16_matches_torch_conversion_of_fp32():
    g = torch.Generator().manual_seed(7)
    x = torch.randn(200000, generator=g) * torch.exp(torch.randn(200000, generator=g) * 4)
    # add exact ties: fp32 bit patterns whose low 16 bits are 0x8000
    bits = torch.randint(0x00800000, 0x7F000000, (50000,), generator=g, dtype=torch.int64)
    bits = (bits & ~0xFFFF) | 0x8000
    ties = torch.from_numpy(bits.to(torch.int32).numpy().view(np.float32))
    x = torch.cat([x, ties, -ties])
    ref = x.to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(x.numpy().astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_bit_decoding():
    t = torch.tensor([1.0, -2.5, 0.0078125, 3.0e38, -1.0e-30]).to(torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits_to_float(bits), t.to(torch.float64).numpy())
    assert np.array_equal(as_float64(bits), t.to(torch.float64).numpy())
    assert as_float64(np.array([1.5], dtype=np.float32))[0] == 1.5


def test_round_bf16_is_idempotent_and_monotone():
    rng = np.random.default_rng(3)
    x = np.sort(rng.standard_normal(100000) * 100)
    r = round_bf16(x)
    assert np.array_equal(round_bf16(r), r)
    assert np.all(np.diff(r) >= 0)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0**-8)
