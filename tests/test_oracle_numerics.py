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


# ----------------------------------------------------------------------------- fp8 (E4M3)

def test_round_fp8_e4m3_hand_values():
    from oracle.numerics import round_fp8_e4m3
    cases = [
        (1.0, 1.0), (1.0625, 1.0),    # halfway between 1 and 1.125: the even fraction (0) wins
        (1.1875, 1.25),               # halfway between 1.125 and 1.25: 1.25 (fraction 2) wins
        (-0.3, -0.3125),              # spacing 2^-5 in [0.25, 0.5)
        (448.0, 448.0), (460.0, 448.0), (470.0, 448.0), (1e6, 448.0), (-1e6, -448.0),  # saturation
        (2.0 ** -9, 2.0 ** -9),       # smallest subnormal
        (2.0 ** -10, 0.0),            # halfway between 0 and 2^-9: even (0)
        (3 * 2.0 ** -10, 2.0 ** -8),  # halfway between 2^-9 and 2^-8: even (2 * 2^-9)
        (2.0 ** -6, 2.0 ** -6),       # smallest normal
        (0.0, 0.0),
    ]
    for x, want in cases:
        assert round_fp8_e4m3(x) == want, x


def test_fp8_e4m3_matches_torch_conversion():
    import torch
    from oracle.numerics import fp8_e4m3_bits_to_float, round_fp8_e4m3
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mine = fp8_e4m3_bits_to_float(codes.numpy())
    finite = ~np.isnan(ref)
    assert np.array_equal(np.isnan(mine), ~finite)
    assert np.array_equal(mine[finite], ref[finite])
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(200000), rng.uniform(-448, 448, 100000),
                        rng.standard_normal(100000) * 2.0 ** -7]).astype(np.float32)
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(round_fp8_e4m3(x.astype(np.float64)), t)


def test_round_fp8_e4m3_is_idempotent_on_the_grid():
    from oracle.numerics import fp8_e4m3_bits_to_float, round_fp8_e4m3
    vals = fp8_e4m3_bits_to_float(np.arange(256, dtype=np.uint8))
    vals = vals[~np.isnan(vals)]
    assert np.array_equal(round_fp8_e4m3(vals), vals)
    assert len(np.unique(vals)) == 253  # 254 finite codes, +0 and -0 equal
