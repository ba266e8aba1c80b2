"""Pins for the oracle's bf16 rounding (``f64_to_bf16_bits``): IEEE round to nearest, ties to even,
at bf16's 8 significant bits over float32's exponent range."""
import numpy as np
import torch

from oracle import ffd_oracle as O


def bits(x):
    return int(O.f64_to_bf16_bits(np.array([x], dtype=np.float64))[0])


def test_hand_values_ties_to_even():
    assert bits(1.0) == 0x3F80
    assert bits(1 + 2 ** -7) == 0x3F81
    assert bits(1 + 2 ** -8) == 0x3F80                 # tie, even neighbour 1.0
    assert bits(1 + 3 * 2 ** -8) == 0x3F82             # tie, even neighbour 1 + 2^-6
    assert bits(-(1 + 3 * 2 ** -8)) == 0xBF82
    assert bits(1 + 2 ** -8 + 2 ** -30) == 0x3F81      # just above the tie: up, not a double rounding
    assert bits(1 + 2 ** -8 - 2 ** -40) == 0x3F80
    assert bits(3.0) == 0x4040 and bits(-2.5) == 0xC020
    assert bits(0.1) == 0x3DCD                         # 0.1 = 0x3DCCCCCD in float32


def test_overflow_nan_inf_and_zeros():
    top = (2 - 2 ** -7) * 2.0 ** 127                   # largest finite bf16
    assert bits(top) == 0x7F7F
    assert bits((2 - 2 ** -8) * 2.0 ** 127) == 0x7F80  # tie with 2^128, odd neighbour: overflow
    assert bits((2 - 2 ** -8) * 2.0 ** 127 - 2.0 ** 100) == 0x7F7F
    assert bits(-(2 - 2 ** -8) * 2.0 ** 127) == 0xFF80
    assert bits(1e300) == 0x7F80 and bits(-1e300) == 0xFF80
    assert bits(np.inf) == 0x7F80 and bits(-np.inf) == 0xFF80
    assert bits(np.nan) == 0x7FC0 and bits(-np.nan) == 0xFFC0
    assert bits(0.0) == 0x0000 and bits(-0.0) == 0x8000


def test_subnormals():
    assert bits(2.0 ** -133) == 0x0001                 # smallest subnormal
    assert bits(2.0 ** -134) == 0x0000                 # tie with 0: even
    assert bits(-(2.0 ** -134)) == 0x8000
    assert bits(2.0 ** -134 + 2.0 ** -170) == 0x0001
    assert bits(3 * 2.0 ** -134) == 0x0002             # tie between 1 and 2 quanta: even
    assert bits(127 * 2.0 ** -133) == 0x007F           # largest subnormal
    assert bits(2.0 ** -126) == 0x0080                 # smallest normal
    assert bits(127.5 * 2.0 ** -133) == 0x0080         # tie, even neighbour: the smallest normal
    assert bits(1e-300) == 0x0000


def test_every_bf16_value_round_trips():
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = O.bf16_to_f64(allbits)
    finite = ~np.isnan(vals)
    assert np.array_equal(O.f64_to_bf16_bits(vals[finite]), allbits[finite])


def test_float32_inputs_match_the_library_conversion():
    """On float32 inputs (exact in float64) the rounding is torch's float32 -> bfloat16 conversion,
    an independent round-to-nearest-even routine: random bit patterns and every bf16 value with
    each of the 2^16 low halves' representative offsets (ties, just above, just below)."""
    rng = np.random.default_rng(5)
    u = rng.integers(0, 2 ** 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    hi = np.arange(65536, dtype=np.uint32) << np.uint32(16)
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    u = np.concatenate([u, (hi[:, None] | lows[None, :]).ravel()])
    f = u.view(np.float32)
    f = f[~np.isnan(f)]
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.f64_to_bf16_bits(f.astype(np.float64)), ref)
