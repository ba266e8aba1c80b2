"""Pins for the oracle's key decomposition (App. A formulation; Sec. 3.1 residual reading)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ffd_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def all_finite_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = O.bf16_to_f64(bits)
    return x[np.isfinite(x)]


def test_worked_example_matches_hand_computation():
    g = json.load(open(os.path.join(GOLDEN, "quantizer_worked_example.json")))
    x = np.array(g["x"], dtype=np.float64)
    codes, M, resid = O.quantize_keys(x)
    assert M == g["M"]
    assert codes.tolist() == g["codes"]
    assert resid.tolist() == g["resid"]
    assert O.thumbnail(codes, M).tolist() == g["thumbnail"]
    # the full reconstruction is M * n / 381 with the hand-derived n
    full = O.thumbnail(codes, M) + O.residual_part(resid, M)
    np.testing.assert_allclose(full, g["M"] * np.array(g["n"]) / 381.0, rtol=0, atol=1e-15)


def _exact_nearest_code(x: float, M: float) -> int:
    """Brute force over the codebook with exact rationals; a tie goes to the upper level."""
    xf, Mf = Fraction(x), Fraction(M)
    best, best_d = None, None
    for c, level in enumerate((-3, -1, 1, 3)):        # levels times 2: |x/s - lvl| ~ |3x - lvl*M|
        d = abs(3 * xf - level * Mf)
        if best_d is None or d <= best_d:             # '<=' with increasing levels -> upper wins ties
            best, best_d = c, d
    return best


@pytest.mark.parametrize("M", [1.0, 1.5, 2.5, 3.140625, 0.0078125, 117.0, 3.0e38, 1.0e-38])
def test_codes_exhaustive_over_bf16(M):
    Mb = O.bf16_to_f64(O.f64_to_bf16_bits(np.array([M])))[0]
    x = all_finite_bf16()
    x = x[np.abs(x) <= Mb]
    vec = np.stack([x, np.full_like(x, Mb)], axis=1)      # absmax of each row is Mb
    codes, Mv, _ = O.quantize_keys(vec)
    assert np.all(Mv == Mb)
    # brute force on a deterministic subsample (all values near the edges + a stride of the rest)
    s = Mb / 1.5
    edge = np.isclose(np.abs(x) / s, 1.0, rtol=1e-2) | (np.abs(x) <= s * 1e-2)
    idx = np.unique(np.concatenate([np.nonzero(edge)[0], np.arange(0, x.size, 97)]))
    for i in idx:
        assert codes[i, 0] == _exact_nearest_code(float(x[i]), float(Mb)), (x[i], Mb)
    # and the thumbnail error bound |x - x_hat| <= s/2 everywhere
    xhat = O.thumbnail(codes, Mv)[:, 0]
    assert np.all(np.abs(x - xhat) <= s / 2 * (1 + 1e-15))


def test_edges_tie_upward_and_negative_zero():
    M = 1.5                                   # s = 1, bin edges at -1, 0, +1
    x = np.array([1.0, 0.0, -0.0, -1.0, 1.5, -1.5])
    codes, _, _ = O.quantize_keys(np.concatenate([x, [M]]))
    assert codes[:6].tolist() == [3, 2, 2, 1, 3, 0]


def test_extreme_element_maps_to_outer_level_with_zero_residual():
    rng = np.random.default_rng(0)
    K = O.bf16_to_f64(O.f64_to_bf16_bits(rng.standard_normal((200, 128))))
    codes, M, resid = O.quantize_keys(K)
    i = np.argmax(np.abs(K), axis=1)
    rows = np.arange(K.shape[0])
    lvl = O.CODEBOOK[codes[rows, i]]
    assert np.all(np.abs(lvl) == 1.5)
    assert np.all(np.sign(lvl) == np.sign(K[rows, i]))
    assert np.all(resid[rows, i] == 0)


def test_zero_vector():
    codes, M, resid = O.quantize_keys(np.zeros((3, 128)))
    assert np.all(M == 0) and np.all(codes == 2) and np.all(resid == 0)
    assert np.all(O.thumbnail(codes, M) == 0)
    assert np.all(O.residual_part(resid, M) == 0)


def _exact_nearest_grid(x: float, M: float) -> int:
    """Nearest j in [-381, 381] of the grid j*M/381 (ties to even j), exact rationals."""
    t = Fraction(x) * 381 / Fraction(M)
    fl = t.numerator // t.denominator
    frac = t - fl
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and fl % 2 == 1):
        return fl + 1
    return fl


@pytest.mark.parametrize("seed", [1, 2])
def test_residual_brute_force_and_bounds(seed):
    rng = np.random.default_rng(seed)
    K = O.bf16_to_f64(O.f64_to_bf16_bits(rng.standard_normal((64, 128)) * rng.uniform(0.01, 50)))
    codes, M, resid = O.quantize_keys(K)
    assert resid.min() >= -127 and resid.max() <= 127
    n = resid + 254 * codes - 381
    for r in range(0, 64, 7):
        for c in range(128):
            assert n[r, c] == _exact_nearest_grid(float(K[r, c]), float(M[r])), (r, c)
    full = O.thumbnail(codes, M) + O.residual_part(resid, M)
    # closed form of the 2+8 reconstruction, and its error bound M/762
    assert np.all(np.abs(full - M[:, None] * n / 381.0) <= 1e-14 * M[:, None])
    assert np.all(np.abs(K - full) <= M[:, None] / 762.0 * (1 + 1e-12))


def test_residual_exhaustive_ties_to_even():
    """All bf16 values against M = 1.5: the residual grid index is rint(254 x) with ties to even."""
    x = all_finite_bf16()
    x = x[np.abs(x) <= 1.5]
    codes, M, resid = O.quantize_keys(np.stack([x, np.full_like(x, 1.5)], axis=1))
    n = resid[:, 0] + 254 * codes[:, 0] - 381
    t = x * 254.0                                   # exact: 254 * bf16 fits in float64
    fl = np.floor(t)
    fr = t - fl
    expect = np.where(fr > 0.5, fl + 1, np.where(fr < 0.5, fl, np.where(fl % 2 == 0, fl, fl + 1)))
    assert np.array_equal(n, expect.astype(np.int64))
    assert (fr == 0.5).sum() > 0                    # the sweep does contain exact ties


def test_quantization_in_pieces_equals_the_whole(monkeypatch):
    """Large inputs are quantized in pieces of rows (each row independently): same results."""
    rng = np.random.default_rng(21)
    K = O.bf16_to_f64(O.f64_to_bf16_bits(rng.standard_normal((9000, 128)) * 3))
    K[17] = 0.0
    for bits in (2, 4, 8):
        a = O.quantize_keys(K, bits)
        monkeypatch.setattr(O, "_QUANT_ROWS", 1 << 30)
        b = O.quantize_keys(K, bits)
        monkeypatch.undo()
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
