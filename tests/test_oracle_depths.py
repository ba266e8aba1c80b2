"""Pins for the oracle's wider thumbnails, the 4+8 and 8+8 depths of App. C (App. A's mid-rise
formulation with 2^b levels; the 8-bit residual of Sec. 3.1 on the step s/254)."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import ffd_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
WIDE = (4, 8)


def all_finite_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = O.bf16_to_f64(bits)
    return x[np.isfinite(x)]


def bf16(x):
    return O.bf16_to_f64(O.f64_to_bf16_bits(x))


def test_worked_examples_match_hand_computation():
    g = json.load(open(os.path.join(GOLDEN, "quantizer_depths_worked_example.json")))
    for case in g["cases"]:
        b = case["bits"]
        x = np.array(case["x"], dtype=np.float64)
        codes, M, resid = O.quantize_keys(x, b)
        assert M == case["M"]
        assert codes.tolist() == case["codes"], b
        assert resid.tolist() == case["resid"], b
        assert O.thumbnail(codes, M, b).tolist() == case["thumbnail"], b
        N = O.full_levels(b)
        full = O.thumbnail(codes, M, b) + O.residual_part(resid, M, b)
        np.testing.assert_allclose(full, case["M"] * np.array(case["n"]) / N, rtol=0, atol=1e-12)
        if "stored_bytes" in case:
            vec = np.zeros((64, 128))
            vec[0, :8] = x
            vec[0, 8] = case["M"]
            c, _, _ = O.quantize_keys(vec, b)
            p = O.pack_codes(c, b)
            # token 0, dims 0..7: lane 0, words 0 and 1 (stored at [0, 0, 0, w]), byte i of word k is dim 4k + i
            got = [int(np.int8(np.uint8((int(p[0, 0, 0, e // 4]) >> (8 * (e % 4))) & 0xFF))) for e in range(8)]
            assert got == case["stored_bytes"]


def test_constants():
    assert [O.top_level(b) for b in (2, 4, 8)] == [1.5, 7.5, 127.5]
    assert [O.full_levels(b) for b in (2, 4, 8)] == [381, 1905, 32385]
    assert O.codebook(2).tolist() == O.CODEBOOK.tolist()
    assert O.codebook(8)[0] == -127.5 and O.codebook(8)[-1] == 127.5


def _exact_nearest_code(x: float, M: float, bits: int) -> int:
    """Brute force over the 2^b levels with exact rationals; a tie goes to the upper level.
    |x/s - (c - Lv)| is proportional to |(2^b - 1) x - (2c - 2^b + 1) M|."""
    xf, Mf = Fraction(x), Fraction(M)
    best, best_d = None, None
    for c in range(2 ** bits):
        d = abs((2 ** bits - 1) * xf - (2 * c - 2 ** bits + 1) * Mf)
        if best_d is None or d <= best_d:
            best, best_d = c, d
    return best


@pytest.mark.parametrize("bits", WIDE)
@pytest.mark.parametrize("M", [1.0, 7.5, 2.5, 127.5, 0.0078125, 3.0e38, 1.0e-38])
def test_codes_exhaustive_over_bf16(bits, M):
    Mb = O.bf16_to_f64(O.f64_to_bf16_bits(np.array([M])))[0]
    x = all_finite_bf16()
    x = x[np.abs(x) <= Mb]
    vec = np.stack([x, np.full_like(x, Mb)], axis=1)
    codes, Mv, _ = O.quantize_keys(vec, bits)
    assert np.all(Mv == Mb)
    s = Mb / O.top_level(bits)
    # every value on a bin edge (x/s an integer) and a stride of the rest, by brute force
    xs = x / s
    edge = (xs == np.round(xs)) | np.isclose(xs, np.round(xs), rtol=0, atol=1e-3)
    step = 7 if bits == 4 else 41                       # the 256-level brute force is slower
    idx = np.unique(np.concatenate([np.nonzero(edge)[0][::step], np.arange(0, x.size, 30 * step)]))
    for i in idx:
        assert codes[i, 0] == _exact_nearest_code(float(x[i]), float(Mb), bits), (x[i], Mb, bits)
    xhat = O.thumbnail(codes, Mv, bits)[:, 0]
    assert np.all(np.abs(x - xhat) <= s / 2 + 4e-16 * Mb)     # rounding of (c - Lv) * s is ~eps M
    assert codes.min() >= 0 and codes.max() <= 2 ** bits - 1


def _exact_nearest_grid(x: float, M: float, N: int) -> int:
    """Nearest j of the grid j*M/N (ties to even j), exact rationals."""
    t = Fraction(x) * N / Fraction(M)
    fl = t.numerator // t.denominator
    frac = t - fl
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and fl % 2 == 1):
        return fl + 1
    return fl


@pytest.mark.parametrize("bits", WIDE)
@pytest.mark.parametrize("seed", [1, 2])
def test_residual_brute_force_and_bounds(bits, seed):
    rng = np.random.default_rng(seed + 10 * bits)
    K = bf16(rng.standard_normal((64, 128)) * rng.uniform(0.01, 50))
    codes, M, resid = O.quantize_keys(K, bits)
    N = O.full_levels(bits)
    assert resid.min() >= -127 and resid.max() <= 127
    n = resid + 254 * codes - N
    for r in range(0, 64, 7):
        for c in range(128):
            assert n[r, c] == _exact_nearest_grid(float(K[r, c]), float(M[r]), N), (r, c)
    full = O.thumbnail(codes, M, bits) + O.residual_part(resid, M, bits)
    assert np.all(np.abs(full - M[:, None] * n / N) <= 1e-13 * M[:, None])
    assert np.all(np.abs(K - full) <= M[:, None] / (2 * N) + 1e-14 * M[:, None])   # ties reach it


@pytest.mark.parametrize("bits", WIDE)
def test_residual_exhaustive_ties_to_even(bits):
    """All bf16 values against M = Lv (s = 1): the residual grid index is rint(254 x), ties to even."""
    Lv = O.top_level(bits)
    x = all_finite_bf16()
    x = x[np.abs(x) <= Lv]
    codes, M, resid = O.quantize_keys(np.stack([x, np.full_like(x, Lv)], axis=1), bits)
    n = resid[:, 0] + 254 * codes[:, 0] - O.full_levels(bits)
    t = x * 254.0
    fl = np.floor(t)
    fr = t - fl
    expect = np.where(fr > 0.5, fl + 1, np.where(fr < 0.5, fl, np.where(fl % 2 == 0, fl, fl + 1)))
    assert np.array_equal(n, expect.astype(np.int64))
    assert (fr == 0.5).sum() > 0


@pytest.mark.parametrize("bits", WIDE)
def test_extreme_element_and_zero_vector(bits):
    rng = np.random.default_rng(bits)
    K = bf16(rng.standard_normal((200, 128)))
    codes, M, resid = O.quantize_keys(K, bits)
    i = np.argmax(np.abs(K), axis=1)
    rows = np.arange(K.shape[0])
    lvl = O.codebook(bits)[codes[rows, i]]
    assert np.all(np.abs(lvl) == O.top_level(bits))
    assert np.all(np.sign(lvl) == np.sign(K[rows, i]))
    assert np.all(resid[rows, i] == 0)
    codes, M, resid = O.quantize_keys(np.zeros((3, 128)), bits)
    assert np.all(M == 0) and np.all(codes == 2 ** (bits - 1)) and np.all(resid == 0)
    assert np.all(O.thumbnail(codes, M, bits) == 0)


def test_two_bit_depth_is_the_app_a_formulation():
    """bits = 2 of the general rule equals App. A's explicit comparisons, on every bf16 value."""
    x = all_finite_bf16()
    x = x[np.abs(x) <= 1.5]
    vec = np.stack([x, np.full_like(x, 1.5)], axis=1)
    codes, _, _ = O.quantize_keys(vec, 2)
    explicit = np.where(3 * x >= 3.0, 3, np.where(x >= 0, 2, np.where(3 * x >= -3.0, 1, 0)))
    assert np.array_equal(codes[:, 0], explicit)


@pytest.mark.parametrize("bits", (2, 4, 8))
def test_scan_score_error_bound_shrinks_with_depth(bits):
    """|s_hat - alpha q.k| <= alpha |q|_1 s / 2 with s = M / Lv (thumbnail error bound)."""
    rng = np.random.default_rng(21)
    q, K = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((300, 128)) * 2)
    codes, M, _ = O.quantize_keys(K, bits)
    alpha = 1 / math.sqrt(128)
    err = np.abs(O.scan_scores(q, codes, M, alpha, bits) - alpha * q @ K.T)
    bound = alpha * np.abs(q).sum(1)[:, None] * (M[None, :] / O.top_level(bits)) / 2
    assert np.all(err <= bound * (1 + 1e-9))


@pytest.mark.parametrize("bits", WIDE)
def test_infinite_delta_equals_dense_attention_on_reconstructed_keys(bits):
    rng = np.random.default_rng(3 + bits)
    L = 200
    q, K, V = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((L, 128))), \
        bf16(rng.standard_normal((L, 128)))
    alpha = 1 / math.sqrt(128)
    r = O.decode_group(q, K, V, L, delta=np.inf, n_sink=64, n_local=256, block=64, alpha=alpha,
                       bits=bits)
    assert r["keep"].all()
    codes, M, resid = O.quantize_keys(K, bits)
    N = O.full_levels(bits)
    K_full = M[:, None] * (resid + 254 * codes - N) / N
    qt, Kt, Vt = (torch.tensor(a, dtype=torch.float64) for a in (q, K_full, V))
    o_t = torch.softmax(alpha * qt @ Kt.T, dim=-1) @ Vt
    np.testing.assert_allclose(r["out"], o_t.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("bits", WIDE)
def test_pack_codes_single_token_hand_checked(bits):
    """Token 81 = block 1, t4 = 1, n = 1; dim 16 + 5 = cc 0, g 1, e 5 (k 1, i 1) -> lane 17.
    4-bit: word (2*1 + 0)*2 + 1//2 = 4 (stored at [1, 1, 17, 0]), bit 8 + 4*(1%2) = 12. 8-bit: word
    (2*1 + 0)*4 + 1 = 9 (stored at [1, 2, 17, 1]), bit 8, holding the byte c - 128."""
    codes = np.zeros((128, 128), dtype=np.int64)
    c = 13 if bits == 4 else 200
    codes[81, 16 + 5] = c
    p = O.pack_codes(codes, bits)
    if bits == 4:
        nz = np.argwhere(p)
        assert nz.tolist() == [[1, 1, 17, 0]] and int(p[1, 1, 17, 0]) == 13 << 12
    else:
        # every other code is 0 -> byte 0x80; the one entry holds 200 - 128 = 72
        assert (int(p[1, 2, 17, 1]) >> 8) & 0xFF == 72
        assert int(p[1, 2, 17, 1]) & 0xFFFF00FF == 0x80800080
        assert np.count_nonzero(p != 0x80808080) == 1


@pytest.mark.parametrize("bits", (2, 4, 8))
def test_pack_codes_fast_equals_loop_and_roundtrips(bits):
    rng = np.random.default_rng(bits)
    codes = rng.integers(0, 2 ** bits, size=(128, 128))
    p = O.pack_codes(codes, bits)
    assert np.array_equal(O.pack_codes_fast(codes, bits), p)
    assert np.array_equal(O.unpack_codes(p, 128, bits), codes)


@pytest.mark.parametrize("bits", WIDE)
def test_quantize_cache_range_only_defines_live_tokens(bits):
    from ffd_inputs import small_case
    c = small_case(seed=3, B=1, Hq=4, Hkv=1, seq_lens=(128,))
    codes, absmax, resid = O.quantize_cache(c.k, 32, 96, bits)
    full = O.quantize_cache(c.k, bits=bits)
    assert codes.shape[-3:] == (bits, 64, 4)
    cu = O.unpack_codes(codes[0, 0], 128, bits)
    cf = O.unpack_codes(full[0][0, 0], 128, bits)
    assert np.array_equal(cu[32:96], cf[32:96])
    # undefined tokens are zero words in the packed form
    w = O.lane_words(codes[0, 0], bits).reshape(2, 4, 16, 4, 2, -1)   # j, g, n, t4, cc, word
    live = np.zeros(128, bool)
    live[32:96] = True
    for j in range(2):
        for n in range(16):
            for t4 in range(4):
                if not live[64 * j + 16 * t4 + n]:
                    assert not w[j, :, n, t4].any()
