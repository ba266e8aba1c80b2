"""Pins for the oracle's packing of the quantized copy into this implementation's storage format."""
import numpy as np

from oracle import ffd_oracle as O


def test_pack_codes_single_token_hand_checked():
    """Token 81 is block 1, t4 = 1, n = 1; dim 16 + 5 is cc = 0, g = 1, e = 5 -> lane 1 + 16 = 17,
    word 2*1 + 0 = 2 (stored at [block, 2 // 4, lane, 2 % 4]), bit 8*(5%4) + 2*(5//4) = 10."""
    codes = np.zeros((128, 128), dtype=np.int64)
    codes[81, 16 + 5] = 3
    p = O.pack_codes(codes)
    assert p.shape == (2, 2, 64, 4)
    nz = np.argwhere(p)
    assert nz.tolist() == [[1, 0, 17, 2]]
    assert int(p[1, 0, 17, 2]) == 3 << 10


def test_pack_codes_fast_equals_loop_and_roundtrips():
    rng = np.random.default_rng(0)
    codes = rng.integers(0, 4, size=(128, 128))
    p = O.pack_codes(codes)
    assert np.array_equal(O.pack_codes_fast(codes), p)
    assert np.array_equal(O.unpack_codes(p, 128), codes)


def test_pack_absmax_and_resid_index_maps():
    L = 128
    M = np.arange(L, dtype=np.uint16)
    pm = O.pack_absmax(M)
    for j in range(L // 64):
        for n in range(16):
            for t4 in range(4):
                assert pm[j, n, t4] == 64 * j + 16 * t4 + n
    r = (np.arange(L * 128) % 251 - 125).reshape(L, 128)
    pr = O.pack_resid(r)
    for T in range(L // 16):
        for cc in range(2):
            for g in range(4):
                for n in range(16):
                    for e in range(16):
                        assert pr[T, cc, n + 16 * g, e] == r[16 * T + n, 64 * cc + 16 * g + e]


def test_quantize_cache_range_only_defines_live_tokens():
    from ffd_inputs import small_case
    c = small_case(seed=3, B=1, Hq=4, Hkv=1, seq_lens=(128,))
    codes, absmax, resid = O.quantize_cache(c.k, 32, 96)
    full = O.quantize_cache(c.k)
    cu = O.unpack_codes(codes[0, 0], 128)
    cf = O.unpack_codes(full[0][0, 0], 128)
    assert np.array_equal(cu[32:96], cf[32:96])
    assert not cu[:32].any() and not cu[96:].any()
