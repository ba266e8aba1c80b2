"""Pins for the oracle's fixed-budget (top-k) selection, the rule Table 3 compares top-delta with."""
import math

import numpy as np
import pytest

from oracle import ffd_oracle as O

ALPHA = 1 / math.sqrt(128)


def bf16(x):
    return O.bf16_to_f64(O.f64_to_bf16_bits(x))


def _brute_topk(row, k):
    """k times: take the largest remaining score, the lowest block index among equals."""
    left = list(range(len(row)))
    kept = []
    for _ in range(min(k, len(row))):
        best = left[0]
        for j in left[1:]:
            if row[j] > row[best]:
                best = j
        kept.append(best)
        left.remove(best)
    return sorted(kept)


@pytest.mark.parametrize("seed", range(5))
def test_topk_brute_force_with_ties(seed):
    rng = np.random.default_rng(seed)
    sigma = np.round(rng.standard_normal((3, 23)), 1)     # rounding makes ties common
    sigma[1, 5:12] = 0.3
    for k in (1, 2, 5, 11, 23, 40):
        keep = O.select_topk(sigma, k)
        for h in range(3):
            assert np.nonzero(keep[h])[0].tolist() == _brute_topk(sigma[h], k), (k, h)


def test_topk_invariants():
    rng = np.random.default_rng(9)
    sigma = rng.standard_normal((4, 50))
    prev = np.zeros_like(sigma, dtype=bool)
    for k in range(0, 55, 3):
        keep = O.select_topk(sigma, k)
        assert np.all(keep.sum(1) == min(k, 50))
        assert np.all(keep >= prev)                       # nested in k
        for h in range(4):
            if 0 < keep[h].sum() < 50:
                assert sigma[h][keep[h]].min() >= sigma[h][~keep[h]].max()
        prev = keep
    equal = np.zeros((2, 10))
    assert np.nonzero(O.select_topk(equal, 4)[0])[0].tolist() == [0, 1, 2, 3]


def test_topk_decode_uses_the_block_scores_and_full_budget_is_dense():
    rng = np.random.default_rng(11)
    L = 700
    q, K, V = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((L, 128))), \
        bf16(rng.standard_normal((L, 128)))
    r = O.decode_group(q, K, V, L, delta=5.0, n_sink=64, n_local=256, block=64, alpha=ALPHA, topk=3)
    np.testing.assert_array_equal(r["keep"], O.select_topk(r["sigma"], 3))
    assert np.all(r["keep"].sum(1) == 3)
    nblk = -(-L // 64)
    full = O.decode_group(q, K, V, L, delta=5.0, n_sink=64, n_local=256, block=64, alpha=ALPHA, topk=nblk)
    dense = O.decode_group(q, K, V, L, delta=np.inf, n_sink=64, n_local=256, block=64, alpha=ALPHA)
    assert full["keep"].all()
    np.testing.assert_array_equal(full["out"], dense["out"])
    np.testing.assert_array_equal(full["lse"], dense["lse"])
