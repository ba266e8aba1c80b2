"""Pins for the oracle's scan, pseudo-max and top-delta selection (Alg. 1; Sec. 3.2 Eq. 1-3; Sec. 5.2)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import ffd_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16(x):
    return O.bf16_to_f64(O.f64_to_bf16_bits(x))


def brute_force_pipeline(q, K, L, delta, n_sink, n_local, block):
    """Everything with explicit Python loops from the definitions, for tiny d and L."""
    G, d = len(q), len(q[0])
    alpha = 1.0 / math.sqrt(d)
    levels = (-1.5, -0.5, 0.5, 1.5)
    khat = []
    for t in range(L):
        M = max(abs(K[t][i]) for i in range(d))
        row = []
        for i in range(d):
            if M == 0:
                row.append(0.0)
                continue
            x = K[t][i] / (M / 1.5)
            best = None
            for lv in levels:                               # nearest level, upper wins ties
                if best is None or abs(x - lv) <= abs(x - best) + 1e-12:
                    best = lv
            row.append(best * M / 1.5)
        khat.append(row)
    s = [[alpha * sum(q[h][i] * khat[t][i] for i in range(d)) for t in range(L)] for h in range(G)]
    window = sorted(set(range(min(n_sink, L))) | set(range(max(0, L - n_local), L)))
    m_t = [max(s[h][t] for t in window) for h in range(G)]
    nblk = (L + block - 1) // block
    keep = [[max(s[h][t] for t in range(j * block, min(j * block + block, L))) >= m_t[h] - delta
             for j in range(nblk)] for h in range(G)]
    return s, m_t, keep


@pytest.mark.parametrize("d,L,block,n_sink,n_local,delta,seed", [
    (4, 17, 4, 4, 4, 0.3, 0), (8, 32, 4, 2, 6, 0.5, 1), (8, 13, 4, 0, 3, 1.0, 2),
    (4, 32, 4, 8, 0, 0.0, 3), (8, 5, 4, 64, 256, 0.2, 4), (8, 31, 4, 3, 5, 2.0, 5),
])
def test_scan_select_match_brute_force(d, L, block, n_sink, n_local, delta, seed):
    rng = np.random.default_rng(seed)
    q = bf16(rng.standard_normal((3, d)))
    K = bf16(rng.standard_normal((L, d)))
    r = O.decode_group(q, K, bf16(rng.standard_normal((L, d))), L, delta=delta, n_sink=n_sink,
                       n_local=n_local, block=block, alpha=1 / math.sqrt(d))
    s, m_t, keep = brute_force_pipeline(q.tolist(), K.tolist(), L, delta, n_sink, n_local, block)
    np.testing.assert_allclose(r["s_hat"], np.array(s), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["m_tilde"], np.array(m_t), rtol=0, atol=1e-12)
    assert r["keep"].tolist() == keep


def test_scan_error_within_deterministic_bound():
    """|s_hat - s| <= alpha * (s_q/2) * |q|_1 since each |k_i - k^quant_i| <= s/2 (App. B setup)."""
    rng = np.random.default_rng(7)
    q = bf16(rng.standard_normal((4, 128)))
    K = bf16(rng.standard_normal((2000, 128)) * 1.7)
    codes, M, _ = O.quantize_keys(K)
    alpha = 1 / math.sqrt(128)
    err = np.abs(O.scan_scores(q, codes, M, alpha) - alpha * q @ K.T)
    bound = alpha * (M[None, :] / 1.5 / 2) * np.abs(q).sum(axis=1)[:, None]
    assert np.all(err <= bound * (1 + 1e-12))
    assert err.max() > 0.05 * bound.max()          # the bound is not vacuous for the check


def test_concentration_of_scanning_error_app_b():
    """Thm B.1: P(|e| >= lam) <= 2 exp(-lam^2 / (2 sigma^2 a^2)) with |q| = a sqrt(d).

    The per-channel noise is bounded by s/2, hence sub-Gaussian with sigma = s/2 (Hoeffding).
    """
    rng = np.random.default_rng(11)
    d = 128
    q = bf16(rng.standard_normal((1, d)))[0]
    K = bf16(rng.standard_normal((20000, d)))
    codes, M, _ = O.quantize_keys(K)
    e = O.scan_scores(q[None], codes, M, 1 / math.sqrt(d))[0] - (q @ K.T) / math.sqrt(d)
    a = np.linalg.norm(q) / math.sqrt(d)
    sigma = np.median(M) / 1.5 / 2
    for lam in (0.5, 1.0, 1.5, 2.0):
        assert np.mean(np.abs(e) >= lam) <= 2 * math.exp(-lam ** 2 / (2 * sigma ** 2 * a ** 2))


def _case(seed, L=700, G=4, d=128, block=64):
    rng = np.random.default_rng(seed)
    q = bf16(rng.standard_normal((G, d)))
    K = bf16(rng.standard_normal((L, d)))
    V = bf16(rng.standard_normal((L, d)))
    # a few planted blocks so the selection is non-trivial
    u = q.mean(0) / np.linalg.norm(q.mean(0)) * math.sqrt(d)
    for j in rng.choice(np.arange(1, L // block - 2), 2, replace=False):
        K[j * block:(j + 1) * block] = bf16(2.5 * u + 0.5 * rng.standard_normal((block, d)))
    return q, K, V


@pytest.mark.parametrize("seed", range(4))
def test_selection_invariants(seed):
    q, K, V = _case(seed)
    L, block, alpha = K.shape[0], 64, 1 / math.sqrt(128)
    codes, M, _ = O.quantize_keys(K)
    s_hat = O.scan_scores(q, codes, M, alpha)
    m_t = O.pseudo_max(s_hat, L, 64, 256)
    sigma = O.block_scores(s_hat, L, block)
    # m~ <= the global max of the same scores (Sec. 5.2)
    assert np.all(m_t <= s_hat.max(axis=1))
    keeps = {dl: O.select_blocks(sigma, m_t, dl) for dl in (0.0, 1.0, 3.0, 5.0, 7.0, np.inf)}
    # monotone in delta
    for a, b in [(0.0, 1.0), (1.0, 3.0), (3.0, 5.0), (5.0, 7.0), (7.0, np.inf)]:
        assert np.all(keeps[a] <= keeps[b])
    assert keeps[np.inf].all()
    for dl in (0.0, 3.0, 5.0, 7.0):
        k = keeps[dl]
        # fail-safe: superset of the selection made with the true (global) max (Sec. 5.2)
        assert np.all(O.select_blocks(sigma, s_hat.max(axis=1), dl) <= k)
        # the block holding the pseudo-max's argmax always passes, so no head is empty
        win = O.pseudo_max_tokens(L, 64, 256)
        for h in range(q.shape[0]):
            t = win[np.argmax(s_hat[h, win])]
            assert k[h, t // block]
        # every token of a dropped block is below e^-delta of the pseudo-max (Eq. 2)
        tok_keep = np.stack([O.token_mask_from_blocks(k[h], L, block) for h in range(q.shape[0])])
        dropped = ~tok_keep
        assert np.all(np.exp(s_hat - m_t[:, None])[dropped] < math.exp(-dl))


def test_top_delta_mass_matches_paper_numbers():
    g = json.load(open(os.path.join(GOLDEN, "top_delta_mass.json")))
    assert round(100 * math.exp(-5), 2) == g["delta_5_percent"]
    # the paper quotes 1/e^-delta truncated to an integer: e^5 = 148.4, e^7 = 1096.6
    assert math.floor(1 / math.exp(-5)) == g["delta_5_one_over"]
    assert math.floor(1 / math.exp(-7)) == g["delta_7_one_over"]


def test_pseudo_max_windows():
    assert O.pseudo_max_tokens(1000, 64, 256).tolist() == list(range(64)) + list(range(744, 1000))
    assert O.pseudo_max_tokens(100, 64, 256).tolist() == list(range(100))
    assert O.pseudo_max_tokens(10, 0, 3).tolist() == [7, 8, 9]
    assert O.pseudo_max_tokens(0, 64, 256).size == 0


# ---- near_threshold: the band around Eq. 1's threshold m~ - delta that parity reports apart ----

def test_near_threshold_hand_values():
    """Threshold m~ - delta = 10 - 5 = 5 with a band of 2^-10 (exact in binary): strictly inside
    the band on both sides, not at or beyond its edges, never on the wrong side of m~ + delta."""
    band = 2.0 ** -10
    m_t = np.array([10.0])
    sig = np.array([[5.0, 5.0 + band / 2, 5.0 - band / 2, 5.0 + band, 5.0 - band,
                     5.0 + 2 * band, 15.0, 10.0, 0.0, -np.inf]])
    got = O.near_threshold(sig, m_t, 5.0, band)
    assert got.tolist() == [[True, True, True, False, False, False, False, False, False, False]]


def test_near_threshold_default_band_is_one_thousandth():
    m_t = np.array([3.0, -1.5])
    sig = np.array([[1.0, 1.0009, 0.9991, 1.0011, 0.9989, 3.0],
                    [-3.5, -3.4995, -3.5005, -3.498, -3.502, -1.5]])
    got = O.near_threshold(sig, m_t, 2.0)
    assert got.tolist() == [[True, True, True, False, False, False],
                            [True, True, True, False, False, False]]


def test_near_threshold_infinite_cases():
    sig = np.array([[-np.inf, 0.0, 1e30, -1e30]])
    # an empty window: m~ = -inf, so the threshold is -inf and no finite score is near it
    assert not O.near_threshold(sig, np.array([-np.inf]), 5.0).any()
    # delta = inf keeps everything: no score is near the threshold
    assert not O.near_threshold(sig, np.array([2.0]), np.inf).any()
    # an empty block (sigma = -inf) is never near, even at an infinite threshold
    assert not O.near_threshold(np.array([[-np.inf]]), np.array([-np.inf]), 0.0).any()
    # delta = 0: the band sits around m~ itself
    assert O.near_threshold(np.array([[2.0, 2.0005, 1.0]]), np.array([2.0]), 0.0).tolist() == [[True, True, False]]


def test_near_threshold_broadcasts_heads_over_blocks():
    """[B, H, nblk] scores against [B, H] pseudo-maxima: each head uses its own threshold."""
    m_t = np.array([[1.0, 4.0], [0.0, -2.0]])
    sig = np.stack([m_t - 3.0 + 2e-4, m_t - 3.0 + 0.5, m_t], axis=-1)
    assert O.near_threshold(sig, m_t, 3.0).tolist() == [[[True, False, False]] * 2] * 2
    # swapping the heads' thresholds moves every band
    assert not O.near_threshold(sig[:, ::-1, :1], m_t, 3.0).any()


def test_near_threshold_agrees_with_a_loop_over_the_definition():
    rng = np.random.default_rng(3)
    m_t = rng.normal(size=4)
    delta = 1.5
    sig = (m_t[:, None] - delta) + rng.choice([-1, 1], size=(4, 200)) * rng.uniform(0, 3e-3, size=(4, 200))
    sig[0, :5] = -np.inf
    got = O.near_threshold(sig, m_t, delta)
    for h in range(4):
        for j in range(200):
            s = sig[h, j]
            want = bool(np.isfinite(s) and abs(s - (m_t[h] - delta)) < 1e-3)
            assert got[h, j] == want
    assert 100 < got.sum() < 700
