"""Pins for the oracle's fidelity diagnostics (Sec. 5.1 recall and LSE error, Sec. 5.2 pseudo-max
gap) and the pseudo-max variants (Eq. 3's window scores: thumbnail, refined or exact)."""
import math

import numpy as np
import pytest

from oracle import ffd_oracle as O

ALPHA = 1 / math.sqrt(128)


def bf16(x):
    return O.bf16_to_f64(O.f64_to_bf16_bits(x))


def _case(seed, L=900, heavy=True):
    rng = np.random.default_rng(seed)
    q = bf16(rng.standard_normal((4, 128)))
    K = rng.standard_normal((L, 128))
    if heavy:                                   # a few keys aligned with the queries, mid-sequence
        u = q.mean(0) / np.linalg.norm(q.mean(0)) * math.sqrt(128)
        for t in rng.choice(np.arange(100, L - 300), 6, replace=False):
            K[t] = 2.5 * u + 0.5 * rng.standard_normal(128)
    return q, bf16(K), bf16(rng.standard_normal((L, 128)))


def test_diagnostics_brute_force_tiny():
    a = np.array([[1.0, 2.0, 2.0], [0.0, 0.0, 0.0], [3.0, 0.0, 4.0]])
    b = np.array([[2.0, 4.0, 4.0], [0.0, 0.0, 0.0], [0.0, 5.0, 0.0]])
    cos = O.recall_cosine(a, b)
    assert cos[0] == pytest.approx(1.0, abs=1e-15) and cos[1] == 1.0 and cos[2] == 0.0
    # explicit loop for a random pair
    rng = np.random.default_rng(1)
    x, y = rng.standard_normal(16), rng.standard_normal(16)
    dot = sum(x[i] * y[i] for i in range(16))
    nx, ny = math.sqrt(sum(v * v for v in x)), math.sqrt(sum(v * v for v in y))
    assert O.recall_cosine(x, y) == pytest.approx(dot / (nx * ny), abs=1e-14)
    assert O.lse_abs_error([1.5, -np.inf, 2.0], [1.0, -np.inf, 3.0]).tolist() == [0.5, 0.0, 1.0]
    assert O.pseudo_max_gap([2.0, -np.inf], [1.25, -np.inf]).tolist() == [0.75, 0.0]


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_exact_pseudo_max_never_exceeds_the_true_max(seed):
    """Sec. 5.2: m~ <= m when both are taken over exact scores, with equality iff the argmax lies in
    a window; the gap is then the distance to the best window token."""
    q, K, V = _case(seed)
    L = K.shape[0]
    m = O.exact_max(q, K, L, ALPHA)
    s = ALPHA * (q @ K.T)
    for n_sink, n_local in ((64, 256), (1, 1), (0, 16)):
        r = O.decode_group(q, K, V, L, delta=5.0, n_sink=n_sink, n_local=n_local, block=64,
                           alpha=ALPHA, pm_source="exact")
        win = O.pseudo_max_tokens(L, n_sink, n_local)
        assert np.all(r["m_tilde"] <= m)
        np.testing.assert_array_equal(r["m_tilde"], s[:, win].max(1))
        gap = O.pseudo_max_gap(m, r["m_tilde"])
        in_win = np.isin(s.argmax(1), win)
        assert np.all(gap[in_win] == 0) and np.all(gap[~in_win] > 0)


@pytest.mark.parametrize("seed", [4, 5])
def test_variants_differ_by_at_most_the_reconstruction_error(seed):
    """Over the window tokens: |s_hat - s| <= alpha |q|_1 s_t / 2 (thumbnail, App. B) and
    |z - s| <= alpha |q|_1 M_t / 762 (2+8 reconstruction), so the pseudo-maxes differ by at most the
    largest such bound among the window tokens."""
    q, K, V = _case(seed)
    L = K.shape[0]
    win = O.pseudo_max_tokens(L, 64, 256)
    _, M, _ = O.quantize_keys(K)
    q1 = np.abs(q).sum(1)
    pm = {src: O.decode_group(q, K, V, L, delta=5.0, n_sink=64, n_local=256, block=64, alpha=ALPHA,
                              pm_source=src)["m_tilde"] for src in O.PM_SOURCES}
    b_thumb = ALPHA * q1 * (M[win].max() / 1.5) / 2
    b_ref = ALPHA * q1 * M[win].max() / 762
    assert np.all(np.abs(pm["thumbnail"] - pm["exact"]) <= b_thumb * (1 + 1e-9))
    assert np.all(np.abs(pm["refined"] - pm["exact"]) <= b_ref * (1 + 1e-9))
    assert np.any(pm["thumbnail"] != pm["refined"])


def test_lse_error_shrinks_with_delta_and_is_bounded_by_the_dropped_tokens():
    """With the refined logits z: lse over a superset of tokens is larger, so lse_ffd grows with delta
    towards lse over every token (delta = inf); every dropped token has z below m~ - delta plus its
    thumbnail error, which bounds the lse deficit."""
    q, K, V = _case(7)
    L = K.shape[0]
    codes, M, resid = O.quantize_keys(K)
    z = O.refined_logits(q, codes, M, resid, ALPHA)
    full = np.log(np.exp(z - z.max(1, keepdims=True)).sum(1)) + z.max(1)
    err = ALPHA * np.abs(q).sum(1)[:, None] * (M[None, :] / 1.5) / 2 + ALPHA * np.abs(q).sum(1)[:, None] * M[None, :] / 762
    prev = None
    for delta in (0.0, 1.0, 3.0, 5.0, 7.0, np.inf):
        r = O.decode_group(q, K, V, L, delta=delta, n_sink=64, n_local=256, block=64, alpha=ALPHA)
        deficit = full - r["lse"]
        assert np.all(deficit >= -1e-12)
        if prev is not None:
            assert np.all(r["lse"] >= prev - 1e-12)
        prev = r["lse"]
        for h in range(4):
            drop = ~O.token_mask_from_blocks(r["keep"][h], L, 64)
            if not drop.any():
                assert abs(deficit[h]) < 1e-12
                continue
            bound_z = r["m_tilde"][h] - delta + err[h, drop]      # each dropped logit is below this
            assert np.all(z[h, drop] <= bound_z + 1e-9)
            extra = np.exp(bound_z - r["lse"][h]).sum()
            assert deficit[h] <= math.log1p(extra) + 1e-12


def test_recall_and_lse_error_against_dense_reach_the_reconstruction_limit():
    """At delta = inf the FFD output is dense attention on the 2+8 reconstruction: its recall
    against exact dense attention is that of the reconstruction (close to 1) and its LSE error is at
    most the largest score error alpha |q|_1 M / 762."""
    q, K, V = _case(8)
    L = K.shape[0]
    dense_o, dense_lse = O.dense_attention(q, K, V, L, ALPHA)
    r = O.decode_group(q, K, V, L, delta=np.inf, n_sink=64, n_local=256, block=64, alpha=ALPHA)
    _, M, _ = O.quantize_keys(K)
    assert np.all(O.recall_cosine(r["out"], dense_o) > 0.9999)
    assert np.all(O.lse_abs_error(r["lse"], dense_lse) <= ALPHA * np.abs(q).sum(1) * M.max() / 762)
    # and recall at delta = 5 is no better than at delta = inf for the same heads' lse
    r5 = O.decode_group(q, K, V, L, delta=5.0, n_sink=64, n_local=256, block=64, alpha=ALPHA)
    assert np.all(r5["lse"] <= r["lse"] + 1e-12)


def test_unknown_source_rejected():
    q, K, V = _case(9, L=100, heavy=False)
    with pytest.raises(ValueError):
        O.decode_group(q, K, V, 100, delta=5.0, n_sink=4, n_local=4, block=64, alpha=ALPHA,
                       pm_source="bogus")
