"""Pins for the oracle's refinement, sparse attention, dense attention and split merge.

Library routines (torch on the CPU, float64) stand in for the textbook definitions; explicit
loops check the tiny cases.
"""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import ffd_oracle as O


def bf16(x):
    return O.bf16_to_f64(O.f64_to_bf16_bits(x))


def torch_attention(q, K, V, alpha):
    qt, Kt, Vt = (torch.tensor(a, dtype=torch.float64) for a in (q, K, V))
    out = torch.nn.functional.scaled_dot_product_attention(
        qt[None, :, None, :], Kt[None, None].expand(1, qt.shape[0], -1, -1),
        Vt[None, None].expand(1, qt.shape[0], -1, -1), scale=alpha)[0, :, 0]
    lse = torch.logsumexp(alpha * qt @ Kt.T, dim=-1)
    return out.numpy(), lse.numpy()


@pytest.mark.parametrize("L", [1, 63, 64, 65, 700])
def test_dense_matches_library_attention(L):
    rng = np.random.default_rng(L)
    q, K, V = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((L, 128))), \
        bf16(rng.standard_normal((L, 128)))
    o, lse = O.dense_attention(q, K, V, L, 1 / math.sqrt(128))
    o_t, lse_t = torch_attention(q, K, V, 1 / math.sqrt(128))
    np.testing.assert_allclose(o, o_t, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_t, rtol=0, atol=1e-12)


def test_infinite_delta_equals_dense_attention_on_reconstructed_keys():
    """With delta = +inf every block is kept: FFD is dense attention on k^quant + k^res."""
    rng = np.random.default_rng(3)
    L = 333
    q, K, V = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((L, 128))), \
        bf16(rng.standard_normal((L, 128)))
    r = O.decode_group(q, K, V, L, delta=np.inf, n_sink=64, n_local=256, block=64,
                       alpha=1 / math.sqrt(128))
    assert r["keep"].all()
    codes, M, resid = O.quantize_keys(K)
    n = resid + 254 * codes - 381
    K_full = M[:, None] * n / 381.0                      # closed form, not the oracle's path
    o_t, lse_t = torch_attention(q, K_full, V, 1 / math.sqrt(128))
    np.testing.assert_allclose(r["out"], o_t, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["lse"], lse_t, rtol=0, atol=1e-12)


def test_refined_logits_close_to_exact_scores():
    """|z - s| <= alpha (M/762) |q|_1 from the 2+8 reconstruction error bound."""
    rng = np.random.default_rng(5)
    q, K = bf16(rng.standard_normal((4, 128))), bf16(rng.standard_normal((500, 128)) * 3)
    codes, M, resid = O.quantize_keys(K)
    alpha = 1 / math.sqrt(128)
    z = O.refined_logits(q, codes, M, resid, alpha)
    bound = alpha * (M[None, :] / 762) * np.abs(q).sum(1)[:, None]
    assert np.all(np.abs(z - alpha * q @ K.T) <= bound * (1 + 1e-9))


def test_softmax_weights_sum_to_one_and_brute_force():
    rng = np.random.default_rng(9)
    z = rng.standard_normal(37) * 4
    V = rng.standard_normal((37, 8))
    o, lse = O.softmax_attend(z, V)
    w = [math.exp(zi) for zi in z]
    tot = sum(w)
    assert abs(sum(wi / tot for wi in w) - 1.0) < 1e-15
    brute = [sum(w[t] / tot * V[t][i] for t in range(37)) for i in range(8)]
    np.testing.assert_allclose(o, brute, rtol=0, atol=1e-13)
    assert abs(lse - math.log(tot)) < 1e-13
    o0, lse0 = O.softmax_attend(np.zeros(0), V[:0])
    assert np.all(o0 == 0) and lse0 == -np.inf


def test_sparse_attention_brute_force_tiny():
    """Explicit loops: softmax over kept-block tokens of the refined logits, times V."""
    rng = np.random.default_rng(13)
    d, L, block = 8, 22, 4
    q, K, V = bf16(rng.standard_normal((2, d))), bf16(rng.standard_normal((L, d))), \
        bf16(rng.standard_normal((L, d)))
    alpha = 1 / math.sqrt(d)
    r = O.decode_group(q, K, V, L, delta=0.7, n_sink=2, n_local=3, block=block, alpha=alpha)
    codes, M, resid = O.quantize_keys(K)
    for h in range(2):
        toks = [t for t in range(L) if r["keep"][h][t // block]]
        z = {}
        for t in toks:
            z[t] = alpha * sum(q[h][i] * (M[t] * (resid[t][i] + 254 * codes[t][i] - 381) / 381)
                               for i in range(d))
        mx = max(z.values())
        w = {t: math.exp(z[t] - mx) for t in toks}
        tot = sum(w.values())
        o = [sum(w[t] * V[t][i] for t in toks) / tot for i in range(d)]
        np.testing.assert_allclose(r["out"][h], o, rtol=0, atol=1e-12)
        assert abs(r["lse"][h] - (mx + math.log(tot))) < 1e-12


@pytest.mark.parametrize("nblk", [1, 2, 5, 8])
def test_lse_merge_of_every_contiguous_partition_equals_unsplit(nblk):
    rng = np.random.default_rng(nblk)
    block = 3
    z = rng.standard_normal(nblk * block) * 5
    V = rng.standard_normal((nblk * block, 6))
    o_ref, lse_ref = O.softmax_attend(z, V)
    for cuts in itertools.chain.from_iterable(
            itertools.combinations(range(1, nblk), k) for k in range(nblk)):
        edges = [0, *cuts, nblk]
        states = [O.partial_state(z[a * block:b * block], V[a * block:b * block])
                  for a, b in zip(edges[:-1], edges[1:])]
        states.append(O.partial_state(z[:0], V[:0]))          # an empty split is ignored
        o, lse = O.lse_merge(states)
        np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
        assert abs(lse - lse_ref) < 1e-12


def test_batch_driver_gqa_mapping_and_ragged_lengths():
    """decode_batch maps query head h to KV head h // G and honours per-sequence lengths."""
    from ffd_inputs import small_case
    c = small_case(seed=21, B=2, Hq=8, Hkv=2, seq_lens=(300, 129))
    r = O.decode_batch(c.q, c.k, c.v, c.seq_lens, delta=5.0, n_sink=64, n_local=256)
    for b in range(2):
        L = int(c.seq_lens[b])
        for h in range(8):
            kv = h // 4
            q = O.bf16_to_f64(c.q[b, h:h + 1])
            K = O.bf16_to_f64(c.k[b, kv, :L])
            V = O.bf16_to_f64(c.v[b, kv, :L])
            g = O.decode_group(q, K, V, L, delta=5.0, n_sink=64, n_local=256, block=64,
                               alpha=1 / math.sqrt(128))
            np.testing.assert_allclose(r["out"][b, h], g["out"][0], rtol=0, atol=1e-13)
            nb = -(-L // 64)
            assert r["keep"][b, h, :nb].tolist() == g["keep"][0].tolist()
            assert not r["keep"][b, h, nb:].any()
