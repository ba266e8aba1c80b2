"""CPU oracle for Faster Flash Decoding (FFD) decode attention.

TEST INFRASTRUCTURE ONLY. Only the tests, the package smoke check and the benchmark's CPU-baseline
leg may import this module. The product path (the HIP library and its binding) never calls it.

Plain, slow, obviously correct: numpy in float64, one function per step of the method, each
citing the passage of the paper it follows. It shares no code with the HIP path.

Notation (paper): ``q`` query of one head, ``k`` key, ``d`` head dimension, ``alpha = 1/sqrt(d)``;
``k^quant`` the 2-bit thumbnail, ``k^res`` the 8-bit residual; ``m~`` the pseudo-max;
``delta`` the top-delta margin; ``S_global`` sink tokens, ``S_local`` local tokens.

Readings of the paper taken where it is silent or ambiguous (each is listed in the design notes):

* Quantizer (App. A): one scale per token per KV head over its ``d`` channels, ``s = M / 1.5`` with
  ``M = max_i |k_i|``; nearest level of ``{-1.5, -0.5, 0.5, 1.5}``; a tie at a bin edge goes to the
  upper level; ``M = 0`` gives code 2 (level +0.5) and a zero reconstruction.
* Residual (Sec. 3.1 "8-bit residual"): an int8 ``r`` on the shared step ``s / 254`` so that
  ``k^quant + k^res = (s)(level + r/254) = M n / 381`` with ``n = rint(381 k / M)`` (ties to even)
  and ``r = n - 254 c + 381`` in ``[-127, 127]``.
* Wider thumbnails (App. C, the 4+8 and 8+8 depths): the same mid-rise scheme with ``2^b`` levels
  ``c - Lv``, ``Lv = (2^b - 1)/2``, ``s = M / Lv``, and the same 8-bit residual on ``s / 254``, so
  ``n = rint(254 Lv k / M)`` and ``r = n - 254 c + 254 Lv``. ``b = 2`` is the formulation above.
* All scores (scan, pseudo-max, block score, refined logits) carry the ``1/sqrt(d)`` of Eq. 1.
* The pseudo-max (Alg. 1; Eq. 3) is taken over thumbnail scores of the first ``n_sink`` tokens and
  the last ``n_local`` tokens of the sequence. Eq. 3's own reading (the window tokens' true scores)
  is available as a variant: ``pm_source="refined"`` (thumbnail + residual, Eq. 4's logits) or
  ``"exact"`` (the bf16 keys themselves).
* A block is tokens ``[B*j, min(B*j + B, L))``; only valid tokens enter its score and the softmax.
* Masks are per query head; a KV head's residual/values are read for the union over its group.
* An empty selection or an empty sequence gives output 0 and ``lse = -inf``.
"""
from __future__ import annotations

import numpy as np

# App. A: the 4-level symmetric mid-rise codebook; code c in {0,1,2,3} stands for level c - 1.5.
CODEBOOK = np.array([-1.5, -0.5, 0.5, 1.5], dtype=np.float64)
RESID_STEPS = 254          # residual step is s / 254 (Sec. 3.1 8-bit residual reading)
FULL_LEVELS = 381          # 1.5 * 254: k^quant + k^res = M * n / 381
THUMB_BITS = (2, 4, 8)     # thumbnail depths of App. C (2+8, 4+8, 8+8)


def top_level(bits: int = 2) -> float:
    """``Lv = (2^b - 1) / 2``: the outer level of the b-bit mid-rise codebook (1.5 for App. A)."""
    return (2 ** bits - 1) / 2.0


def codebook(bits: int = 2) -> np.ndarray:
    """The ``2^b`` levels ``c - Lv`` for ``c = 0 .. 2^b - 1`` (App. A's codebook when ``b = 2``)."""
    return np.arange(2 ** bits, dtype=np.float64) - top_level(bits)


def full_levels(bits: int = 2) -> int:
    """``254 Lv``: thumbnail plus residual is ``M n / full_levels`` (381 for 2+8, 32385 for 8+8)."""
    return RESID_STEPS * (2 ** bits - 1) // 2


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) into float64 values (exact)."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return u32.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 bit patterns: one IEEE round to nearest, ties to even.

    bf16 keeps 8 significant bits over float32's exponent range, so the quantum of a value
    ``m 2^e`` (``0.5 <= |m| < 1``) is ``2^(e - 8)``, and never finer than the subnormal step
    ``2^-133``. The value is scaled to units of that quantum (exact), rounded with ``rint``
    (half to even) and scaled back: a bf16 value, or ``2^128`` and beyond, which becomes infinity.
    NaN maps to the quiet NaN of its sign; signed zeros and infinities are kept. (Rounding to
    float32 first would round twice: ``1 + 2^-8 + 2^-30`` would become the tie ``1 + 2^-8`` and
    then ``1`` instead of ``1 + 2^-7``.)
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e.astype(np.int64) - 8, -133)
    with np.errstate(over="ignore", invalid="ignore"):
        y = np.ldexp(np.rint(np.ldexp(x, -q)), q).astype(np.float32)
    bits = (np.ascontiguousarray(y).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    nan = np.where(np.signbit(x), np.uint16(0xFFC0), np.uint16(0x7FC0))
    return np.where(np.isnan(x), nan, bits).astype(np.uint16)


# ------------------------------------------------------------------------------------------------
# Q1/Q2. Key decomposition k -> {k^quant, k^res} (Sec. 3.1; App. A formulation).
# ------------------------------------------------------------------------------------------------

_QUANT_ROWS = 4096


def quantize_keys(K: np.ndarray, bits: int = 2):
    """Thumbnail codes, absmax and residual of every key vector (App. A; Sec. 3.1; App. C depths).

    ``K``: float64 ``[..., d]`` of bf16-exact values. Returns ``codes`` (int64 in ``0 .. 2^b - 1``),
    ``M`` (float64 ``[...]``, the per-vector absmax) and ``resid`` (int64 in -127..127).

    Nearest level: with ``x/s = Lv k / M`` the edges between consecutive levels ``c - 1 - Lv`` and
    ``c - Lv`` are the integers ``c - 2^(b-1)``, so the nearest level has ``c = floor(x/s) + 2^(b-1)``
    and a value on an edge goes to the upper level. ``floor(x/s) = floor((2^b - 1) k / (2M))`` is
    taken in float64 and then settled by exact comparisons (``(2^b - 1) k`` and ``i * 2M`` are
    products of two 8-bit significands, exact in float64). For ``b = 2`` this is ``3k`` against
    ``-2M, 0, 2M``.

    Residual: ``n = rint(254 Lv k / M)`` (round half to even). ``254 Lv k`` is exact in float64; a
    quotient ``Q`` that is not a tie lies at least ``2^-24 Q`` from every half-integer (its distance
    is a multiple of half the unit of ``k`` over ``M``, and ``254 Lv < 2^15``), while the division
    moves it by at most ``2^-53 Q``, so the rounding is the exact one.
    """
    K = np.asarray(K, dtype=np.float64)
    if K.ndim >= 2 and K.shape[0] > _QUANT_ROWS:
        # rows are independent: quantize them in pieces, so the temporaries stay small
        parts = [quantize_keys(K[i:i + _QUANT_ROWS], bits) for i in range(0, K.shape[0], _QUANT_ROWS)]
        return tuple(np.concatenate([p[k] for p in parts]) for k in range(3))
    M = np.max(np.abs(K), axis=-1)
    Mx = M[..., None]
    u = (2 ** bits - 1) * K
    D = 2.0 * Mx
    zero = Mx == 0.0
    with np.errstate(divide="ignore", invalid="ignore"):
        i = np.floor(u / D)
    i = np.where(zero, 0.0, i)
    i = np.where((i + 1.0) * D <= u, i + 1.0, i)
    i = np.where(i * D > u, i - 1.0, i)
    codes = np.clip(i + 2 ** (bits - 1), 0, 2 ** bits - 1).astype(np.int64)
    codes = np.where(zero, 2 ** (bits - 1), codes)
    N = full_levels(bits)
    with np.errstate(divide="ignore", invalid="ignore"):
        n = np.rint(N * K / Mx)                    # round half to even
    n = np.where(zero, 0.0, n).astype(np.int64)
    resid = np.where(zero, 0, n - RESID_STEPS * codes + N).astype(np.int64)
    return codes, M, resid


def thumbnail(codes: np.ndarray, M: np.ndarray, bits: int = 2) -> np.ndarray:
    """Dequantized thumbnail ``k^quant = (c - Lv) s`` with ``s = M / Lv`` (App. A reconstruction)."""
    s = np.asarray(M, dtype=np.float64)[..., None] / top_level(bits)
    return codebook(bits)[codes] * s


def residual_part(resid: np.ndarray, M: np.ndarray, bits: int = 2) -> np.ndarray:
    """The residual's contribution ``k^res = s r / 254`` (Sec. 3.1 reading; Eq. 4's second term)."""
    s = np.asarray(M, dtype=np.float64)[..., None] / top_level(bits)
    return s * (np.asarray(resid, dtype=np.float64) / RESID_STEPS)


# ------------------------------------------------------------------------------------------------
# S1. Thumbnail scan (Alg. 1 top-delta loop; Sec. 3.3 step 2), scaled by 1/sqrt(d) (Eq. 1).
# ------------------------------------------------------------------------------------------------

def scan_scores(q: np.ndarray, codes: np.ndarray, M: np.ndarray, alpha: float,
                bits: int = 2) -> np.ndarray:
    """``s_hat[h, t] = alpha * q_h . k^quant_t`` for every head of the group and every token."""
    return alpha * (np.asarray(q, dtype=np.float64) @ thumbnail(codes, M, bits).T)


# ------------------------------------------------------------------------------------------------
# S2. Pseudo-max over sink and local tokens (Alg. 1 pseudo-max lines; Sec. 3.2 Eq. 3).
# ------------------------------------------------------------------------------------------------

def pseudo_max_tokens(L: int, n_sink: int, n_local: int) -> np.ndarray:
    """Indices of ``S_global`` (first ``n_sink``) and ``S_local`` (last ``n_local``), clipped to L."""
    sink = np.arange(0, min(n_sink, L))
    local = np.arange(max(0, L - n_local), L)
    return np.union1d(sink, local).astype(np.int64)


PM_SOURCES = ("thumbnail", "refined", "exact")


def window_scores(source, s_hat, z, q, K, L, alpha):
    """The scores the pseudo-max is taken over: the thumbnail scores (Alg. 1, the default), the
    refined logits (thumbnail + residual, Eq. 4), or the exact scores of the bf16 keys (Eq. 3's
    ``s_it``). Only the window tokens' entries are used."""
    if source == "thumbnail":
        return s_hat
    if source == "refined":
        return z
    if source == "exact":
        return alpha * (np.asarray(q, dtype=np.float64) @ np.asarray(K[:L], dtype=np.float64).T)
    raise ValueError(f"pm_source must be one of {PM_SOURCES}")


def pseudo_max(s_hat: np.ndarray, L: int, n_sink: int, n_local: int) -> np.ndarray:
    """``m~_h = max(max_{S_global} s_hat, max_{S_local} s_hat)`` per head; ``-inf`` if both are empty."""
    idx = pseudo_max_tokens(L, n_sink, n_local)
    if idx.size == 0:
        return np.full(s_hat.shape[0], -np.inf)
    return np.max(s_hat[:, idx], axis=1)


# ------------------------------------------------------------------------------------------------
# S3. Block score and top-delta decision (Alg. 1 selection; Eq. 1 with m replaced by m~).
# ------------------------------------------------------------------------------------------------

def block_scores(s_hat: np.ndarray, L: int, block: int) -> np.ndarray:
    """``sigma[h, j] = max`` of ``s_hat`` over the valid tokens of block ``j``."""
    nblk = -(-L // block)
    out = np.full((s_hat.shape[0], nblk), -np.inf)
    for j in range(nblk):
        out[:, j] = np.max(s_hat[:, j * block:min(j * block + block, L)], axis=1)
    return out


def select_blocks(sigma: np.ndarray, m_tilde: np.ndarray, delta: float) -> np.ndarray:
    """Keep block ``j`` for head ``h`` iff ``sigma[h, j] >= m~_h - delta`` (inclusive, Eq. 1)."""
    return sigma >= (m_tilde[:, None] - delta)


def select_topk(sigma: np.ndarray, k: int) -> np.ndarray:
    """The fixed-budget rule the paper compares against (Table 3; Fig. 1 (a)): keep, per head, the
    ``k`` blocks with the largest block scores (all of them if there are fewer). Equal scores are
    taken in block order, i.e. the first ``k`` of a stable sort by decreasing score."""
    sigma = np.asarray(sigma, dtype=np.float64)
    keep = np.zeros(sigma.shape, dtype=bool)
    for h in range(sigma.shape[0]):
        order = np.argsort(-sigma[h], kind="stable")
        keep[h, order[:min(k, sigma.shape[1])]] = True
    return keep


# ------------------------------------------------------------------------------------------------
# S4. Refinement with scan reuse (Alg. 1 refinement; Sec. 3.3 Eq. 4).
# ------------------------------------------------------------------------------------------------

def refined_logits(q, codes, M, resid, alpha, bits=2):
    """``s_final = (q . k^quant + q . k^res) / sqrt(d)``: the scan term plus the residual term."""
    q = np.asarray(q, dtype=np.float64)
    return alpha * (q @ thumbnail(codes, M, bits).T + q @ residual_part(resid, M, bits).T)


# ------------------------------------------------------------------------------------------------
# S5. Sparse softmax . V over the selected tokens (Alg. 1 output line).
# ------------------------------------------------------------------------------------------------

def softmax_attend(z: np.ndarray, V: np.ndarray):
    """Softmax of ``z`` over its tokens times ``V``; returns ``(o, lse)``. Empty -> ``(0, -inf)``."""
    V = np.asarray(V, dtype=np.float64)
    if z.size == 0:
        return np.zeros(V.shape[-1]), -np.inf
    m = np.max(z)
    p = np.exp(z - m)
    l = np.sum(p)
    return (p @ V) / l, m + np.log(l)


def token_mask_from_blocks(keep_blocks: np.ndarray, L: int, block: int) -> np.ndarray:
    """Expand a per-block keep vector to the valid tokens ``t < L``."""
    return np.repeat(np.asarray(keep_blocks, dtype=bool), block)[:L]


# ------------------------------------------------------------------------------------------------
# S6. Exact dense attention (the comparator's definition) over the exact bf16 keys.
# ------------------------------------------------------------------------------------------------

def dense_attention(q, K, V, L, alpha):
    """``softmax(alpha q K^T) V`` over tokens ``t < L`` for every head of the group."""
    q = np.asarray(q, dtype=np.float64)
    outs, lses = [], []
    for h in range(q.shape[0]):
        z = alpha * (np.asarray(K[:L], dtype=np.float64) @ q[h])
        o, lse = softmax_attend(z, V[:L])
        outs.append(o)
        lses.append(lse)
    return np.stack(outs), np.array(lses)


# ------------------------------------------------------------------------------------------------
# Split-K partials and their log-sum-exp merge (flash-decoding split along the sequence, Sec. 2).
# ------------------------------------------------------------------------------------------------

def partial_state(z, V):
    """One split's ``(m, l, acc)``: running max, sum of ``exp(z - m)``, unnormalised output."""
    if z.size == 0:
        return -np.inf, 0.0, np.zeros(np.asarray(V).shape[-1])
    m = np.max(z)
    p = np.exp(z - m)
    return m, np.sum(p), p @ np.asarray(V, dtype=np.float64)


def lse_merge(states):
    """Merge split states: ``M* = max m_s``, ``l* = sum e^{m_s - M*} l_s``, ``o = sum e^{m_s-M*} acc_s / l*``."""
    ms = np.array([s[0] for s in states], dtype=np.float64)
    if ms.size == 0 or not np.isfinite(ms).any():
        return np.zeros_like(states[0][2]) if states else None, -np.inf
    Mx = np.max(ms)
    w = np.where(np.isfinite(ms), np.exp(ms - Mx), 0.0)
    l = sum(wi * s[1] for wi, s in zip(w, states))
    acc = sum(wi * s[2] for wi, s in zip(w, states))
    return acc / l, Mx + np.log(l)


# ------------------------------------------------------------------------------------------------
# The whole decode step for one (sequence, KV head) group, and for a batch.
# ------------------------------------------------------------------------------------------------

def decode_group(q, K, V, L, *, delta, n_sink, n_local, block, alpha, keep=None, bits=2,
                 pm_source="thumbnail", topk=0):
    """FFD decode for the ``G`` query heads ``q [G, d]`` sharing keys ``K [Lcap, d]``, values ``V``.

    Follows Alg. 1 in order: quantize, pseudo-max, top-delta selection, refinement, softmax . V.
    When ``keep`` (bool ``[G, nblk]``) is given, attention runs on that mask instead of the
    oracle's own selection (used to compare outputs given the GPU's mask). ``bits`` is the
    thumbnail depth (App. C); ``pm_source`` the scores the pseudo-max is taken over
    (:func:`window_scores`); ``topk > 0`` replaces the top-delta rule by :func:`select_topk`.
    """
    codes, M, resid = quantize_keys(K[:L], bits)
    return decode_group_quantized(q, codes, M, resid, V, L, delta=delta, n_sink=n_sink,
                                  n_local=n_local, block=block, alpha=alpha, keep=keep, bits=bits,
                                  pm_source=pm_source, K=K, topk=topk)


def decode_group_quantized(q, codes, M, resid, V, L, *, delta, n_sink, n_local, block, alpha,
                           keep=None, bits=2, pm_source="thumbnail", K=None, topk=0):
    """The decode step of :func:`decode_group` given the already quantized keys (Alg. 1 from the
    pseudo-max on; the quantization happens when the cache is written, Fig. 2). ``K`` (the exact
    keys) is needed only for ``pm_source="exact"``."""
    s_hat = scan_scores(q, codes, M, alpha, bits)
    z_all = refined_logits(q, codes, M, resid, alpha, bits)
    m_tilde = pseudo_max(window_scores(pm_source, s_hat, z_all, q, K, L, alpha), L, n_sink, n_local)
    sigma = block_scores(s_hat, L, block)
    own_keep = select_topk(sigma, topk) if topk > 0 else select_blocks(sigma, m_tilde, delta)
    use = own_keep if keep is None else np.asarray(keep, dtype=bool)[:, :sigma.shape[1]]
    outs, lses = [], []
    for h in range(q.shape[0]):
        tok = token_mask_from_blocks(use[h], L, block)
        o, lse = softmax_attend(z_all[h, :L][tok], np.asarray(V[:L], dtype=np.float64)[tok])
        outs.append(o)
        lses.append(lse)
    return dict(out=np.stack(outs), lse=np.array(lses), keep=own_keep, sigma=sigma,
                m_tilde=m_tilde, s_hat=s_hat)


def decode_batch(q_bits, k_bits, v_bits, seq_lens, *, delta, n_sink, n_local, block=64,
                 softmax_scale=None, keep=None, heads=None, bits=2, pm_source="thumbnail", topk=0):
    """FFD decode for a batch. Inputs are bf16 bit patterns ``q [B,Hq,d]``, ``k, v [B,Hkv,Lcap,d]``.

    Returns float64 ``out [B,Hq,d]``, ``lse [B,Hq]``, the per-head block mask ``keep [B,Hq,nblk]``
    (blocks at or beyond a sequence's end are False), ``sigma`` and ``m_tilde``.
    ``heads`` optionally restricts work to a list of ``(b, kvh)`` pairs (others left as NaN);
    ``bits`` is the thumbnail depth (App. C), ``pm_source`` the pseudo-max's scores, ``topk > 0``
    the fixed-budget rule instead of top-delta.
    """
    B, Hq, d = q_bits.shape
    Hkv, Lcap = k_bits.shape[1], k_bits.shape[2]
    G = Hq // Hkv
    alpha = 1.0 / np.sqrt(d) if not softmax_scale else float(softmax_scale)
    nblk = -(-Lcap // block)
    out = np.full((B, Hq, d), np.nan)
    lse = np.full((B, Hq), np.nan)
    mask = np.zeros((B, Hq, nblk), dtype=bool)
    sigma = np.full((B, Hq, nblk), -np.inf)
    m_tilde = np.full((B, Hq), np.nan)
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hkv)]
    for b, h in pairs:
        L = int(seq_lens[b])
        sl = slice(h * G, (h + 1) * G)
        q = bf16_to_f64(q_bits[b, sl])
        if L == 0:
            out[b, sl] = 0.0
            lse[b, sl] = -np.inf
            m_tilde[b, sl] = -np.inf
            continue
        K = bf16_to_f64(k_bits[b, h, :L])
        V = bf16_to_f64(v_bits[b, h, :L])
        kb = None if keep is None else np.asarray(keep[b, sl], dtype=bool)
        r = decode_group(q, K, V, L, delta=delta, n_sink=n_sink, n_local=n_local, block=block,
                         alpha=alpha, keep=kb, bits=bits, pm_source=pm_source, topk=topk)
        nb = r["sigma"].shape[1]
        out[b, sl] = r["out"]
        lse[b, sl] = r["lse"]
        mask[b, sl, :nb] = r["keep"]
        sigma[b, sl, :nb] = r["sigma"]
        m_tilde[b, sl] = r["m_tilde"]
    return dict(out=out, lse=lse, keep=mask, sigma=sigma, m_tilde=m_tilde)


def dense_batch(q_bits, k_bits, v_bits, seq_lens, *, softmax_scale=None, heads=None):
    """Exact dense attention over bf16 keys/values for a batch (the dense baseline's definition)."""
    B, Hq, d = q_bits.shape
    Hkv = k_bits.shape[1]
    G = Hq // Hkv
    alpha = 1.0 / np.sqrt(d) if not softmax_scale else float(softmax_scale)
    out = np.full((B, Hq, d), np.nan)
    lse = np.full((B, Hq), np.nan)
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hkv)]
    for b, h in pairs:
        L = int(seq_lens[b])
        sl = slice(h * G, (h + 1) * G)
        o, l = dense_attention(bf16_to_f64(q_bits[b, sl]), bf16_to_f64(k_bits[b, h, :L]),
                               bf16_to_f64(v_bits[b, h, :L]), L, alpha)
        out[b, sl] = o
        lse[b, sl] = l
    return dict(out=out, lse=lse)


# ------------------------------------------------------------------------------------------------
# Fidelity diagnostics (Sec. 5.1 recall and LSE error; Sec. 5.2 pseudo-max gap).
# ------------------------------------------------------------------------------------------------

def exact_max(q, K, L, alpha):
    """``m_h = max_{t < L} alpha q_h . k_t``, the true maximum score the pseudo-max estimates
    (Sec. 5.2); ``-inf`` for an empty sequence."""
    if L == 0:
        return np.full(np.asarray(q).shape[0], -np.inf)
    return np.max(alpha * (np.asarray(q, dtype=np.float64) @ np.asarray(K[:L], dtype=np.float64).T), axis=1)


def pseudo_max_gap(m, m_tilde):
    """``m - m~`` per head (Sec. 5.2, Fig. 5); 0 where both are ``-inf``."""
    m, mt = np.asarray(m, dtype=np.float64), np.asarray(m_tilde, dtype=np.float64)
    with np.errstate(invalid="ignore"):
        return np.where(np.isneginf(m) & np.isneginf(mt), 0.0, m - mt)


def recall_cosine(out, ref):
    """Sec. 5.1 recall: the cosine similarity of the sparse output and the dense output, per head
    (the last axis is the head dimension); 1 where both are zero."""
    a, b = np.asarray(out, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    na, nb = np.linalg.norm(a, axis=-1), np.linalg.norm(b, axis=-1)
    dot = np.sum(a * b, axis=-1)
    with np.errstate(invalid="ignore", divide="ignore"):
        c = dot / (na * nb)
    return np.where((na == 0) & (nb == 0), 1.0, c)


def lse_abs_error(lse, ref):
    """Sec. 5.1 LSE error: ``|lse - lse_dense|`` per head (0 where both are ``-inf``)."""
    a, b = np.asarray(lse, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    with np.errstate(invalid="ignore"):
        return np.where(np.isneginf(a) & np.isneginf(b), 0.0, np.abs(a - b))


def near_threshold(sigma, m_tilde, delta, band=1e-3):
    """Blocks whose score lies strictly within ``band`` of the threshold ``m~ - delta`` of Eq. 1:
    ``|sigma - (m~ - delta)| < band`` with ``sigma`` finite. Their keep decision may differ between
    two correct implementations that round the scores differently, so parity reports them apart.
    ``sigma`` is ``[..., nblk]`` and ``m_tilde`` ``[...]``; an empty block (``sigma = -inf``), an
    empty window (``m~ = -inf``) and ``delta = inf`` give no near block."""
    thr = np.asarray(m_tilde)[..., None] - delta
    with np.errstate(invalid="ignore"):
        return np.isfinite(sigma) & (np.abs(sigma - thr) < band)


# ------------------------------------------------------------------------------------------------
# Storage layouts of the quantized copy (this implementation's format; the paper fixes none).
# They are written out independently of the HIP code, from the format's definition:
#
#  codes  uint32 [B, Hkv, Lcap/64, b, 64, 4] for a b-bit thumbnail. Block j (tokens 64j..64j+63)
#         holds 4b words for each lane l = n + 16g; word w of lane l is element [j, w // 4, l, w % 4].
#         Lane l's words hold, for token 64j + 16*t4 + n and 64-dim chunk cc, the codes of dims
#         64cc + 16g + e (e = 4k + i, k, i in 0..3) in the b/2 words starting at (2*t4 + cc) * b/2:
#         dim e sits in word (2*t4 + cc) * b/2 + k // (8/b), at bit 8i + b * (k % (8/b)). The field
#         holds c for b = 2, 4 and the byte c - 128 (two's complement) for b = 8. For b = 2 this is
#         word 2*t4 + cc, bit 8i + 2k.
#  absmax bf16 [B, Hkv, Lcap/64, 16, 4]. Element [j, n, t4] is M of token 64j + 16*t4 + n.
#  resid  int8 [B, Hkv, Lcap/16, 2, 64, 16]. Element [T, cc, n + 16g, e] is the residual of token
#         16T + n at dim 64cc + 16g + e.
# ------------------------------------------------------------------------------------------------

def _code_field(c: int, bits: int) -> int:
    """The stored field of code ``c``: ``c`` itself, or the byte ``c - 128`` for 8-bit codes."""
    return (int(c) - 128) & 0xFF if bits == 8 else int(c)


def pack_codes(codes: np.ndarray, bits: int = 2) -> np.ndarray:
    """Pack ``codes [Lcap, 128]`` (``0 .. 2^b - 1``) into the ``[Lcap/64, b, 64, 4]`` uint32 layout."""
    Lcap = codes.shape[0]
    per = 8 // bits                                   # codes per byte
    out = np.zeros((Lcap // 64, bits, 64, 4), dtype=np.uint32)
    for j in range(Lcap // 64):
        for g in range(4):
            for n in range(16):
                for t4 in range(4):
                    t = 64 * j + 16 * t4 + n
                    for cc in range(2):
                        w0 = (2 * t4 + cc) * (bits // 2)
                        for e in range(16):
                            k, i = divmod(e, 4)
                            w = w0 + k // per
                            f = _code_field(codes[t, 64 * cc + 16 * g + e], bits)
                            out[j, w // 4, n + 16 * g, w % 4] |= np.uint32(f << (8 * i + bits * (k % per)))
    return out


def unpack_codes(packed: np.ndarray, Lcap: int, bits: int = 2) -> np.ndarray:
    """Inverse of :func:`pack_codes`."""
    packed = np.asarray(packed, dtype=np.uint32).reshape(Lcap // 64, bits, 64, 4)
    per = 8 // bits
    codes = np.zeros((Lcap, 128), dtype=np.int64)
    for j in range(Lcap // 64):
        for g in range(4):
            for n in range(16):
                for t4 in range(4):
                    for cc in range(2):
                        w0 = (2 * t4 + cc) * (bits // 2)
                        for e in range(16):
                            k, i = divmod(e, 4)
                            w = w0 + k // per
                            word = int(packed[j, w // 4, n + 16 * g, w % 4])
                            f = (word >> (8 * i + bits * (k % per))) & (2 ** bits - 1)
                            c = (f + 128) & 0xFF if bits == 8 else f
                            codes[64 * j + 16 * t4 + n, 64 * cc + 16 * g + e] = c
    return codes


def pack_codes_fast(codes: np.ndarray, bits: int = 2) -> np.ndarray:
    """Vectorised :func:`pack_codes` (checked equal to the loop form on small inputs)."""
    Lcap = codes.shape[0]
    per = 8 // bits
    c = np.asarray(codes, dtype=np.int64)
    f = ((c - 128) & 0xFF) if bits == 8 else c
    # axes: j, t4, n, cc, g, (k // per), (k % per), i
    f = f.astype(np.uint32).reshape(Lcap // 64, 4, 16, 2, 4, bits // 2, per, 4)
    f = f.transpose(0, 4, 2, 1, 3, 5, 6, 7)           # j, g, n, t4, cc, k // per, k % per, i
    shift = (8 * np.arange(4)[None, :] + bits * np.arange(per)[:, None]).astype(np.uint32)
    words = np.bitwise_or.reduce((f << shift).reshape(*f.shape[:6], 4 * per), axis=-1)
    return piece_major(words.reshape(Lcap // 64, 64, 4 * bits).astype(np.uint32), bits)


def piece_major(lane_words: np.ndarray, bits: int) -> np.ndarray:
    """``[J, 64, 4b]`` (lane, word) -> the stored ``[J, b, 64, 4]`` order (word w at [w // 4, l, w % 4])."""
    J = lane_words.shape[0]
    return np.ascontiguousarray(lane_words.reshape(J, 64, bits, 4).transpose(0, 2, 1, 3))


def lane_words(packed: np.ndarray, bits: int) -> np.ndarray:
    """Inverse of :func:`piece_major`."""
    J = packed.shape[0]
    return np.ascontiguousarray(packed.reshape(J, bits, 64, 4).transpose(0, 2, 1, 3)).reshape(J, 64, 4 * bits)


def pack_absmax(M_bits: np.ndarray) -> np.ndarray:
    """Permute per-token absmax bits ``[Lcap]`` into the ``[Lcap/64, 16, 4]`` layout above."""
    Lcap = M_bits.shape[0]
    return np.asarray(M_bits).reshape(Lcap // 64, 4, 16).transpose(0, 2, 1).copy()


def pack_resid(resid: np.ndarray) -> np.ndarray:
    """Tile residuals ``[Lcap, 128]`` into the ``[Lcap/16, 2, 64, 16]`` int8 layout above."""
    Lcap = resid.shape[0]
    r = np.asarray(resid, dtype=np.int8).reshape(Lcap // 16, 16, 2, 4, 16)  # T,n,cc,g,e
    return r.transpose(0, 2, 3, 1, 4).reshape(Lcap // 16, 2, 64, 16).copy()


def quantize_cache(k_bits: np.ndarray, t_begin: int = 0, t_end: int | None = None, bits: int = 2):
    """Oracle for the quantization pass: packed ``(codes, absmax_bits, resid)`` for ``[B,Hkv,Lcap,128]``
    with a ``bits``-bit thumbnail.

    Only tokens in ``[t_begin, t_end)`` are defined; the others are returned as zero.
    """
    B, Hkv, Lcap, d = k_bits.shape
    t_end = Lcap if t_end is None else t_end
    codes = np.zeros((B, Hkv, Lcap // 64, bits, 64, 4), dtype=np.uint32)
    absmax = np.zeros((B, Hkv, Lcap // 64, 16, 4), dtype=np.uint16)
    resid = np.zeros((B, Hkv, Lcap // 16, 2, 64, 16), dtype=np.int8)
    live = np.zeros(Lcap, dtype=bool)
    live[t_begin:t_end] = True
    for b in range(B):
        for h in range(Hkv):
            K = bf16_to_f64(k_bits[b, h])
            c, M, r = quantize_keys(K, bits)
            c = np.where(live[:, None], c, 0)
            r = np.where(live[:, None], r, 0)
            Mb = np.where(live, f64_to_bf16_bits(M), 0).astype(np.uint16)
            packed = pack_codes_fast(c, bits)
            if bits == 8:                             # tokens outside the range hold zero words
                dead = ~live.reshape(Lcap // 64, 4, 16).transpose(0, 2, 1)   # j, n, t4
                lw = lane_words(packed, bits).reshape(Lcap // 64, 4, 16, 4, 2, 4)   # j, g, n, t4, cc, k
                lw[np.broadcast_to(dead[:, None, :, :, None, None], lw.shape)] = 0
                packed = piece_major(lw.reshape(Lcap // 64, 64, 32), bits)
            codes[b, h] = packed
            absmax[b, h] = pack_absmax(Mb)
            resid[b, h] = pack_resid(r)
    return codes, absmax, resid
