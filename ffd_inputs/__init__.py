"""Seeded synthetic decode-attention inputs shaped like the workloads of Faster Flash Decoding.

This module is shared by the CPU oracle and by the GPU path. It holds none of the method's
arithmetic: it only draws queries, keys and values, plants structure (heavy blocks, an attention
sink, a recent window), and rounds float32 draws to bfloat16 bit patterns.

Recipe:

1. ``numpy.random.default_rng(seed)``: ragged workloads draw the per-sequence lengths first, then
   ``q ~ N(0, 1)`` of shape ``[B, Hq, D]``, rounded to bf16;
2. each sequence ``b`` and KV head ``kvh`` has its own stream ``default_rng([seed, b, kvh])``:
   ``K ~ N(0, 1)`` and ``V ~ N(0, 1)`` of shape ``[Lcap, D]``, then that pair's structure draws.
   Pairs are independent, so they are generated in parallel threads.

Structure. A planted direction per ``(b, kvh)`` is ``u = sqrt(D) * qbar / |qbar|`` where ``qbar``
is the mean of the group's bf16 queries; ``|u| = sqrt(D)`` is the norm of a typical N(0,1) key.
A planted key is ``a * u + N(0, 0.5**2)`` per element. Heavy blocks (``a = 2.5``) are drawn without
replacement among blocks that hold neither token 0 nor any of the last ``n_local`` tokens (nor
the recent window, when there is one). The sink is token 0 planted with ``a = 2.5``. Tokens at or
beyond a sequence's length hold a deterministic poison (keys ``3u``, values ``64``) so that any
read past the end shows up in the results.

Arrays are returned as ``uint16`` bf16 bit patterns.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

BLOCK = 64
HEAD_DIM = 128
DEFAULT_N_SINK = 64
DEFAULT_N_LOCAL = 256
HEAVY_AMPLITUDE = 2.5
RECENT_AMPLITUDE = 1.5
PLANT_NOISE_STD = 0.5
POISON_KEY_SCALE = 3.0
POISON_VALUE = 64.0


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even) and return the bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Case:
    """One decode step's inputs. Keys/values are ``[B, Hkv, Lcap, D]``, queries ``[B, Hq, D]``."""

    name: str
    seed: int
    B: int
    Hq: int
    Hkv: int
    D: int
    Lcap: int
    block: int
    seq_lens: np.ndarray          # int32 [B]
    q: np.ndarray                 # uint16 bf16 bits [B, Hq, D]
    k: np.ndarray                 # uint16 bf16 bits [B, Hkv, Lcap, D]
    v: np.ndarray                 # uint16 bf16 bits [B, Hkv, Lcap, D]
    n_sink: int = DEFAULT_N_SINK
    n_local: int = DEFAULT_N_LOCAL
    deltas: tuple = (5.0,)
    heavy_blocks: dict = field(default_factory=dict)   # (b, kvh) -> sorted list of block ids
    sink: np.ndarray | None = None                     # bool [B]
    recent_tokens: int = 0

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


def _planted_direction(q_bits_group: np.ndarray) -> np.ndarray:
    qbar = bf16_bits_to_f32(q_bits_group).astype(np.float64).mean(axis=0)
    nrm = np.linalg.norm(qbar)
    if nrm == 0.0:
        qbar = np.ones_like(qbar)
        nrm = np.linalg.norm(qbar)
    return (np.sqrt(qbar.size) * qbar / nrm).astype(np.float32)


def _eligible_blocks(L: int, block: int, exclude_tail: int) -> np.ndarray:
    """Blocks j >= 1 lying wholly before the last ``exclude_tail`` tokens."""
    last = (L - exclude_tail) // block          # blocks [0, last) end at or before L - exclude_tail
    return np.arange(1, max(last, 1), dtype=np.int64)


def _random_blocks(rng, L, block, exclude_tail, count):
    pool = _eligible_blocks(L, block, exclude_tail)
    count = int(min(count, pool.size))
    if count <= 0:
        return []
    return sorted(int(x) for x in rng.choice(pool, size=count, replace=False))


def _clustered_blocks(rng, L, block, exclude_tail, sizes):
    """Non-overlapping runs of ``sizes`` blocks, placed uniformly at random (in the given order)."""
    pool = _eligible_blocks(L, block, exclude_tail)
    total = int(sum(sizes))
    free = int(pool.size) - total
    if free < 0:
        raise ValueError("clusters do not fit")
    slots = np.sort(rng.choice(free + len(sizes), size=len(sizes), replace=False))
    out, used = [], 0
    for i, (slot, size) in enumerate(zip(slots, sizes)):
        start = int(pool[0]) + int(slot) - i + used
        out.extend(range(start, start + size))
        used += size
    return sorted(out)


def generate(*, name, seed, B, Hq, Hkv, Lcap, seq_lens, heavy_fn, sink_fn=lambda b: True,
             recent_tokens=0, D=HEAD_DIM, block=BLOCK, n_sink=DEFAULT_N_SINK,
             n_local=DEFAULT_N_LOCAL, deltas=(5.0,), rng=None) -> Case:
    """Draw one case. ``heavy_fn(rng, b, kvh, L)`` returns that pair's heavy block ids."""
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    rng = np.random.default_rng(seed) if rng is None else rng
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    G = Hq // Hkv
    q = f32_to_bf16_bits(rng.standard_normal((B, Hq, D), dtype=np.float32))
    k = np.empty((B, Hkv, Lcap, D), dtype=np.uint16)
    v = np.empty((B, Hkv, Lcap, D), dtype=np.uint16)
    sinks = np.array([bool(sink_fn(b)) for b in range(B)], dtype=bool)

    def one_pair(b, h):
        prng = np.random.default_rng([seed, b, h])
        L = int(seq_lens[b])
        kf = prng.standard_normal((Lcap, D), dtype=np.float32)
        vf = prng.standard_normal((Lcap, D), dtype=np.float32)
        u = _planted_direction(q[b, h * G:(h + 1) * G])
        blocks = list(heavy_fn(prng, b, h, L))
        for j in blocks:
            lo, hi = j * block, min(j * block + block, L)
            noise = prng.standard_normal((hi - lo, D), dtype=np.float32)
            kf[lo:hi] = HEAVY_AMPLITUDE * u + PLANT_NOISE_STD * noise
        if sinks[b] and L > 0:
            kf[0] = HEAVY_AMPLITUDE * u + PLANT_NOISE_STD * prng.standard_normal(D, dtype=np.float32)
        if recent_tokens and L > 0:
            lo = max(0, L - recent_tokens)
            noise = prng.standard_normal((L - lo, D), dtype=np.float32)
            kf[lo:L] = RECENT_AMPLITUDE * u + PLANT_NOISE_STD * noise
        kf[L:] = POISON_KEY_SCALE * u
        vf[L:] = POISON_VALUE
        k[b, h] = f32_to_bf16_bits(kf)
        v[b, h] = f32_to_bf16_bits(vf)
        return (b, h), blocks

    pairs = [(b, h) for b in range(B) for h in range(Hkv)]
    workers = max(1, min(len(pairs), 16, os.cpu_count() or 1))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        heavy = dict(ex.map(lambda bh: one_pair(*bh), pairs))
    return Case(name=name, seed=seed, B=B, Hq=Hq, Hkv=Hkv, D=D, Lcap=Lcap, block=block,
                seq_lens=seq_lens, q=q, k=k, v=v, n_sink=n_sink, n_local=n_local,
                deltas=tuple(deltas), heavy_blocks=heavy, sink=sinks, recent_tokens=recent_tokens)


# ---------------------------------------------------------------------------------------------
# The five workloads. Each is named by its shape; seeds default to 1000 + its number.
# ---------------------------------------------------------------------------------------------

WORKLOADS = {
    1: "tiny-4k-b1-8q2kv",
    2: "llama3-8b-32k-b1-32q8kv",
    3: "llama3-8b-128k-b4-32q8kv",
    4: "llama3-8b-256k-b1-32q8kv-clustered",
    5: "ragged-8k-128k-b16-32q8kv",
}


def workload(n: int, seed: int | None = None) -> Case:
    """Build workload ``n`` (1..5) at its full size."""
    seed = 1000 + n if seed is None else seed
    name = WORKLOADS[n]
    if n == 1:
        L = 4096
        return generate(name=name, seed=seed, B=1, Hq=8, Hkv=2, Lcap=L, seq_lens=[L],
                        heavy_fn=lambda rng, b, h, L: _random_blocks(rng, L, BLOCK, DEFAULT_N_LOCAL,
                                                                      round(0.03 * (L // BLOCK))),
                        deltas=(3.0, 5.0, 7.0))
    if n == 2:
        L = 32768
        return generate(name=name, seed=seed, B=1, Hq=32, Hkv=8, Lcap=L, seq_lens=[L],
                        heavy_fn=lambda rng, b, h, L: _random_blocks(rng, L, BLOCK, DEFAULT_N_LOCAL,
                                                                      round(0.02 * (L // BLOCK))),
                        deltas=(5.0,))
    if n == 3:
        L = 131072

        def heavy3(rng, b, h, L):
            f = rng.uniform(0.005, 0.05)
            return _random_blocks(rng, L, BLOCK, DEFAULT_N_LOCAL, round(f * (L // BLOCK)))
        return generate(name=name, seed=seed, B=4, Hq=32, Hkv=8, Lcap=L, seq_lens=[L] * 4,
                        heavy_fn=heavy3, deltas=(3.0, 5.0, 7.0))
    if n == 4:
        L = 262144
        sizes = (6, 5, 5, 5, 5, 5, 5, 5)
        return generate(name=name, seed=seed, B=1, Hq=32, Hkv=8, Lcap=L, seq_lens=[L],
                        heavy_fn=lambda rng, b, h, L: _clustered_blocks(rng, L, BLOCK, 512, sizes),
                        recent_tokens=512, deltas=(5.0,))
    if n == 5:
        Lcap, B = 131072, 16
        rng = np.random.default_rng(seed)
        lens = rng.integers(8192, 131072, size=B, endpoint=True)   # drawn before q

        def heavy5(rng, b, h, L):
            if b % 2:
                return []
            return _random_blocks(rng, L, BLOCK, DEFAULT_N_LOCAL, round(0.01 * (L // BLOCK)))
        return generate(name=name, seed=seed, B=B, Hq=32, Hkv=8, Lcap=Lcap, seq_lens=lens,
                        heavy_fn=heavy5, sink_fn=lambda b: b % 2 == 0, deltas=(5.0,), rng=rng)
    raise KeyError(n)


def context_case(L: int, seed: int | None = None) -> Case:
    """Workload 2's layout (B = 1, 32 q / 8 KV heads, 2% heavy blocks + sink) at context length L,
    for the context-length sweep (4K .. 256K)."""
    if L <= 0 or L % BLOCK:
        raise ValueError("L must be a positive multiple of 64")
    seed = 2000 + L // 1024 if seed is None else seed
    return generate(name=f"ctx-sweep-{L // 1024}k-b1-32q8kv", seed=seed, B=1, Hq=32, Hkv=8, Lcap=L,
                    seq_lens=[L],
                    heavy_fn=lambda rng, b, h, L: _random_blocks(rng, L, BLOCK, DEFAULT_N_LOCAL,
                                                                  round(0.02 * (L // BLOCK))),
                    deltas=(5.0,))


def small_case(*, seed, B=1, Hq=8, Hkv=2, seq_lens=(1000,), Lcap=None, heavy_frac=0.03,
               sink=True, recent_tokens=0, n_sink=DEFAULT_N_SINK, n_local=DEFAULT_N_LOCAL,
               deltas=(5.0,), name="small") -> Case:
    """A small case with the same recipe, for parity tests (ragged tails, odd lengths, GQA ratios)."""
    seq_lens = list(seq_lens)
    if Lcap is None:
        Lcap = max(BLOCK, -(-max(seq_lens) // BLOCK) * BLOCK)

    def heavy(rng, b, h, L):
        return _random_blocks(rng, L, BLOCK, n_local, round(heavy_frac * (L // BLOCK)))
    return generate(name=name, seed=seed, B=B, Hq=Hq, Hkv=Hkv, Lcap=Lcap, seq_lens=seq_lens,
                    heavy_fn=heavy, sink_fn=lambda b: sink, recent_tokens=recent_tokens,
                    n_sink=n_sink, n_local=n_local, deltas=deltas)
