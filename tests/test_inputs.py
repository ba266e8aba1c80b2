"""The seeded input generator: reproducible and with the planted structure it promises."""
import numpy as np

import ffd_inputs as I


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e38], dtype=np.float32)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6
    bits = I.f32_to_bf16_bits(x)
    back = I.bf16_bits_to_f32(bits)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.015625 and back[3] == -2.5


def test_reproducible_and_seed_sensitive():
    a = I.small_case(seed=5, B=2, seq_lens=(200, 77))
    b = I.small_case(seed=5, B=2, seq_lens=(200, 77))
    c = I.small_case(seed=6, B=2, seq_lens=(200, 77))
    assert np.array_equal(a.k, b.k) and np.array_equal(a.v, b.v) and np.array_equal(a.q, b.q)
    assert not np.array_equal(a.k, c.k)


def test_workload1_structure():
    c = I.workload(1)
    assert (c.B, c.Hq, c.Hkv, c.D, c.Lcap) == (1, 8, 2, 128, 4096)
    for (b, h), blocks in c.heavy_blocks.items():
        assert len(blocks) == 2
        assert all(1 <= j and (j + 1) * 64 <= 4096 - 256 for j in blocks)
    assert c.deltas == (3.0, 5.0, 7.0)


def test_poison_beyond_length():
    c = I.small_case(seed=1, B=1, seq_lens=(100,), Lcap=192)
    v = I.bf16_bits_to_f32(c.v[0, 0])
    assert np.all(v[100:] == I.POISON_VALUE)
    assert not np.any(v[:100] == I.POISON_VALUE)


def test_clustered_blocks_are_contiguous_and_disjoint():
    rng = np.random.default_rng(0)
    sizes = (6, 5, 5, 5, 5, 5, 5, 5)
    for _ in range(20):
        blocks = I._clustered_blocks(rng, 262144, 64, 512, sizes)
        assert len(blocks) == len(set(blocks)) == 41
        assert min(blocks) >= 1 and (max(blocks) + 1) * 64 <= 262144 - 512
        runs, cur = [], 1
        for a, b in zip(blocks[:-1], blocks[1:]):
            if b == a + 1:
                cur += 1
            else:
                runs.append(cur)
                cur = 1
        runs.append(cur)
        assert sum(runs) == 41 and len(runs) <= 8
