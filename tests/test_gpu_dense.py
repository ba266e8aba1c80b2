"""ffd_dense_decode_attention on the GPU against the oracle's exact dense attention."""
import numpy as np
import pytest
import torch

import ffd_inputs as I
from tests.gpu_util import Uploaded, bf16_to_f64, compare_dense

pytestmark = pytest.mark.gpu


def _dense(up, num_splits=0):
    from paper_2609_00097_amd import ffd
    out, lse = ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens, num_splits=num_splits)
    torch.cuda.synchronize()
    return out, lse


def test_workload1():
    c = I.workload(1)
    print(f"case {c.name} seed {c.seed}", flush=True)
    up = Uploaded(c)
    out, lse = _dense(up)
    compare_dense(c, out, lse)


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (8, 4), (8, 2), (16, 2)])
@pytest.mark.parametrize("lens", [(1,), (63, 64, 65), (1000, 4097)])
def test_gqa_ratios_and_ragged_lengths(Hq, Hkv, lens):
    c = I.small_case(seed=len(lens) * 100 + Hq + Hkv, B=len(lens), Hq=Hq, Hkv=Hkv, seq_lens=lens)
    print(f"case dense Hq={Hq} Hkv={Hkv} lens={lens}", flush=True)
    out, lse = _dense(Uploaded(c))
    compare_dense(c, out, lse)


def test_split_count_invariance_and_empty_sequence():
    c = I.small_case(seed=31, B=3, Hq=8, Hkv=2, seq_lens=(3000, 0, 777), Lcap=3072)
    up = Uploaded(c)
    ref_out, ref_lse = _dense(up, 1)
    for s in (2, 5, 48, 0):
        out, lse = _dense(up, s)
        np.testing.assert_allclose(bf16_to_f64(out), bf16_to_f64(ref_out), rtol=1e-2, atol=2e-3)
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse.cpu().numpy(), rtol=0, atol=1e-4)
    assert np.all(bf16_to_f64(ref_out)[1] == 0) and np.all(np.isneginf(ref_lse.cpu().numpy()[1]))
    compare_dense(c, ref_out, ref_lse)


def test_full_size_workload3_sampled():
    """128K x B=4 at the benchmark's launch configuration; oracle on sampled (b, kvh) pairs."""
    c = I.workload(3)
    print(f"case {c.name} seed {c.seed}", flush=True)
    out, lse = _dense(Uploaded(c))
    compare_dense(c, out, lse, heads=[(0, 0), (3, 7), (2, 4)])


def test_full_size_ragged_workload5_sampled():
    """The ragged batch of 16 sequences (8K..128K): workgroups are given to the sequences in
    proportion to their blocks; oracle on sampled pairs, the shortest and the longest included."""
    c = I.workload(5)
    order = np.argsort(c.seq_lens)
    heads = [(int(order[0]), 0), (int(order[-1]), 7), (int(order[len(order) // 2]), 3)]
    print(f"case {c.name} seed {c.seed} pairs {heads}", flush=True)
    out, lse = _dense(Uploaded(c))
    compare_dense(c, out, lse, heads=heads)


def test_more_sequences_than_the_balanced_mode_takes():
    """300 sequences (more than 256): equal runs per sequence instead of the balanced allocation."""
    lens = [1 + (53 * b) % 700 for b in range(300)]
    c = I.small_case(seed=37, B=300, Hq=4, Hkv=1, seq_lens=lens, Lcap=704, heavy_frac=0.0)
    print("case dense 300 sequences", flush=True)
    out, lse = _dense(Uploaded(c), 2)
    compare_dense(c, out, lse, heads=[(0, 0), (1, 0), (150, 0), (299, 0)])
