"""ffd_decode_attention on the GPU: block masks and outputs against the oracle (Alg. 1; Eq. 1-4).

Masks must be bit-exact except blocks whose score lies within 1e-3 of the threshold (counted and
printed); outputs and lse are compared with the oracle's attention on the GPU's own mask.
"""
import functools
import warnings

import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import Uploaded, bf16_to_f64, check_close, check_lse, compare_ffd

pytestmark = pytest.mark.gpu


class NearThresholdReport(UserWarning):
    """Near-threshold block counts of the full-size parity cases, shown in pytest's warnings summary."""


def _quant(up):
    from paper_2609_00097_amd import ffd
    return ffd.quantize_keys(up.k)


KERNELS = ["fused", "split"]


def _ffd(up, qk, delta, n_sink=None, n_local=None, num_splits=0, kernels="auto"):
    from paper_2609_00097_amd import ffd
    c = up.case
    out, lse, mask = ffd.decode_attention(
        up.q, *qk, up.v, up.seq_lens, delta=delta,
        n_sink=c.n_sink if n_sink is None else n_sink, n_local=c.n_local if n_local is None else n_local,
        num_splits=num_splits, return_lse=True, return_mask=True, kernels=kernels)
    torch.cuda.synchronize()
    return out, lse, mask


@pytest.mark.parametrize("kernels", KERNELS)
@pytest.mark.parametrize("delta", [3.0, 5.0, 7.0])
def test_workload1_delta_sweep(delta, kernels):
    c = I.workload(1)
    print(f"case {c.name} seed {c.seed} delta {delta} kernels {kernels}", flush=True)
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), delta, kernels=kernels)
    near, flipped = compare_ffd(c, delta, out, lse, mask)
    print(f"near-threshold blocks {near}, flipped among them {flipped}; kept {int(mask.sum())}")


@pytest.mark.parametrize("kernels", KERNELS)
def test_workload2(kernels):
    c = I.workload(2)
    print(f"case {c.name} seed {c.seed} kernels {kernels}", flush=True)
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), 5.0, kernels=kernels)
    near, flipped = compare_ffd(c, 5.0, out, lse, mask)
    print(f"near-threshold blocks {near}, flipped {flipped}; kept {int(mask.sum())}")


@pytest.mark.parametrize("kernels", KERNELS)
@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 4), (8, 2), (16, 2)])
@pytest.mark.parametrize("lens", [(1,), (63, 64, 65), (320, 1000, 4097)])
def test_gqa_ratios_and_ragged_lengths(Hq, Hkv, lens, kernels):
    c = I.small_case(seed=7 * len(lens) + Hq + 3 * Hkv, B=len(lens), Hq=Hq, Hkv=Hkv, seq_lens=lens)
    print(f"case ffd Hq={Hq} Hkv={Hkv} lens={lens} kernels {kernels}", flush=True)
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), 5.0, kernels=kernels)
    compare_ffd(c, 5.0, out, lse, mask)


@pytest.mark.parametrize("kernels", KERNELS)
@pytest.mark.parametrize("n_sink,n_local", [(0, 0), (0, 64), (64, 0), (1, 1), (5000, 10)])
def test_window_sizes(n_sink, n_local, kernels):
    c = I.small_case(seed=41, B=2, Hq=8, Hkv=2, seq_lens=(2500, 700), Lcap=2560)
    print(f"case windows {n_sink},{n_local} kernels {kernels}", flush=True)
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), 5.0, n_sink, n_local, kernels=kernels)
    compare_ffd(c, 5.0, out, lse, mask, n_sink=n_sink, n_local=n_local)
    if n_sink == 0 and n_local == 0:
        assert mask.cpu().numpy()[0, :, :40].all()    # m~ = -inf keeps every block


@pytest.mark.parametrize("kernels", KERNELS)
def test_delta_zero_and_infinite(kernels):
    c = I.small_case(seed=43, B=2, Hq=8, Hkv=2, seq_lens=(1500, 4000))
    up = Uploaded(c)
    qk = _quant(up)
    out0, lse0, mask0 = _ffd(up, qk, 0.0, kernels=kernels)
    compare_ffd(c, 0.0, out0, lse0, mask0)
    outi, lsei, maski = _ffd(up, qk, float("inf"), kernels=kernels)
    m = maski.cpu().numpy()
    for b, L in enumerate(c.seq_lens):
        nb = -(-int(L) // 64)
        assert m[b, :, :nb].all() and not m[b, :, nb:].any()
    # delta = inf is dense attention on the 2+8 reconstruction (pinned in the oracle tests)
    compare_ffd(c, float("inf"), outi, lsei, maski)


@pytest.mark.parametrize("kernels,num_splits", [("fused", 0), ("fused", 3), ("split", 0)])
def test_zero_keys_and_short_sequences(kernels, num_splits):
    """All-zero key tokens (M = 0), sequences shorter than the windows, and an empty sequence."""
    c = I.small_case(seed=47, B=4, Hq=8, Hkv=2, seq_lens=(300, 1, 0, 129), Lcap=320)
    c.k[0, :, 10:80] = 0
    c.k[3, 1, :] = 0
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), 5.0, num_splits=num_splits, kernels=kernels)
    compare_ffd(c, 5.0, out, lse, mask)
    o = bf16_to_f64(out)
    assert np.all(o[2] == 0) and np.all(np.isneginf(lse.cpu().numpy()[2]))
    assert not mask.cpu().numpy()[2].any()


@pytest.mark.parametrize("kernels", KERNELS)
def test_zero_queries(kernels):
    """All-zero queries: every score is 0, so m~ = 0, every block ties it and is kept, and the output
    is the mean of the values. Two heads of sequence 0 and every head of sequence 1 are zero."""
    c = I.small_case(seed=79, B=2, Hq=8, Hkv=2, seq_lens=(700, 1500), Lcap=1536)
    c.q[0, 0:2] = 0
    c.q[1] = 0
    up = Uploaded(c)
    out, lse, mask = _ffd(up, _quant(up), 5.0, kernels=kernels)
    compare_ffd(c, 5.0, out, lse, mask)
    m = mask.cpu().numpy()
    assert m[1, :, :(1500 + 63) // 64].all() and m[0, 0:2, :(700 + 63) // 64].all()
    v = bf16_to_f64(up.v)
    o = bf16_to_f64(out)
    check_close("zero-query output", o[1], np.repeat(v[1, :, :1500].mean(axis=1), c.G, axis=0))
    assert np.allclose(lse.cpu().numpy()[1], np.log(1500.0), atol=1e-3)


def test_split_count_invariance():
    """Both kernel paths at several split counts give the same mask and, to rounding, the same
    outputs (the fused kernel with one split writes its outputs directly, without the merge)."""
    c = I.small_case(seed=53, B=2, Hq=8, Hkv=2, seq_lens=(6000, 2222), heavy_frac=0.05)
    up = Uploaded(c)
    qk = _quant(up)
    ref_out, ref_lse, ref_mask = _ffd(up, qk, 5.0, num_splits=1, kernels="split")
    for kernels, s in [("fused", 1), ("fused", 2), ("fused", 7), ("fused", 64), ("fused", 0),
                       ("split", 2), ("split", 7), ("split", 64), ("split", 0), ("auto", 0)]:
        out, lse, mask = _ffd(up, qk, 5.0, num_splits=s, kernels=kernels)
        assert torch.equal(mask, ref_mask)
        np.testing.assert_allclose(bf16_to_f64(out), bf16_to_f64(ref_out), rtol=1e-2, atol=2e-3)
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse.cpu().numpy(), rtol=0, atol=1e-4)
    compare_ffd(c, 5.0, ref_out, ref_lse, ref_mask)


def test_one_workspace_serves_repeated_and_alternating_calls():
    """One workspace reused by repeated, alternating calls gives identical results."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=61, B=2, Hq=8, Hkv=2, seq_lens=(3000, 1200), heavy_frac=0.05)
    up = Uploaded(c)
    qk = _quant(up)
    ws = ffd.new_workspace(c.B, c.Hq, c.Hkv, c.Lcap, 5, "cuda")
    ref_out, ref_lse, ref_mask = _ffd(up, qk, 5.0, num_splits=5)
    dref_out, dref_lse = ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens, num_splits=5)
    for _ in range(4):
        out, lse, _ = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, num_splits=5,
                                           workspace=ws)
        dout, dlse = ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens, num_splits=5,
                                                workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
        assert torch.equal(dout, dref_out) and torch.equal(dlse, dref_lse)


@pytest.mark.parametrize("num_splits", [0, 4])
def test_stage_events_time_the_kernels_without_changing_results(num_splits):
    """Stage events around the fused kernel and the merge (none with one split) leave the results
    unchanged; the first interval (the fused kernel) is positive, the middle one is empty."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=67, B=2, Hq=8, Hkv=2, seq_lens=(3000, 1200), heavy_frac=0.05)
    up = Uploaded(c)
    qk = _quant(up)
    ref_out, ref_lse, _ = _ffd(up, qk, 5.0, num_splits=num_splits)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in evs:
        e.record()
    out, lse, _ = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, stage_events=evs,
                                       num_splits=num_splits)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
    stages = [evs[i].elapsed_time(evs[i + 1]) for i in range(3)]
    assert stages[0] > 0 and all(t >= 0 for t in stages), stages
    if num_splits > 1:
        assert stages[2] > 0, stages
    with pytest.raises(ValueError):
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, stage_events=evs[:3])


def test_argument_errors_return_status_without_launch():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=1, B=1, Hq=8, Hkv=2, seq_lens=(100,))
    up = Uploaded(c)
    qk = _quant(up)
    with pytest.raises(ffd.FfdError) as e:
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=-1.0)
    assert e.value.status == 1
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(ffd.FfdError) as e:
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, workspace=ws)
    assert e.value.status == 3


@functools.lru_cache(maxsize=1)
def _workload(wl):
    return I.workload(wl)


def _largest_planted(c, n):
    """The n (sequence, KV head) pairs with the most planted heavy blocks: the largest unions of
    kept blocks, chosen from the generator's structure (not from any GPU output)."""
    return sorted(c.heavy_blocks, key=lambda bh: (-len(c.heavy_blocks[bh]), bh))[:n]


def _full_size(wl, delta, heads, kernels="auto"):
    c = _workload(wl)
    heads = heads(c) if callable(heads) else heads
    print(f"case {c.name} seed {c.seed} delta {delta} pairs {heads} kernels {kernels}", flush=True)
    up = Uploaded(c)
    qk = _quant(up)
    out, lse, mask = _ffd(up, qk, delta, kernels=kernels)
    near, flipped = compare_ffd(c, delta, out, lse, mask, heads=heads)
    keep = mask.cpu().numpy()
    G = c.G
    union = [keep[b, h * G:(h + 1) * G].any(axis=0).mean() for b, h in heads]
    msg = (f"{c.name} delta {delta} kernels {kernels}: near-threshold blocks {near}, flipped {flipped}; "
           f"kept head-blocks {keep.mean():.4f}; union keep of the checked pairs "
           f"{[round(float(u), 4) for u in union]}")
    print(msg, flush=True)
    warnings.warn(msg, NearThresholdReport)
    # no head anywhere ends with an empty selection (the pseudo-max's own block always passes)
    for b, L in enumerate(c.seq_lens):
        if L > 0:
            assert keep[b].any(axis=-1).all()


@pytest.mark.parametrize("wl,delta,heads,kernels", [
    (3, 5.0, [(0, 0), (1, 3), (3, 7)], "auto"),
    (3, 3.0, lambda c: _largest_planted(c, 3) + [(2, 4)], "auto"),
    (3, 7.0, lambda c: _largest_planted(c, 3) + [(1, 1)], "auto"),
    (3, 5.0, lambda c: _largest_planted(c, 2) + [(0, 3)], "fused"),
    (4, 5.0, [(0, h) for h in range(8)], "auto"),
    (4, 5.0, [(0, 1), (0, 6)], "split"),
    (5, 5.0, [(0, 0), (1, 2), (6, 5), (15, 7)], "auto"),
    (5, 5.0, [(1, 0), (8, 4)], "fused"),
], ids=["wl3-d5", "wl3-d3", "wl3-d7", "wl3-d5-fused", "wl4-d5-all-heads", "wl4-d5-split", "wl5-d5",
        "wl5-d5-fused"])
def test_full_size_workloads_sampled(wl, delta, heads, kernels):
    """Workloads 3-5 at full size in the benchmark's launch configuration (automatic splits);
    masks and outputs against the oracle on sampled (sequence, KV head) pairs: at workload 3 for
    each delta of its sweep (for 3 and 7 on the pairs with the most planted blocks, whose unions
    are the largest), at workload 4 on all eight KV heads (the recent window's scores straddle
    m~ - delta there); each workload also through the kernels the automatic choice does not take."""
    _full_size(wl, delta, heads, kernels)


@pytest.mark.parametrize("kernels", KERNELS)
def test_maximum_capacity(kernels):
    """The library's largest cache, Lcap = 2^24 tokens: grids and workspace are sized by the capacity
    (256 scan workgroups per KV group, most with nothing to scan); two sequences in it, one ragged,
    against the oracle. Tokens past the sequences are zero and never read."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=97, B=2, Hq=4, Hkv=1, seq_lens=(3000, 70001), Lcap=70016, heavy_frac=0.03)
    print("case maximum capacity Lcap=2^24", flush=True)
    up = Uploaded(c)
    cap = 1 << 24
    k = torch.zeros((c.B, c.Hkv, cap, 128), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    k[:, :, :c.Lcap] = up.k
    v[:, :, :c.Lcap] = up.v
    qk = ffd.quantize_keys(k)
    out, lse, mask = ffd.decode_attention(up.q, *qk, v, up.seq_lens, delta=5.0, return_lse=True,
                                          return_mask=True, kernels=kernels)
    torch.cuda.synchronize()
    nb = c.Lcap // 64
    assert not mask[:, :, nb:].any()
    near, flipped = compare_ffd(c, 5.0, out, lse, mask[:, :, :nb].contiguous())
    print(f"near-threshold blocks {near}, flipped {flipped}")
    dense_out, dense_lse = ffd.dense_decode_attention(up.q, k, v, up.seq_lens)
    torch.cuda.synchronize()
    from tests.gpu_util import compare_dense
    compare_dense(c, dense_out, dense_lse)


def test_allocation_for_more_than_1024_kv_groups():
    """More than 1024 (sequence, KV head) groups: the refinement sums the scan counts per group in
    passes with LDS atomics instead of its per-wave allocation; outputs against the oracle."""
    lens = [1 + (37 * b) % 64 for b in range(1030)]
    c = I.small_case(seed=61, B=1030, Hq=1, Hkv=1, seq_lens=lens, Lcap=64, heavy_frac=0.0)
    print("case 1030 groups of one block", flush=True)
    up = Uploaded(c)
    qk = _quant(up)
    out, lse, mask = _ffd(up, qk, 5.0, kernels="split")
    compare_ffd(c, 5.0, out, lse, mask)
    out, lse, mask = _ffd(up, qk, 5.0, kernels="fused")
    compare_ffd(c, 5.0, out, lse, mask)


@pytest.mark.parametrize("B", [200, 300])
def test_allocation_fills_the_grid_with_many_groups(B):
    """Many KV groups and one refinement split (W <= 2 B*Hkv): the allocation grows its effective W
    until the grid is full, in the per-wave allocation (200 groups) and in the LDS-cached one (300
    groups); ragged lengths, empty sequences among them, both through the oracle."""
    from paper_2609_00097_amd import ffd
    lens = [0 if b % 37 == 5 else 1 + (97 * b) % 2000 for b in range(B)]
    c = I.small_case(seed=71 + B, B=B, Hq=4, Hkv=1, seq_lens=lens, Lcap=2048, heavy_frac=0.03)
    assert ffd.resolve_splits(B, 1, 2048, 0) == 1
    print(f"case {B} groups, one refinement split", flush=True)
    up = Uploaded(c)
    qk = _quant(up)
    out, lse, mask = _ffd(up, qk, 5.0, kernels="split")
    compare_ffd(c, 5.0, out, lse, mask)


def test_share_longer_than_the_per_wave_staging():
    """One split: a single refinement workgroup refines all 1094 kept blocks of the group, staged in
    two chunks with workgroup barriers (shares of up to 256 blocks are staged by each wave alone)."""
    c = I.small_case(seed=62, B=1, Hq=4, Hkv=1, seq_lens=(70000,), heavy_frac=0.02)
    print("case one workgroup, 1094 kept blocks", flush=True)
    up = Uploaded(c)
    qk = _quant(up)
    out, lse, mask = _ffd(up, qk, float("inf"), num_splits=1, kernels="split")
    assert mask.cpu().numpy()[:, :, :1094].all()
    compare_ffd(c, float("inf"), out, lse, mask)
