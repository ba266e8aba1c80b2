"""Fixed-budget (top-k) selection on the GPU, the rule top-delta is compared with (Sec. 1, Fig. 1 (a);
Table 3): per head the k blocks with the largest thumbnail block scores, equal scores in block order.

Masks against the oracle's selection: every head keeps exactly min(k, blocks) blocks; bit-exact
except blocks whose score lies within 1e-3 of the head's k-th largest score (counted); where the
scores tie exactly, bit-exact with no band. Outputs and lse against the oracle's attention on the
GPU's own mask.
"""
import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import NEAR_BAND, Uploaded, bf16_to_f64, check_close, check_lse

pytestmark = pytest.mark.gpu


def _rows(case, heads):
    G = case.G
    pairs = heads if heads is not None else [(b, h) for b in range(case.B) for h in range(case.Hkv)]
    rows = [(b, h * G + i) for b, h in pairs for i in range(G)]
    return np.array([r[0] for r in rows]), np.array([r[1] for r in rows])


def _near_kth(sigma_row, nb, k):
    """Blocks whose score is within the band of the k-th largest of the first nb scores."""
    near = np.zeros(sigma_row.shape, dtype=bool)
    if k >= nb or nb == 0:
        return near
    kth = np.sort(sigma_row[:nb])[::-1][k - 1]
    near[:nb] = np.abs(sigma_row[:nb] - kth) < NEAR_BAND
    return near


def compare_topk(case, k, out, lse, mask, *, heads=None, bits=2, exact=False):
    """Returns (near-threshold blocks, mismatches among them)."""
    gmask = mask.cpu().numpy().astype(bool)
    ref = O.decode_batch(case.q, case.k, case.v, case.seq_lens, delta=5.0, n_sink=case.n_sink,
                         n_local=case.n_local, heads=heads, bits=bits, topk=k)
    bi, hi = _rows(case, heads)
    near_n = flipped = 0
    for b, h in zip(bi, hi):
        nb = -(-int(case.seq_lens[b]) // 64)
        assert gmask[b, h].sum() == min(k, nb), (b, h, int(gmask[b, h].sum()), min(k, nb))
        assert not gmask[b, h, nb:].any()
        diff = gmask[b, h] != ref["keep"][b, h]
        near = np.zeros_like(diff) if exact else _near_kth(ref["sigma"][b, h], nb, k)
        assert not (diff & ~near).any(), f"top-k mask mismatch at head {(b, h)} blocks {np.nonzero(diff & ~near)[0][:8]}"
        near_n += int(near.sum())
        flipped += int((diff & near).sum())
    on_mask = O.decode_batch(case.q, case.k, case.v, case.seq_lens, delta=5.0, n_sink=case.n_sink,
                             n_local=case.n_local, keep=gmask, heads=heads, bits=bits)
    check_close("out", bf16_to_f64(out)[bi, hi], on_mask["out"][bi, hi])
    if lse is not None:
        check_lse("lse", lse.cpu().numpy()[bi, hi], on_mask["lse"][bi, hi])
    return near_n, flipped


def _run(up, qk, k, **kw):
    from paper_2609_00097_amd import ffd
    out, lse, mask = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, return_lse=True,
                                          return_mask=True, top_k=k, **kw)
    torch.cuda.synchronize()
    return out, lse, mask


@pytest.mark.parametrize("k", [1, 2, 5, 17, 63, 64, 1000])
def test_workload1_budgets(k):
    from paper_2609_00097_amd import ffd
    c = I.workload(1)
    print(f"case {c.name} top-k {k}", flush=True)
    up = Uploaded(c)
    out, lse, mask = _run(up, ffd.quantize_keys(up.k), k)
    near, flipped = compare_topk(c, k, out, lse, mask)
    print(f"near-threshold blocks {near}, flipped {flipped}")


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 4), (8, 2), (16, 2)])
@pytest.mark.parametrize("lens", [(1,), (63, 64, 65), (320, 1000, 4097)])
def test_gqa_ratios_and_ragged_lengths(Hq, Hkv, lens):
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=17 * len(lens) + Hq + 5 * Hkv, B=len(lens), Hq=Hq, Hkv=Hkv, seq_lens=lens)
    print(f"case top-k Hq={Hq} Hkv={Hkv} lens={lens}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    for k in (3, 40):
        out, lse, mask = _run(up, qk, k)
        compare_topk(c, k, out, lse, mask)


@pytest.mark.parametrize("template", ["repeated", "zero", "three"])
def test_ties_go_in_block_order(template):
    """Blocks that are copies of each other score exactly alike on both sides: the first ones in block
    order are kept, bit for bit (no near-threshold allowance). All-zero keys score +-0, which tie."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=71, B=2, Hq=8, Hkv=2, seq_lens=(2048, 1280), Lcap=2048)
    rng = np.random.default_rng(5)
    for b in range(c.B):
        for h in range(c.Hkv):
            L = int(c.seq_lens[b])
            if template == "zero":
                c.k[b, h, :L] = 0
            elif template == "repeated":
                c.k[b, h, :L] = np.tile(c.k[b, h, 64:128], (L // 64, 1))
            else:
                pick = rng.integers(0, 3, L // 64)
                tpl = [c.k[b, h, 64 * (i + 1):64 * (i + 2)].copy() for i in range(3)]
                for j in range(L // 64):
                    c.k[b, h, 64 * j:64 * (j + 1)] = tpl[pick[j]]
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    for k in (1, 7, 19, 20, 32):
        print(f"case ties {template} k {k}", flush=True)
        out, lse, mask = _run(up, qk, k)
        compare_topk(c, k, out, lse, mask, exact=True)


def test_full_budget_equals_delta_infinity():
    """Keeping every block through the budget gives the mask of delta = inf bit for bit, and the same
    outputs and lse up to the rounding of a different partition of the work (the top-k path refines
    in its own kernel, top-delta in the fused one); both match the oracle's delta = inf outputs."""
    from paper_2609_00097_amd import ffd
    from tests.gpu_util import compare_ffd
    c = I.small_case(seed=73, B=3, Hq=16, Hkv=2, seq_lens=(3000, 4096, 700), heavy_frac=0.05)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out_k, lse_k, mask_k = _run(up, qk, 64)
    out_i, lse_i, mask_i = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=float("inf"),
                                                return_lse=True, return_mask=True)
    torch.cuda.synchronize()
    assert torch.equal(mask_k, mask_i)
    np.testing.assert_allclose(out_k.float().cpu().numpy(), out_i.float().cpu().numpy(), rtol=1e-2, atol=2e-3)
    np.testing.assert_allclose(lse_k.cpu().numpy(), lse_i.cpu().numpy(), rtol=0, atol=1e-4)
    compare_ffd(c, float("inf"), out_k, lse_k, mask_k)
    compare_ffd(c, float("inf"), out_i, lse_i, mask_i)


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (16, 2)])
def test_wider_thumbnails(bits, Hq, Hkv):
    """The refinement recomputes the thumbnail scores from 4- and 8-bit codes (App. C depths)."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=79 + bits + Hq, B=2, Hq=Hq, Hkv=Hkv, seq_lens=(3000, 640), heavy_frac=0.05)
    print(f"case top-k bits={bits} Hq={Hq}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k, bits=bits)
    out, lse, mask = _run(up, qk, 6)
    compare_topk(c, 6, out, lse, mask, bits=bits)


def test_split_count_and_mask_output_invariance():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=83, B=2, Hq=8, Hkv=2, seq_lens=(6000, 2222), heavy_frac=0.05)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    ref_out, ref_lse, ref_mask = _run(up, qk, 9, num_splits=1)
    for s in (3, 64, 0):
        out, lse, mask = _run(up, qk, 9, num_splits=s)
        assert torch.equal(mask, ref_mask)
        np.testing.assert_allclose(bf16_to_f64(out), bf16_to_f64(ref_out), rtol=1e-2, atol=2e-3)
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse.cpu().numpy(), rtol=0, atol=1e-4)
    out_nm, lse_nm, none = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, top_k=9)
    torch.cuda.synchronize()
    assert none is None
    out0, lse0, _ = _run(up, qk, 9)
    assert torch.equal(out_nm, out0) and torch.equal(lse_nm, lse0)
    compare_topk(c, 9, ref_out, ref_lse, ref_mask)


def test_empty_sequence_and_argument_errors():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=89, B=3, Hq=8, Hkv=2, seq_lens=(500, 0, 64), Lcap=512)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out, lse, mask = _run(up, qk, 4)
    compare_topk(c, 4, out, lse, mask)
    assert np.all(bf16_to_f64(out)[1] == 0) and np.isneginf(lse.cpu().numpy()[1]).all()
    assert not mask.cpu().numpy()[1].any()
    mt = torch.empty((c.B, c.Hq), dtype=torch.float32, device="cuda")
    with pytest.raises(ffd.FfdError) as e:
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, top_k=4, m_tilde=mt)
    assert e.value.status == 1
    with pytest.raises(ffd.FfdError) as e:
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, top_k=-2)
    assert e.value.status == 1


@pytest.mark.parametrize("wl,k,heads", [(3, 57, [(0, 0), (1, 3), (3, 7)]), (4, 41, [(0, 0), (0, 5)]),
                                        (5, 20, [(0, 0), (1, 2), (6, 5), (15, 7)])])
def test_full_size_workloads_sampled(wl, k, heads):
    """Workloads 3-5 at full size (automatic splits), a budget near top-delta's keep ratio at
    delta = 5; masks and outputs against the oracle on sampled (sequence, KV head) pairs."""
    from paper_2609_00097_amd import ffd
    c = I.workload(wl)
    print(f"case {c.name} top-k {k} pairs {heads}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out, lse, mask = _run(up, qk, k)
    near, flipped = compare_topk(c, k, out, lse, mask, heads=heads)
    keep = mask.cpu().numpy()
    for b, L in enumerate(c.seq_lens):
        nb = -(-int(L) // 64)
        assert np.all(keep[b, :, :nb].sum(-1) == min(k, nb))
    print(f"near-threshold blocks {near}, flipped {flipped}")


def test_maximum_capacity():
    """Top-k in the library's largest cache (Lcap = 2^24 tokens); at G = 8 the 70001-token sequence's
    1094 block scores per head span two of the selection kernel's 1024-block tiles."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=101, B=2, Hq=8, Hkv=1, seq_lens=(3000, 70001), Lcap=70016, heavy_frac=0.03)
    print("case top-k maximum capacity Lcap=2^24", flush=True)
    up = Uploaded(c)
    cap = 1 << 24
    k = torch.zeros((c.B, c.Hkv, cap, 128), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    k[:, :, :c.Lcap] = up.k
    v[:, :, :c.Lcap] = up.v
    qk = ffd.quantize_keys(k)
    up2 = Uploaded(c)
    up2.k, up2.v = k, v
    out, lse, mask = _run(up2, qk, 29)
    nb = c.Lcap // 64
    assert not mask[:, :, nb:].any()
    compare_topk(c, 29, out, lse, mask[:, :, :nb].contiguous())
