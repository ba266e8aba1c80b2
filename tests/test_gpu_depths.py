"""The 4+8 and 8+8 thumbnail depths (App. C) on the GPU: the scan and selection read 4- and 8-bit
codes, the refinement the same 8-bit residual on the finer step; masks, outputs and lse against the
oracle at the same depth, and the decode-step append writes the oracle's quantization bit for bit."""
import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import Uploaded, bf16_to_f64, bits_to_bf16, compare_ffd

pytestmark = pytest.mark.gpu
WIDE = [4, 8]


def _run(c, bits, delta, **kw):
    from paper_2609_00097_amd import ffd
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k, bits=bits)
    out, lse, mask = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=delta, return_lse=True,
                                          return_mask=True, **kw)
    torch.cuda.synchronize()
    return out, lse, mask


@pytest.mark.parametrize("bits", WIDE)
@pytest.mark.parametrize("delta", [3.0, 5.0])
def test_workload1(bits, delta):
    c = I.workload(1)
    print(f"case {c.name} seed {c.seed} bits {bits} delta {delta}", flush=True)
    out, lse, mask = _run(c, bits, delta)
    near, flipped = compare_ffd(c, delta, out, lse, mask, bits=bits)
    print(f"near-threshold blocks {near}, flipped {flipped}; kept {int(mask.sum())}")


@pytest.mark.parametrize("bits", WIDE)
@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (16, 2)])
def test_gqa_ratios_and_ragged_lengths(bits, Hq, Hkv):
    lens = (1, 63, 65, 4097)
    c = I.small_case(seed=101 + Hq + bits, B=len(lens), Hq=Hq, Hkv=Hkv, seq_lens=lens)
    print(f"case depths bits={bits} Hq={Hq} Hkv={Hkv} lens={lens}", flush=True)
    out, lse, mask = _run(c, bits, 5.0)
    compare_ffd(c, 5.0, out, lse, mask, bits=bits)


@pytest.mark.parametrize("bits", WIDE)
def test_zero_keys_short_sequences_and_infinite_delta(bits):
    c = I.small_case(seed=107, B=4, Hq=8, Hkv=2, seq_lens=(300, 1, 0, 129), Lcap=320)
    c.k[0, :, 10:80] = 0
    c.k[3, 1, :] = 0
    print(f"case depths zero keys bits={bits}", flush=True)
    out, lse, mask = _run(c, bits, 5.0)
    compare_ffd(c, 5.0, out, lse, mask, bits=bits)
    assert np.all(bf16_to_f64(out)[2] == 0) and np.all(np.isneginf(lse.cpu().numpy()[2]))
    out, lse, mask = _run(c, bits, float("inf"))
    compare_ffd(c, float("inf"), out, lse, mask, bits=bits)


@pytest.mark.parametrize("bits", WIDE)
def test_full_size_benchmark_workload_sampled(bits):
    """4 sequences of 128K tokens, 32 query / 8 KV heads, in the benchmark's launch configuration;
    sampled (sequence, KV head) pairs against the oracle."""
    c = I.workload(3)
    heads = [(0, 0), (3, 7)]
    print(f"case {c.name} seed {c.seed} bits {bits} pairs {heads}", flush=True)
    out, lse, mask = _run(c, bits, 5.0)
    near, flipped = compare_ffd(c, 5.0, out, lse, mask, heads=heads, bits=bits)
    print(f"near-threshold blocks {near}, flipped {flipped}; kept fraction {mask.float().mean().item():.4f}")


@pytest.mark.parametrize("bits", WIDE)
def test_append_matches_oracle_quantization(bits):
    from paper_2609_00097_amd import ffd
    L0, Lcap, T = (0, 500, 1087, 1088), 1088, 3
    c = I.small_case(seed=113 + bits, B=4, Hq=8, Hkv=8, seq_lens=(64, 564, 1088, 1088), Lcap=Lcap)
    k0 = c.k.copy()
    for b, L in enumerate(L0):
        k0[b, :, L:] = 0
    print(f"case depths append bits={bits}", flush=True)
    k_cache, v_cache = bits_to_bf16(k0), bits_to_bf16(c.v)
    qk = ffd.quantize_keys(k_cache, bits=bits)
    lens = torch.tensor(L0, dtype=torch.int32, device="cuda")
    kfull, vfull = bits_to_bf16(c.k), bits_to_bf16(c.v)
    for i in range(T):
        pos = [min(L + i, Lcap - 1) for L in L0]
        k_new = torch.stack([kfull[b, :, p] for b, p in enumerate(pos)]).contiguous()
        v_new = torch.stack([vfull[b, :, p] for b, p in enumerate(pos)]).contiguous()
        ffd.append_kv(k_new, v_new, qk, lens, k_cache=k_cache)
    torch.cuda.synchronize()
    want_lens = [min(L + T, Lcap) for L in L0]
    assert lens.cpu().tolist() == want_lens
    k_want = k0.copy()
    for b, (L, Lw) in enumerate(zip(L0, want_lens)):
        k_want[b, :, L:Lw] = c.k[b, :, L:Lw]
    codes, absmax, resid = O.quantize_cache(k_want, bits=bits)
    np.testing.assert_array_equal(qk[0].cpu().numpy().view(np.uint32), codes)
    np.testing.assert_array_equal(qk[1].cpu().view(torch.int16).numpy().view(np.uint16), absmax)
    np.testing.assert_array_equal(qk[2].cpu().numpy(), resid)


def test_codes_shape_names_the_depth():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=5, B=1, Hq=8, Hkv=2, seq_lens=(100,))
    up = Uploaded(c)
    codes, absmax, resid = ffd.quantize_keys(up.k, bits=4)
    assert codes.shape[-3:] == (4, 64, 4)
    with pytest.raises(ValueError):
        ffd.decode_attention(up.q, codes[..., :3, :, :].contiguous(), absmax, resid, up.v, up.seq_lens,
                             delta=5.0)
    with pytest.raises(ValueError):
        ffd.quantize_keys(up.k, bits=3)
