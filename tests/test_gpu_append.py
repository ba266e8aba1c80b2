"""ffd_append_kv on the GPU: one decode token per sequence appended at its device-side length.

After T appends the bf16 caches hold the appended rows, the quantized cache equals the oracle's
quantization (Sec. 3.1; App. A) of the grown cache bit for bit, and the lengths have advanced
(sequences at capacity unchanged). A captured [append, decode] graph replayed step by step gives
the same results as the eager calls, and the last step's attention matches the oracle.
"""
import dataclasses

import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import bits_to_bf16, compare_ffd

pytestmark = pytest.mark.gpu


def _start(seed, B, Hq, Hkv, L0, Lcap):
    """A case whose first L0[b] tokens are cached; rows from L0[b] on are the tokens to append."""
    c = I.small_case(seed=seed, B=B, Hq=Hq, Hkv=Hkv, seq_lens=tuple(min(L + 64, Lcap) for L in L0),
                     Lcap=Lcap, heavy_frac=0.05)
    k0, v0 = c.k.copy(), c.v.copy()
    for b, L in enumerate(L0):
        k0[b, :, L:] = 0
        v0[b, :, L:] = 0
    return c, k0, v0


def _oracle_quantized(k_bits):
    codes, absmax, resid = O.quantize_cache(k_bits)
    return codes.view(np.int32), absmax, resid


@pytest.mark.parametrize("Hkv", [2, 8, 20])
def test_appended_tokens_match_oracle_quantization(Hkv):
    from paper_2609_00097_amd import ffd
    L0, Lcap, T = (0, 500, 1087, 1088), 1088, 5
    c, k0, v0 = _start(83 + Hkv, 4, Hkv, Hkv, L0, Lcap)
    print(f"case append Hkv={Hkv} L0={L0} Lcap={Lcap} T={T}", flush=True)
    k_cache, v_cache = bits_to_bf16(k0), bits_to_bf16(v0)
    qk = ffd.quantize_keys(k_cache)
    lens = torch.tensor(L0, dtype=torch.int32, device="cuda")
    kfull, vfull = bits_to_bf16(c.k), bits_to_bf16(c.v)
    for i in range(T):
        pos = [min(L + i, Lcap - 1) for L in L0]
        k_new = torch.stack([kfull[b, :, p] for b, p in enumerate(pos)]).contiguous()
        v_new = torch.stack([vfull[b, :, p] for b, p in enumerate(pos)]).contiguous()
        ffd.append_kv(k_new, v_new, qk, lens, k_cache=k_cache, v_cache=v_cache)
    torch.cuda.synchronize()

    want_lens = [min(L + T, Lcap) for L in L0]
    assert lens.cpu().tolist() == want_lens
    k_want, v_want = k0.copy(), v0.copy()
    for b, (L, Lw) in enumerate(zip(L0, want_lens)):
        k_want[b, :, L:Lw] = c.k[b, :, L:Lw]
        v_want[b, :, L:Lw] = c.v[b, :, L:Lw]
    np.testing.assert_array_equal(k_cache.cpu().view(torch.int16).numpy().view(np.uint16), k_want)
    np.testing.assert_array_equal(v_cache.cpu().view(torch.int16).numpy().view(np.uint16), v_want)
    codes, absmax, resid = _oracle_quantized(k_want)
    np.testing.assert_array_equal(qk[0].cpu().numpy(), codes)
    np.testing.assert_array_equal(qk[1].cpu().view(torch.int16).numpy().view(np.uint16), absmax)
    np.testing.assert_array_equal(qk[2].cpu().numpy(), resid)


def test_append_without_bf16_caches_and_full_sequences():
    from paper_2609_00097_amd import ffd
    c, k0, _ = _start(89, 2, 8, 2, (64, 128), 128)
    qk = ffd.quantize_keys(bits_to_bf16(k0))
    before = [t.clone() for t in qk]
    lens = torch.tensor([64, 128], dtype=torch.int32, device="cuda")
    kfull, vfull = bits_to_bf16(c.k), bits_to_bf16(c.v)
    ffd.append_kv(kfull[:, :, 64].contiguous(), vfull[:, :, 64].contiguous(), qk, lens)
    torch.cuda.synchronize()
    assert lens.cpu().tolist() == [65, 128]          # the full sequence is left unchanged
    k_want = k0.copy()
    k_want[0, :, 64] = c.k[0, :, 64]
    codes, absmax, resid = _oracle_quantized(k_want)
    np.testing.assert_array_equal(qk[0].cpu().numpy(), codes)
    np.testing.assert_array_equal(qk[2].cpu().numpy(), resid)
    # sequence 1 untouched
    assert torch.equal(qk[0][1], before[0][1]) and torch.equal(qk[2][1], before[2][1])


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_of_append_and_decode_replays_as_the_cache_grows():
    """One capture; each replay appends the next token (whose key and value a host copy puts in
    the graph's input buffers) and attends over the grown cache; compared with the eager calls on a
    second copy of the state, and the last step with the oracle."""
    from paper_2609_00097_amd import ffd
    L0, Lcap, T = (1000, 2900), 3008, 4
    c, k0, v0 = _start(97, 2, 8, 2, L0, Lcap)
    kfull, vfull = bits_to_bf16(c.k), bits_to_bf16(c.v)
    q = bits_to_bf16(c.q)

    def state():
        kc, vc = bits_to_bf16(k0), bits_to_bf16(v0)
        return kc, vc, ffd.quantize_keys(kc), torch.tensor(L0, dtype=torch.int32, device="cuda")

    kc_g, vc_g, qk_g, lens_g = state()
    kc_e, vc_e, qk_e, lens_e = state()
    k_new = torch.empty((c.B, c.Hkv, 128), dtype=torch.bfloat16, device="cuda")
    v_new = torch.empty_like(k_new)
    ws_g = ffd.new_workspace(c.B, c.Hq, c.Hkv, Lcap, 0, "cuda")
    out_g = torch.empty((c.B, c.Hq, 128), dtype=torch.bfloat16, device="cuda")
    lse_g = torch.empty((c.B, c.Hq), dtype=torch.float32, device="cuda")

    def step():
        ffd.append_kv(k_new, v_new, qk_g, lens_g, k_cache=kc_g, v_cache=vc_g)
        ffd.decode_attention(q, *qk_g, vc_g, lens_g, delta=5.0, workspace=ws_g, out=out_g, lse=lse_g)

    # the capture's warm-up call appends a token too: run it on a scratch copy of the state
    saved = (kc_g.clone(), vc_g.clone(), [t.clone() for t in qk_g], lens_g.clone())
    k_new.copy_(kfull[:, :, 0])
    v_new.copy_(vfull[:, :, 0])
    g = _capture(step)
    kc_g.copy_(saved[0]); vc_g.copy_(saved[1]); lens_g.copy_(saved[3])
    for t, s in zip(qk_g, saved[2]):
        t.copy_(s)
    torch.cuda.synchronize()

    for i in range(T):
        k_new.copy_(torch.stack([kfull[b, :, L + i] for b, L in enumerate(L0)]))
        v_new.copy_(torch.stack([vfull[b, :, L + i] for b, L in enumerate(L0)]))
        g.replay()
        ffd.append_kv(k_new, v_new, qk_e, lens_e, k_cache=kc_e, v_cache=vc_e)
        out_e, lse_e, _ = ffd.decode_attention(q, *qk_e, vc_e, lens_e, delta=5.0)
        torch.cuda.synchronize()
        assert lens_g.cpu().tolist() == [L + i + 1 for L in L0]
        assert torch.equal(out_g, out_e) and torch.equal(lse_g, lse_e), f"step {i}"

    final = dataclasses.replace(c, k=kc_g.cpu().view(torch.int16).numpy().view(np.uint16),
                                v=vc_g.cpu().view(torch.int16).numpy().view(np.uint16),
                                seq_lens=lens_g.cpu().numpy().astype(np.int32))
    _, _, mask = ffd.decode_attention(q, *qk_g, vc_g, lens_g, delta=5.0, return_mask=True)
    torch.cuda.synchronize()
    compare_ffd(final, 5.0, out_g, lse_g, mask)
