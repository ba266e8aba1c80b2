"""ffd_quantize_keys on the GPU: bit-exact against the oracle's decomposition and packing."""
import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import Uploaded, bits_to_bf16

pytestmark = pytest.mark.gpu


def _gpu_quantize(k_bits, t_begin=0, t_end=None, fill=None, bits=2):
    from paper_2609_00097_amd import ffd
    k = bits_to_bf16(k_bits)
    B, Hkv, Lcap, _ = k.shape
    codes, absmax, resid = ffd.empty_quantized(B, Hkv, Lcap, "cuda", bits)
    for t in (codes, absmax, resid):
        t.view(torch.uint8).fill_(0 if fill is None else fill)
    ffd.quantize_keys(k, t_begin, t_end, out=(codes, absmax, resid))
    torch.cuda.synchronize()
    return (codes.cpu().numpy().view(np.uint32), absmax.cpu().view(torch.int16).numpy().view(np.uint16),
            resid.cpu().numpy())


def _assert_equal_packed(gpu, ref, name):
    for g, r, what in zip(gpu, ref, ("codes", "absmax", "resid")):
        assert np.array_equal(g, r), f"{name}: {what} differ at {np.argwhere(g != r)[:5].tolist()}"


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_workload1_bit_exact(bits):
    c = I.workload(1)
    print(f"case {c.name} seed {c.seed} bits {bits}", flush=True)
    _assert_equal_packed(_gpu_quantize(c.k, bits=bits), O.quantize_cache(c.k, bits=bits), c.name)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_ragged_small_batch_bit_exact(bits):
    c = I.small_case(seed=7, B=3, Hq=8, Hkv=4, seq_lens=(100, 257, 64), Lcap=320)
    _assert_equal_packed(_gpu_quantize(c.k, bits=bits), O.quantize_cache(c.k, bits=bits), "small")


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("M", [1.5, 3.140625, 0.0078125, 117.0, 1.0e-30, 2.0e30, 3.0e38, 1.0e-38])
def test_every_bf16_value_against_an_absmax(M, bits):
    """All finite bf16 values x with |x| <= M, 127 per token next to the absmax M (App. A edges;
    the bin edges of the 4- and 8-bit codebooks; absmaxes near the top and bottom of the range)."""
    Mb = O.bf16_to_f64(O.f64_to_bf16_bits(np.array([M])))[0]
    x = O.bf16_to_f64(np.arange(65536, dtype=np.uint32).astype(np.uint16))
    x = x[np.isfinite(x) & (np.abs(x) <= Mb)]
    ntok = -(-x.size // 127)
    Lcap = -(-ntok // 64) * 64
    vals = np.zeros((Lcap, 128))
    vals[:, 0] = Mb
    flat = np.zeros(Lcap * 127)
    flat[:x.size] = x
    vals[:, 1:] = flat.reshape(Lcap, 127)
    vals[ntok:] = 0.0                               # zero tokens: M = 0 case
    vals[1::2, 0] = -Mb                             # the absmax element negative on odd tokens
    k_bits = O.f64_to_bf16_bits(vals).reshape(1, 1, Lcap, 128)
    print(f"case every-bf16 M={M} bits={bits}", flush=True)
    _assert_equal_packed(_gpu_quantize(k_bits, bits=bits), O.quantize_cache(k_bits, bits=bits),
                         f"M={M} bits={bits}")


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_partial_range_leaves_other_tokens_untouched(bits):
    c = I.small_case(seed=9, B=1, Hq=4, Hkv=2, seq_lens=(256,))
    got = _gpu_quantize(c.k, 70, 133, fill=0xA5, bits=bits)
    ref = O.quantize_cache(c.k, 70, 133, bits=bits)
    codes = O.unpack_codes(got[0][0, 0], 256, bits)
    ref_codes = O.unpack_codes(ref[0][0, 0], 256, bits)
    assert np.array_equal(codes[70:133], ref_codes[70:133])
    full_sentinel = np.full_like(got[0], 0xA5A5A5A5)
    untouched = O.unpack_codes(full_sentinel[0, 0], 256, bits)
    assert np.array_equal(codes[:70], untouched[:70]) and np.array_equal(codes[133:], untouched[133:])
    # a single appended token (decode-step append)
    got1 = _gpu_quantize(c.k, 200, 201, fill=0, bits=bits)
    ref1 = O.quantize_cache(c.k, 200, 201, bits=bits)
    _assert_equal_packed(got1, ref1, "append one token")
