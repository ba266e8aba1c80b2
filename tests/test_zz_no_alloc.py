"""ffd_decode_attention_noalloc (the entry point for callers that cannot allocate) against
ffd_decode_attention on the same inputs: two calls in a row on the library's fixed scratch, the
second with a smaller input, each equal to the ordinary entry point's result bit for bit (same
kernels, same partition of the work) and within the oracle parity bar."""
import ctypes

import pytest

import ffd_inputs as I


def _run_both(c, delta):
    import torch

    from paper_2609_00097_amd import ffd
    from tests.gpu_util import Uploaded
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out = torch.empty((c.B, c.Hq, c.D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((c.B, c.Hq), dtype=torch.float32, device="cuda")
    mask = torch.empty((c.B, c.Hq, c.Lcap // 64), dtype=torch.uint8, device="cuda")
    ffd.decode_attention_noalloc(up.q, *qk, up.v, up.seq_lens, delta=delta, n_sink=c.n_sink,
                                 n_local=c.n_local, out=out, lse=lse, mask=mask)
    ref_out, ref_lse, ref_mask = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=delta,
                                                      n_sink=c.n_sink, n_local=c.n_local,
                                                      return_lse=True, return_mask=True)
    torch.cuda.synchronize()
    return out, lse, mask, ref_out, ref_lse, ref_mask


@pytest.mark.gpu
def test_noalloc_matches_the_workspace_entry_point_on_consecutive_calls():
    import torch

    from tests.gpu_util import compare_ffd
    cases = [I.small_case(seed=301, B=3, Hq=32, Hkv=8, seq_lens=(9000, 4097, 20000), heavy_frac=0.04),
             I.small_case(seed=302, B=1, Hq=8, Hkv=2, seq_lens=(1500,), heavy_frac=0.05)]
    for i, c in enumerate(cases):
        print(f"noalloc call {i}: B={c.B} Hq={c.Hq} Hkv={c.Hkv} lens={c.seq_lens.tolist()}", flush=True)
        out, lse, mask, ref_out, ref_lse, ref_mask = _run_both(c, 5.0)
        assert torch.equal(mask, ref_mask)
        assert torch.equal(out, ref_out)
        assert torch.equal(lse, ref_lse)
        compare_ffd(c, 5.0, out, lse, mask)


# ---- host-side checks (no GPU): the statuses come before any launch ------------------------------

@pytest.fixture(scope="module")
def so():
    import os

    from paper_2609_00097_amd import ffd
    if not os.path.exists(ffd.LIB_PATH):
        pytest.skip("libffd.so not built (run __graft_entry__.build())")
    return ffd.lib()


def _noalloc(so, fake, B, Hq, Hkv, Lcap, D=128, bits=2, delta=5.0, out=None):
    out = fake if out is None else out
    return so.ffd_decode_attention_noalloc(fake, fake, fake, fake, fake, fake, B, Hq, Hkv, Lcap, D, bits, 64,
                                           delta, 64, 256, 0, 0.0, out, None, None, None)


def test_noalloc_rejects_calls_beyond_its_scratch(so):
    fake = 0x1000
    assert so.ffd_workspace_bytes(64, 32, 8, 131072, 128, 0) > (16 << 20)
    assert _noalloc(so, fake, 64, 32, 8, 131072) == 5
    assert so.ffd_status_string(5) == b"FFD_ERR_SCRATCH_TOO_SMALL"


def test_noalloc_argument_checks_are_the_ordinary_ones(so):
    fake = 0x1000
    assert _noalloc(so, None, 1, 32, 8, 4096) == 1                  # null pointers
    assert _noalloc(so, fake, 1, 32, 8, 4096, D=96) == 2
    assert _noalloc(so, fake, 1, 32, 8, 4096, bits=3) == 2
    assert _noalloc(so, fake, 1, 32, 8, 4096, delta=-1.0) == 1
    assert _noalloc(so, fake, 1, 30, 8, 4096) == 1
    assert _noalloc(so, fake, 0, 32, 8, 4096) == 0                  # nothing to do
    assert _noalloc(so, fake + 2, 1, 32, 8, 4096) == 1              # misaligned


def test_noalloc_scratch_covers_the_benchmark_workloads(so):
    for B, Hq, Hkv, Lcap in ((1, 8, 2, 4096), (1, 32, 8, 32768), (4, 32, 8, 131072),
                             (1, 32, 8, 262144), (16, 32, 8, 131072)):
        assert 0 < so.ffd_workspace_bytes(B, Hq, Hkv, Lcap, 128, 0) <= (16 << 20)
