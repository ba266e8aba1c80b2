"""The decode step captured in a HIP graph: every replay equals the eager call.

Replays are interleaved with eager work on the same workspace (another decode with a different
delta, the dense kernel) and host synchronisations, so a replay must not depend on anything an
earlier replay or eager call left behind.
"""
import pytest
import torch

import ffd_inputs as I
from tests.gpu_util import Uploaded, compare_ffd

pytestmark = pytest.mark.gpu


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


@pytest.mark.parametrize("kernels,num_splits", [("fused", 0), ("fused", 4), ("split", 0)])
@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (16, 2)])
def test_graph_replays_equal_eager(Hq, Hkv, kernels, num_splits):
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=71 + Hq, B=2, Hq=Hq, Hkv=Hkv, seq_lens=(5000, 1700), heavy_frac=0.05)
    print(f"case graph Hq={Hq} Hkv={Hkv} kernels {kernels} splits {num_splits}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    ws = ffd.new_workspace(c.B, c.Hq, c.Hkv, c.Lcap, num_splits, "cuda")
    kw = dict(kernels=kernels, num_splits=num_splits)
    ref_out, ref_lse, ref_mask = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0,
                                                      return_mask=True, workspace=ws, **kw)
    dref_out, dref_lse = ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens, workspace=ws,
                                                    num_splits=num_splits)
    torch.cuda.synchronize()
    compare_ffd(c, 5.0, ref_out, ref_lse, ref_mask)

    out = torch.empty_like(ref_out)
    lse = torch.empty_like(ref_lse)
    dout = torch.empty_like(dref_out)
    dlse = torch.empty_like(dref_lse)
    g = _capture(lambda: ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, workspace=ws,
                                              out=out, lse=lse, **kw))
    gd = _capture(lambda: ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens, workspace=ws,
                                                     out=dout, lse=dlse, num_splits=num_splits))
    other_out = torch.empty_like(ref_out)
    for i in range(3):
        out.fill_(float("nan"))
        dout.fill_(float("nan"))
        g.replay()
        # eager work on the same workspace between replays
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=3.0 + i, workspace=ws, out=other_out,
                             kernels="split" if kernels == "fused" else "fused", num_splits=num_splits)
        gd.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse), f"replay {i}"
        assert torch.equal(dout, dref_out) and torch.equal(dlse, dref_lse), f"dense replay {i}"
