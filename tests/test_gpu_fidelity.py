"""The pseudo-max output and its refined source on the GPU (Sec. 5.2; Eq. 3 read with the 8-bit
residual), against the oracle; and the fidelity metrics of Sec. 5.1 (recall cosine, LSE error)
of the GPU's FFD output against the GPU's dense output."""
import numpy as np
import pytest
import torch

import ffd_inputs as I
from oracle import ffd_oracle as O
from tests.gpu_util import Uploaded, bf16_to_f64, compare_ffd

pytestmark = pytest.mark.gpu


def _run(up, qk, delta, pm, **kw):
    from paper_2609_00097_amd import ffd
    c = up.case
    mt = torch.full((c.B, c.Hq), float("nan"), dtype=torch.float32, device="cuda")
    out, lse, mask = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=delta, return_lse=True,
                                          return_mask=True, m_tilde=mt, pseudo_max=pm, **kw)
    torch.cuda.synchronize()
    return out, lse, mask, mt


@pytest.mark.parametrize("pm", ["thumbnail", "refined"])
@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (16, 2)])
def test_pseudo_max_sources_against_oracle(pm, Hq, Hkv):
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=131 + Hq, B=4, Hq=Hq, Hkv=Hkv, seq_lens=(5000, 1, 0, 700), heavy_frac=0.05)
    print(f"case pseudo-max {pm} Hq={Hq} Hkv={Hkv}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out, lse, mask, mt = _run(up, qk, 5.0, pm)
    near, flipped = compare_ffd(c, 5.0, out, lse, mask, pm_source=pm, m_tilde=mt)
    assert np.isneginf(mt.cpu().numpy()[2]).all()          # empty sequence
    print(f"near-threshold {near}, flipped {flipped}")


@pytest.mark.parametrize("bits", [4, 8])
def test_refined_pseudo_max_at_wider_depths(bits):
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=137 + bits, B=2, Hq=8, Hkv=2, seq_lens=(3000, 640), heavy_frac=0.05)
    print(f"case refined pseudo-max bits={bits}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k, bits=bits)
    out, lse, mask, mt = _run(up, qk, 5.0, "refined")
    compare_ffd(c, 5.0, out, lse, mask, pm_source="refined", m_tilde=mt, bits=bits)


def test_windows_off_and_tiny_windows():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=139, B=2, Hq=8, Hkv=2, seq_lens=(2500, 700), Lcap=2560)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    for n_sink, n_local in ((0, 0), (1, 1), (0, 64)):
        print(f"case refined windows {n_sink},{n_local}", flush=True)
        out, lse, mask, mt = _run(up, qk, 5.0, "refined", n_sink=n_sink, n_local=n_local)
        compare_ffd(c, 5.0, out, lse, mask, n_sink=n_sink, n_local=n_local, pm_source="refined",
                    m_tilde=mt)


def test_full_size_workload_refined_sampled():
    from paper_2609_00097_amd import ffd
    c = I.workload(3)
    heads = [(1, 2), (2, 6)]
    print(f"case {c.name} refined pseudo-max pairs {heads}", flush=True)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    out, lse, mask, mt = _run(up, qk, 5.0, "refined")
    near, flipped = compare_ffd(c, 5.0, out, lse, mask, heads=heads, pm_source="refined", m_tilde=mt)
    print(f"near-threshold {near}, flipped {flipped}")


def test_fidelity_of_gpu_outputs_against_gpu_dense():
    """Sec. 5.1 metrics on the GPU outputs: at delta = inf the recall is that of the 2+8
    reconstruction and the LSE error below its score-error bound; lse grows with delta."""
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=149, B=2, Hq=8, Hkv=2, seq_lens=(4000, 1500), heavy_frac=0.05)
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    dout, dlse = ffd.dense_decode_attention(up.q, up.k, up.v, up.seq_lens)
    prev = None
    for delta in (1.0, 3.0, 5.0, 7.0, float("inf")):
        out, lse, _ = ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=delta)
        torch.cuda.synchronize()
        rec = O.recall_cosine(bf16_to_f64(out), bf16_to_f64(dout))
        err = O.lse_abs_error(lse.cpu().numpy(), dlse.cpu().numpy())
        print(f"delta {delta}: recall min {rec.min():.6f} mean {rec.mean():.6f}; lse err max {err.max():.5f}")
        if prev is not None:
            assert np.all(lse.cpu().numpy() >= prev - 1e-4)
        prev = lse.cpu().numpy()
    assert rec.min() > 0.999 and err.max() < 0.02


def test_bad_pseudo_max_source():
    from paper_2609_00097_amd import ffd
    c = I.small_case(seed=1, B=1, Hq=8, Hkv=2, seq_lens=(100,))
    up = Uploaded(c)
    qk = ffd.quantize_keys(up.k)
    with pytest.raises(ValueError):
        ffd.decode_attention(up.q, *qk, up.v, up.seq_lens, delta=5.0, pseudo_max="exact")
