"""Helpers shared by the GPU parity tests: upload a case, run the library, compare with the oracle."""
from __future__ import annotations

import numpy as np
import torch

from oracle import ffd_oracle as O

# Output tolerance for bf16 results: |gpu - ref| <= ATOL + RTOL * |ref| elementwise.
ATOL, RTOL = 2e-3, 1e-2
LSE_TOL = 1e-3
NEAR_BAND = 1e-3
M_TILDE_TOL = 1e-4          # the pseudo-max: one fp32 rounding of an exact integer dot product (+ residual term)


def bits_to_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class Uploaded:
    def __init__(self, case, device="cuda"):
        self.case = case
        self.q = bits_to_bf16(case.q, device)
        self.k = bits_to_bf16(case.k, device)
        self.v = bits_to_bf16(case.v, device)
        self.seq_lens = torch.from_numpy(case.seq_lens.astype(np.int32)).to(device)


def check_close(name, gpu, ref, atol=ATOL, rtol=RTOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    bad = ~(np.abs(gpu - ref) <= atol + rtol * np.abs(ref))
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{name}: {bad.sum()} of {bad.size} outside tolerance; first {idx.tolist()}: "
                             f"gpu {gpu[bad][:5]} ref {ref[bad][:5]}")


def check_lse(name, gpu, ref, tol=LSE_TOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    both_inf = np.isneginf(gpu) & np.isneginf(ref)
    diff = np.abs(np.where(both_inf, 0.0, gpu) - np.where(both_inf, 0.0, ref))
    bad = ~both_inf & ~(diff <= tol)
    assert not bad.any(), f"{name}: lse mismatch at {np.argwhere(bad)[:5].tolist()} gpu {gpu[bad][:5]} ref {ref[bad][:5]}"


def compare_ffd(case, delta, out, lse, mask, *, heads=None, n_sink=None, n_local=None, bits=2,
                pm_source="thumbnail", m_tilde=None):
    """Masks bit-exact outside the near-threshold band; outputs/lse against the oracle on the
    GPU's own mask (thumbnail depth ``bits``, pseudo-max source ``pm_source``); the GPU's pseudo-max
    ``m_tilde`` when given. Returns (number of near-threshold blocks, number of mismatches inside it)."""
    n_sink = case.n_sink if n_sink is None else n_sink
    n_local = case.n_local if n_local is None else n_local
    gmask = mask.cpu().numpy().astype(bool)
    # one oracle pass: its own selection ("keep", "sigma", "m_tilde") and its attention on the
    # GPU's mask ("out", "lse")
    ref = O.decode_batch(case.q, case.k, case.v, case.seq_lens, delta=delta, n_sink=n_sink,
                         n_local=n_local, keep=gmask, heads=heads, bits=bits, pm_source=pm_source)
    G = case.G
    pairs = heads if heads is not None else [(b, h) for b in range(case.B) for h in range(case.Hkv)]
    rows = [(b, h * G + i) for b, h in pairs for i in range(G)]
    bi = np.array([r[0] for r in rows])
    hi = np.array([r[1] for r in rows])
    near = O.near_threshold(ref["sigma"][bi, hi], ref["m_tilde"][bi, hi], delta, NEAR_BAND)
    diff = gmask[bi, hi] != ref["keep"][bi, hi]
    assert not (diff & ~near).any(), f"mask mismatch outside the near-threshold band at {np.argwhere(diff & ~near)[:5].tolist()}"
    if m_tilde is not None:
        check_lse("m_tilde", m_tilde.cpu().numpy()[bi, hi], ref["m_tilde"][bi, hi], tol=M_TILDE_TOL)
    check_close("out", bf16_to_f64(out)[bi, hi], ref["out"][bi, hi])
    if lse is not None:
        check_lse("lse", lse.cpu().numpy()[bi, hi], ref["lse"][bi, hi])
    return int(near.sum()), int((diff & near).sum())


def compare_dense(case, out, lse, *, heads=None):
    ref = O.dense_batch(case.q, case.k, case.v, case.seq_lens, heads=heads)
    G = case.G
    pairs = heads if heads is not None else [(b, h) for b in range(case.B) for h in range(case.Hkv)]
    rows = [(b, h * G + i) for b, h in pairs for i in range(G)]
    bi = np.array([r[0] for r in rows])
    hi = np.array([r[1] for r in rows])
    check_close("dense out", bf16_to_f64(out)[bi, hi], ref["out"][bi, hi])
    if lse is not None:
        check_lse("dense lse", lse.cpu().numpy()[bi, hi], ref["lse"][bi, hi])
