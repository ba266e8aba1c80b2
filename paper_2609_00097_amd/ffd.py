"""Thin Python binding of libffd.so (ctypes). Argument marshalling only: every step of the decode
path runs in the library's HIP kernels. PyTorch supplies device memory and the current stream.

If the library is not built or cannot be loaded, every call raises ``FfdLibraryError``; there is
no CPU fallback.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libffd.so")

HEAD_DIM = 128
BLOCK = 64
MAX_SPLITS = 1024
THUMB_BITS = (2, 4, 8)      # thumbnail depths: 2+8 (the method), 4+8 and 8+8 (App. C)
STATUS = {0: "FFD_OK", 1: "FFD_ERR_INVALID_ARGUMENT", 2: "FFD_ERR_UNSUPPORTED",
          3: "FFD_ERR_WORKSPACE_TOO_SMALL", 4: "FFD_ERR_HIP", 5: "FFD_ERR_SCRATCH_TOO_SMALL"}
NOALLOC_SCRATCH_BYTES = 16 << 20     # FFD_NOALLOC_SCRATCH_BYTES

EXPORTS = ("ffd_quantize_keys", "ffd_append_kv", "ffd_decode_attention", "ffd_decode_attention_ex",
           "ffd_decode_attention_noalloc", "ffd_dense_decode_attention",
           "ffd_resolve_splits", "ffd_fused_splits", "ffd_select_kernels", "ffd_dense_resolve_splits",
           "ffd_workspace_bytes", "ffd_dense_workspace_bytes", "ffd_status_string")


class FfdLibraryError(RuntimeError):
    """libffd.so is missing or failed to load."""


class FfdError(RuntimeError):
    """A library call returned an error status."""

    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn} -> {detail} ({status})")
        self.status = status


_lib = None
P, I, F, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
PSEUDO_MAX = {"thumbnail": 0, "refined": 1}     # FFD_PSEUDO_MAX_THUMBNAIL, FFD_PSEUDO_MAX_REFINED


KERNELS = {"auto": 0, "fused": 1, "split": 2}     # FFD_KERNELS_AUTO, _FUSED, _SPLIT


class DecodeExtras(ctypes.Structure):
    """``ffd_decode_extras``: stage events, the pseudo-max output, the pseudo-max source, the
    fixed-budget (top-k) selection and the top-delta kernels."""
    _fields_ = [("stage_events", P), ("m_tilde", P), ("pseudo_max", I), ("top_k", I), ("kernels", I)]


def lib() -> ctypes.CDLL:
    """Load libffd.so (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FfdLibraryError(f"{LIB_PATH} is not built; run paper_2609_00097_amd/build.py")
    try:
        so = ctypes.CDLL(LIB_PATH)
    except OSError as e:
        raise FfdLibraryError(f"cannot load {LIB_PATH}: {e}") from e
    so.ffd_quantize_keys.argtypes = [P, P, P, P, I, I, I, I, I, I, I, P]
    so.ffd_append_kv.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, P]
    so.ffd_decode_attention.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, I, F, I, I, I, F,
                                        P, P, P, P, SZ, P]
    so.ffd_decode_attention_ex.argtypes = so.ffd_decode_attention.argtypes + [ctypes.POINTER(DecodeExtras)]
    so.ffd_decode_attention_noalloc.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, I, F, I, I, I, F,
                                                P, P, P, P]
    so.ffd_dense_decode_attention.argtypes = [P, P, P, P, I, I, I, I, I, I, F, P, P, P, SZ, P]
    so.ffd_resolve_splits.argtypes = [I, I, I, I]
    so.ffd_fused_splits.argtypes = [I, I, I, I]
    so.ffd_select_kernels.argtypes = [I, I, I, I]
    so.ffd_dense_resolve_splits.argtypes = [I, I, I, I]
    for name in ("ffd_workspace_bytes", "ffd_dense_workspace_bytes"):
        getattr(so, name).argtypes = [I, I, I, I, I, I]
        getattr(so, name).restype = SZ
    so.ffd_status_string.argtypes = [I]
    so.ffd_status_string.restype = ctypes.c_char_p
    for name in ("ffd_quantize_keys", "ffd_append_kv", "ffd_decode_attention", "ffd_decode_attention_ex",
                 "ffd_decode_attention_noalloc", "ffd_dense_decode_attention", "ffd_resolve_splits",
                 "ffd_fused_splits", "ffd_select_kernels", "ffd_dense_resolve_splits"):
        getattr(so, name).restype = I
    _lib = so
    return so


def _check(fn: str, st: int) -> None:
    if st != 0:
        raise FfdError(fn, st, lib().ffd_status_string(st).decode())


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _need(t, name, dtype, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def resolve_splits(B: int, Hkv: int, Lcap: int, num_splits: int = 0) -> int:
    """Refinement workgroups per KV group (on average) of the split kernels for this ``num_splits``
    (0 = automatic)."""
    return lib().ffd_resolve_splits(B, Hkv, Lcap, num_splits)


def fused_splits(B: int, Hkv: int, Lcap: int, num_splits: int = 0) -> int:
    """Workgroups per KV group of the fused top-delta kernel for this ``num_splits``."""
    return lib().ffd_fused_splits(B, Hkv, Lcap, num_splits)


def select_kernels(B: int, Hkv: int, Lcap: int, num_splits: int = 0) -> str:
    """The top-delta kernels the automatic choice uses: ``"fused"`` or ``"split"``."""
    k = lib().ffd_select_kernels(B, Hkv, Lcap, num_splits)
    return {1: "fused", 2: "split"}[k]


def dense_resolve_splits(B: int, Hkv: int, Lcap: int, num_splits: int = 0) -> int:
    """Splits a dense call with this ``num_splits`` uses (0 = automatic)."""
    return lib().ffd_dense_resolve_splits(B, Hkv, Lcap, num_splits)


def workspace_bytes(B: int, Hq: int, Hkv: int, Lcap: int, num_splits: int = 0,
                    dense: bool = False) -> int:
    """Bytes for ``decode_attention`` (enough for both entry points), or for the dense one only."""
    fn = lib().ffd_dense_workspace_bytes if dense else lib().ffd_workspace_bytes
    return fn(B, Hq, Hkv, Lcap, HEAD_DIM, num_splits)


def new_workspace(B: int, Hq: int, Hkv: int, Lcap: int, num_splits: int = 0, device="cuda",
                  dense: bool = False):
    """A workspace (one per stream): for ``decode_attention`` and the dense entry point alike, or,
    with ``dense=True``, the smaller one the dense entry point needs."""
    return torch.empty(max(workspace_bytes(B, Hq, Hkv, Lcap, num_splits, dense), 16),
                       dtype=torch.uint8, device=device)


def quantized_shapes(B: int, Hkv: int, Lcap: int, bits: int = 2):
    """Shapes of (codes int32, absmax bf16, resid int8) for a cache of capacity Lcap with a
    ``bits``-bit thumbnail."""
    return ((B, Hkv, Lcap // 64, bits, 64, 4), (B, Hkv, Lcap // 64, 16, 4),
            (B, Hkv, Lcap // 16, 2, 64, 16))


def thumb_bits(codes: torch.Tensor) -> int:
    """The thumbnail depth of a codes tensor ``[B, Hkv, Lcap/64, b, 64, 4]``."""
    bits = codes.shape[-3] if codes.dim() == 6 and tuple(codes.shape[-2:]) == (64, 4) else 0
    if bits not in THUMB_BITS:
        raise ValueError(f"codes must be [B, Hkv, Lcap/64, b, 64, 4] with b in {THUMB_BITS}, "
                         f"got {tuple(codes.shape)}")
    return bits


def empty_quantized(B: int, Hkv: int, Lcap: int, device, bits: int = 2):
    sc, sa, sr = quantized_shapes(B, Hkv, Lcap, bits)
    return (torch.empty(sc, dtype=torch.int32, device=device),
            torch.empty(sa, dtype=torch.bfloat16, device=device),
            torch.empty(sr, dtype=torch.int8, device=device))


def _need_quantized(quantized, B, Hkv, Lcap) -> int:
    codes, absmax, resid = quantized
    bits = thumb_bits(codes)
    for t, nm, dt, sh in zip((codes, absmax, resid), ("codes", "absmax", "resid"),
                             (torch.int32, torch.bfloat16, torch.int8),
                             quantized_shapes(B, Hkv, Lcap, bits)):
        _need(t, nm, dt, sh)
    return bits


def quantize_keys(k: torch.Tensor, t_begin: int = 0, t_end: int | None = None, out=None,
                  bits: int = 2):
    """Split bf16 keys ``[B, Hkv, Lcap, 128]`` into (codes, absmax, resid) for ``[t_begin, t_end)``
    with a ``bits``-bit thumbnail (2, 4 or 8; taken from ``out``'s codes shape when given)."""
    if k.dim() != 4:
        raise ValueError("k must be [B, Hkv, Lcap, 128]")
    B, Hkv, Lcap, D = k.shape
    _need(k, "k", torch.bfloat16)
    t_end = Lcap if t_end is None else t_end
    if out is None:
        if bits not in THUMB_BITS:
            raise ValueError(f"bits must be one of {THUMB_BITS}")
        out = empty_quantized(B, Hkv, Lcap, k.device, bits)
    bits = _need_quantized(out, B, Hkv, Lcap)
    codes, absmax, resid = out
    _check("ffd_quantize_keys", lib().ffd_quantize_keys(
        _ptr(k), _ptr(codes), _ptr(absmax), _ptr(resid), B, Hkv, Lcap, D, bits, t_begin, t_end,
        _stream(k.device)))
    return codes, absmax, resid


def append_kv(k_new, v_new, quantized, seq_lens, *, k_cache=None, v_cache=None):
    """Append one token per sequence at position ``seq_lens[b]`` (device-side) to the quantized key
    cache ``(codes, absmax, resid)`` and, when given, the bf16 caches ``[B, Hkv, Lcap, 128]``; then
    ``seq_lens[b] += 1`` for every sequence below capacity. ``k_new``/``v_new``: bf16 ``[B, Hkv, 128]``."""
    codes, absmax, resid = quantized
    B, Hkv, D = k_new.shape
    Lcap = codes.shape[2] * 64
    _need(k_new, "k_new", torch.bfloat16)
    _need(v_new, "v_new", torch.bfloat16, (B, Hkv, D))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    bits = _need_quantized(quantized, B, Hkv, Lcap)
    for t, nm in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        if t is not None:
            _need(t, nm, torch.bfloat16, (B, Hkv, Lcap, D))
    _check("ffd_append_kv", lib().ffd_append_kv(
        _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(codes), _ptr(absmax), _ptr(resid),
        _ptr(seq_lens), B, Hkv, Lcap, D, bits, _stream(k_new.device)))


def _attn_outputs(q, B, Hq, Lcap, want_lse, want_mask, out, lse, mask):
    out = torch.empty((B, Hq, HEAD_DIM), dtype=torch.bfloat16, device=q.device) if out is None else out
    if want_lse and lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    if want_mask and mask is None:
        mask = torch.empty((B, Hq, Lcap // BLOCK), dtype=torch.uint8, device=q.device)
    return out, lse, mask


def decode_attention(q, codes, absmax, resid, v, seq_lens, *, delta: float, n_sink: int = 64,
                     n_local: int = 256, num_splits: int = 0, softmax_scale: float = 0.0,
                     return_lse: bool = True, return_mask: bool = False, workspace=None,
                     out=None, lse=None, mask=None, stage_events=None, m_tilde=None,
                     pseudo_max: str = "thumbnail", top_k: int = 0, kernels: str = "auto"):
    """FFD decode attention. Returns ``(out, lse, mask)`` (lse/mask None unless requested).
    The thumbnail depth is that of ``codes`` (its last dimension is 4 words per bit).

    ``stage_events``: optional four ``torch.cuda.Event`` objects, already recorded once (so that
    they exist), which the library records before the scan kernel, after it, after the refinement
    kernel and after the merge. ``m_tilde``: optional float32 ``[B, Hq]`` receiving each head's
    pseudo-max. ``pseudo_max``: ``"thumbnail"`` (default) or ``"refined"``, the scores of the window
    tokens the pseudo-max is taken over. ``top_k > 0`` replaces the top-delta rule by the fixed
    budget of ``top_k`` blocks per head (largest thumbnail block scores, ties in block order); delta
    and the windows are then unused and ``m_tilde`` must be None. ``kernels``: ``"auto"``,
    ``"fused"`` or ``"split"`` (top-delta's kernels; see ``FFD_KERNELS_*`` in ffd.h)."""
    B, Hq, D = q.shape
    Hkv, Lcap = v.shape[1], v.shape[2]
    _need(q, "q", torch.bfloat16)
    _need(v, "v", torch.bfloat16, (B, Hkv, Lcap, D))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    bits = _need_quantized((codes, absmax, resid), B, Hkv, Lcap)
    out, lse, mask = _attn_outputs(q, B, Hq, Lcap, return_lse or lse is not None,
                                   return_mask or mask is not None, out, lse, mask)
    if workspace is None:
        workspace = new_workspace(B, Hq, Hkv, Lcap, num_splits, q.device)
    if pseudo_max not in PSEUDO_MAX:
        raise ValueError(f"pseudo_max must be one of {tuple(PSEUDO_MAX)}")
    if m_tilde is not None:
        _need(m_tilde, "m_tilde", torch.float32, (B, Hq))
    ev = None
    if stage_events is not None:
        if len(stage_events) != 4 or any(e.cuda_event == 0 for e in stage_events):
            raise ValueError("stage_events must be four recorded torch.cuda.Event objects")
        ev = (ctypes.c_void_p * 4)(*[e.cuda_event for e in stage_events])
    if kernels not in KERNELS:
        raise ValueError(f"kernels must be one of {tuple(KERNELS)}")
    extras = DecodeExtras(ctypes.cast(ev, P) if ev is not None else None, _ptr(m_tilde),
                          PSEUDO_MAX[pseudo_max], int(top_k), KERNELS[kernels])
    _check("ffd_decode_attention", lib().ffd_decode_attention_ex(
        _ptr(q), _ptr(codes), _ptr(absmax), _ptr(resid), _ptr(v), _ptr(seq_lens), B, Hq, Hkv, Lcap,
        D, bits, BLOCK, float(delta), n_sink, n_local, num_splits, float(softmax_scale), _ptr(out),
        _ptr(lse), _ptr(mask), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(q.device), ctypes.byref(extras)))
    return out, lse, mask


def decode_attention_noalloc(q, codes, absmax, resid, v, seq_lens, *, delta: float, n_sink: int = 64,
                             n_local: int = 256, num_splits: int = 0, softmax_scale: float = 0.0,
                             out=None, lse=None, mask=None):
    """``decode_attention`` through ``ffd_decode_attention_noalloc``: the library's fixed device
    scratch stands in for the workspace (no device allocation by the library; calls on one device
    must not overlap in time). ``out`` (and ``lse``/``mask`` when wanted) should be passed in by
    callers that cannot allocate; otherwise they are allocated here. Returns ``(out, lse, mask)``."""
    B, Hq, D = q.shape
    Hkv, Lcap = v.shape[1], v.shape[2]
    _need(q, "q", torch.bfloat16)
    _need(v, "v", torch.bfloat16, (B, Hkv, Lcap, D))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    bits = _need_quantized((codes, absmax, resid), B, Hkv, Lcap)
    if out is None:
        out = torch.empty((B, Hq, HEAD_DIM), dtype=torch.bfloat16, device=q.device)
    _need(out, "out", torch.bfloat16, (B, Hq, D))
    if lse is not None:
        _need(lse, "lse", torch.float32, (B, Hq))
    if mask is not None:
        _need(mask, "mask", torch.uint8, (B, Hq, Lcap // BLOCK))
    _check("ffd_decode_attention_noalloc", lib().ffd_decode_attention_noalloc(
        _ptr(q), _ptr(codes), _ptr(absmax), _ptr(resid), _ptr(v), _ptr(seq_lens), B, Hq, Hkv, Lcap,
        D, bits, BLOCK, float(delta), n_sink, n_local, num_splits, float(softmax_scale), _ptr(out),
        _ptr(lse), _ptr(mask), _stream(q.device)))
    return out, lse, mask


def dense_decode_attention(q, k, v, seq_lens, *, num_splits: int = 0, softmax_scale: float = 0.0,
                           return_lse: bool = True, workspace=None, out=None, lse=None):
    """Exact dense decode attention. Returns ``(out, lse)``."""
    B, Hq, D = q.shape
    Hkv, Lcap = k.shape[1], k.shape[2]
    _need(q, "q", torch.bfloat16)
    _need(k, "k", torch.bfloat16, (B, Hkv, Lcap, D))
    _need(v, "v", torch.bfloat16, (B, Hkv, Lcap, D))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    out, lse, _ = _attn_outputs(q, B, Hq, Lcap, return_lse or lse is not None, False, out, lse, None)
    if workspace is None:
        workspace = new_workspace(B, Hq, Hkv, Lcap, num_splits, q.device, dense=True)
    _check("ffd_dense_decode_attention", lib().ffd_dense_decode_attention(
        _ptr(q), _ptr(k), _ptr(v), _ptr(seq_lens), B, Hq, Hkv, Lcap, D, num_splits,
        float(softmax_scale), _ptr(out), _ptr(lse), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(q.device)))
    return out, lse


def default_scale() -> float:
    return 1.0 / math.sqrt(HEAD_DIM)
