"""The C-ABI library loads without a GPU, exports every symbol ffd.h declares, and rejects bad
arguments with status codes before touching the GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ffd.h")


def declared_functions():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(ffd_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def so():
    from paper_2609_00097_amd import ffd
    if not os.path.exists(ffd.LIB_PATH):
        pytest.skip("libffd.so not built (run __graft_entry__.build())")
    return ffd.lib()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("ffd_quantize_keys", "ffd_append_kv", "ffd_decode_attention", "ffd_decode_attention_ex",
              "ffd_dense_decode_attention", "ffd_resolve_splits", "ffd_dense_resolve_splits", "ffd_workspace_bytes", "ffd_dense_workspace_bytes",
              "ffd_status_string"):
        assert n in names


def test_every_declared_symbol_is_exported(so):
    for n in declared_functions():
        assert hasattr(so, n), n


def test_status_strings(so):
    assert so.ffd_status_string(0) == b"FFD_OK"
    assert so.ffd_status_string(3) == b"FFD_ERR_WORKSPACE_TOO_SMALL"
    assert so.ffd_status_string(99) == b"FFD_ERR_UNKNOWN"


def test_splits_and_workspace_sizes(so):
    # split kernels: (S + 1) * B * Hkv refinement workgroups, one per CU (no GPU here: 256 CUs)
    assert so.ffd_resolve_splits(4, 8, 131072, 0) == 7            # (7 + 1) * 32 = 256 refinement workgroups
    assert so.ffd_resolve_splits(1, 2, 4096, 0) == 8              # capped: 64 blocks / 8 per split
    assert so.ffd_resolve_splits(4, 6, 131072, 0) == 9            # (9 + 1) * 24 = 240 <= 256
    assert so.ffd_resolve_splits(64, 8, 131072, 0) == 1           # at least one split
    assert so.ffd_resolve_splits(4, 8, 131072, 7) == 7
    assert so.ffd_resolve_splits(4, 8, 131072, 5000) == 0
    # fused kernel: S1 workgroups per (sequence, KV head): one for at most 64 blocks, else ~16 blocks
    # each with at most two workgroups per CU in all (512), never fewer than blocks / 256
    assert so.ffd_fused_splits(1, 2, 4096, 0) == 1                # 64 blocks: one workgroup, no merge
    assert so.ffd_fused_splits(1, 8, 8192, 0) == 8                # 128 blocks / 16
    assert so.ffd_fused_splits(1, 8, 131072, 0) == 64             # capped: 512 / 8 groups
    assert so.ffd_fused_splits(1, 8, 262144, 0) == 32             # 512 / 8 leaves 64 blocks: one per CU
    assert so.ffd_fused_splits(2, 8, 131072, 0) == 16             # 512 / 16 leaves 64 blocks: one per CU
    assert so.ffd_fused_splits(4, 8, 131072, 0) == 16             # capped: 512 / 32 groups
    assert so.ffd_fused_splits(4, 6, 131072, 0) == 21             # floor(512 / 24)
    assert so.ffd_fused_splits(64, 8, 131072, 0) == 8             # at least 2048 / 256
    assert so.ffd_fused_splits(4, 8, 131072, 7) == 8              # raised to 2048 / 256
    assert so.ffd_fused_splits(4, 8, 131072, 12) == 12
    assert so.ffd_fused_splits(4, 8, 131072, 5000) == 0
    # automatic kernels: fused while a workgroup covers at most 64 blocks or a sequence fits one
    # workgroup (1 = fused, 2 = split)
    assert so.ffd_select_kernels(1, 2, 4096, 0) == 1
    assert so.ffd_select_kernels(1, 8, 32768, 0) == 1             # 32 workgroups of 16 blocks
    assert so.ffd_select_kernels(1, 8, 131072, 0) == 1            # 64 workgroups of 32 blocks
    assert so.ffd_select_kernels(1, 8, 262144, 0) == 1            # 128 blocks, one workgroup per CU
    assert so.ffd_select_kernels(2, 8, 131072, 0) == 1            # 128 blocks, one workgroup per CU
    assert so.ffd_select_kernels(1, 8, 524288, 0) == 2            # 128 blocks per workgroup
    assert so.ffd_select_kernels(4, 8, 131072, 0) == 2            # 128 blocks per workgroup
    assert so.ffd_select_kernels(4, 8, 131072, 32) == 1           # 64 blocks per workgroup
    assert so.ffd_select_kernels(4, 8, 131072, 5000) == 0
    assert so.ffd_dense_resolve_splits(4, 8, 131072, 0) == 15     # dense: 512 workgroups
    assert so.ffd_dense_resolve_splits(4, 8, 131072, 5) == 5
    assert so.ffd_dense_resolve_splits(16, 8, 131072, 0) == 5     # 128 KV groups: 768 workgroups
    assert so.ffd_dense_resolve_splits(8, 8, 131072, 0) == 11     # 64 KV groups: 768 workgroups
    # partials max((S*P + P)*G, B*Hq*S1) rows of (D+2)*4 bytes | table P*8 | counts P*S1s*4 |
    # lists P*C*4 | block scores P*C*G*4, each region on a 256-byte boundary (S = 7 refinement splits
    # and S1s = 8 scan splits of the split kernels at 4 x 8 x 128K; S1 = 16 for the fused kernel)
    up = lambda x: -(-x // 256) * 256
    P, G, C = 32, 4, 2048
    assert so.ffd_workspace_bytes(4, 32, 8, 131072, 128, 0) == (
        up(max((7 * P + P) * G, 4 * 32 * 16) * 130 * 4) + up(P * 8) + up(P * 8 * 4) + up(P * C * 4)
        + P * C * G * 4)
    # the dense path's balanced partials (S + 1 = 16 rows per head) and table are larger than the FFD
    # layout for few blocks
    dense = up(4 * 32 * 16 * 130 * 4) + 32 * 8
    assert so.ffd_workspace_bytes(4, 32, 8, 8192, 128, 0) == dense
    P, G, C = 2, 8, 64
    assert so.ffd_workspace_bytes(1, 16, 2, 4096, 128, 3) == (
        up((3 * P + P) * G * 130 * 4) + up(P * 8) + up(P * 4 * 4) + up(P * C * 4)
        + P * C * G * 4)
    assert so.ffd_workspace_bytes(1, 8, 8, 1 << 25, 128, 1) == 0         # Lcap beyond 2^24 tokens
    assert so.ffd_dense_workspace_bytes(4, 32, 8, 131072, 128, 0) == dense
    # more than 256 sequences: equal runs per sequence, S rows per head and no table
    assert so.ffd_dense_workspace_bytes(300, 8, 8, 4096, 128, 1) == 300 * 8 * 1 * 130 * 4
    assert so.ffd_workspace_bytes(4, 32, 8, 131072, 96, 0) == 0
    assert so.ffd_dense_workspace_bytes(4, 32, 8, 131072, 96, 0) == 0


def _decode(so, **kw):
    a = dict(q=None, codes=None, absmax=None, resid=None, v=None, lens=None, B=1, Hq=32, Hkv=8,
             Lcap=4096, D=128, bits=2, block=64, delta=5.0, n_sink=64, n_local=256, splits=0, scale=0.0,
             out=None, lse=None, mask=None, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return so.ffd_decode_attention(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(), 1),                                 # null pointers
    (dict(D=96), 2), (dict(block=32), 2), (dict(Hq=12, Hkv=1), 2), (dict(Hq=30), 1),
    (dict(Lcap=100), 1), (dict(delta=-1.0), 1), (dict(delta=float("nan")), 1),
    (dict(n_sink=-1), 1), (dict(splits=2000), 1), (dict(B=0), 0),
    (dict(bits=3), 2), (dict(bits=16), 2), (dict(bits=0), 1), (dict(bits=-2), 1),
    (dict(B=0, bits=4), 0), (dict(B=0, bits=8), 0), (dict(B=0, bits=1), 2),
])
def test_argument_checks_return_before_any_launch(so, kw, status):
    assert _decode(so, **kw) == status


def test_misaligned_and_small_workspace(so):
    fake = 0x1000
    args = dict(q=fake, codes=fake, absmax=fake, resid=fake, v=fake, lens=fake, out=fake, ws=fake)
    assert _decode(so, **args, ws_bytes=16) == 3
    assert _decode(so, **{**args, "q": fake + 2}, ws_bytes=1 << 30) == 1
    # the dense entry point needs only the partials
    need = so.ffd_dense_workspace_bytes(1, 32, 8, 4096, 128, 0)
    assert so.ffd_dense_decode_attention(fake, fake, fake, fake, 1, 32, 8, 4096, 128, 0, 0.0, fake, None,
                                         fake, need - 1, None) == 3


def test_append_argument_checks(so):
    fake = 0x1000
    # null pointers, misalignment, bad shapes: rejected before any launch
    assert so.ffd_append_kv(None, None, None, None, None, None, None, None, 1, 8, 4096, 128, 2, None) == 1
    assert so.ffd_append_kv(fake, fake, None, None, fake, fake, fake, fake + 2, 1, 8, 4096, 128, 2, None) == 1
    assert so.ffd_append_kv(fake, fake + 8, None, None, fake, fake, fake, fake, 1, 8, 4096, 128, 2, None) == 1
    assert so.ffd_append_kv(fake, fake, None, None, fake, fake, fake, fake, 1, 8, 100, 128, 2, None) == 1
    assert so.ffd_append_kv(fake, fake, None, None, fake, fake, fake, fake, 1, 8, 4096, 96, 2, None) == 2
    assert so.ffd_append_kv(fake, fake, None, None, fake, fake, fake, fake, 1, 8, 4096, 128, 3, None) == 2
    assert so.ffd_append_kv(None, None, None, None, None, None, None, None, 0, 8, 4096, 128, 8, None) == 0


def test_quantize_range_checks(so):
    assert so.ffd_quantize_keys(None, None, None, None, 1, 8, 4096, 128, 2, 10, 5, None) == 1
    assert so.ffd_quantize_keys(None, None, None, None, 1, 8, 4096, 128, 2, 0, 5000, None) == 1
    assert so.ffd_quantize_keys(None, None, None, None, 1, 8, 4096, 128, 2, 7, 7, None) == 0
    assert so.ffd_quantize_keys(None, None, None, None, 1, 8, 4096, 96, 2, 0, 1, None) == 2
    for bits, status in ((4, 0), (8, 0), (3, 2), (0, 1)):
        assert so.ffd_quantize_keys(None, None, None, None, 1, 8, 4096, 128, bits, 7, 7, None) == status


def test_extras_pseudo_max_source_checked_before_launch(so):
    from paper_2609_00097_amd import ffd
    fake = 0x1000
    args = [fake] * 6 + [1, 32, 8, 4096, 128, 2, 64, 5.0, 64, 256, 0, 0.0, fake, None, None, fake, 1 << 30, None]
    bad = ffd.DecodeExtras(None, None, 7)
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(bad)) == 1
    mis = ffd.DecodeExtras(None, fake + 2, 0)          # misaligned m_tilde
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(mis)) == 1


def test_extras_top_k_checked_before_launch(so):
    """top_k < 0, or top_k > 0 together with an m_tilde output, is rejected before any launch."""
    from paper_2609_00097_amd import ffd
    fake = 0x1000
    args = [fake] * 6 + [1, 32, 8, 4096, 128, 2, 64, 5.0, 64, 256, 0, 0.0, fake, None, None, fake, 1 << 30, None]
    neg = ffd.DecodeExtras(None, None, 0, -1)
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(neg)) == 1
    with_mt = ffd.DecodeExtras(None, fake, 0, 8)
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(with_mt)) == 1
    # the struct the binding passes has the header's four fields, in order
    assert [f[0] for f in ffd.DecodeExtras._fields_] == ["stage_events", "m_tilde", "pseudo_max", "top_k",
                                                          "kernels"]


def test_extras_kernels_checked_before_launch(so):
    """An unknown kernel choice, or the fused kernel with the top-k rule, is rejected before any launch."""
    from paper_2609_00097_amd import ffd
    fake = 0x1000
    args = [fake] * 6 + [1, 32, 8, 4096, 128, 2, 64, 5.0, 64, 256, 0, 0.0, fake, None, None, fake, 1 << 30, None]
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(ffd.DecodeExtras(None, None, 0, 0, 3))) == 1
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(ffd.DecodeExtras(None, None, 0, 0, -1))) == 1
    assert so.ffd_decode_attention_ex(*args, ctypes.byref(ffd.DecodeExtras(None, None, 0, 8, 1))) == 1
