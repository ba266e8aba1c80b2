"""bench.py's records: the traffic record's staleness check (a comment or whitespace edit to a kernel
source keeps the measured bytes, any change to the code voids them) and the algorithmic byte counts
behind every reported TB/s and roofline fraction."""
import json
import os

import numpy as np

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def digest_of(tmp_path, text):
    p = tmp_path / "k.hip"
    p.write_text(text)
    return bench.code_digest(str(p))


def test_comments_and_whitespace_do_not_change_the_digest(tmp_path):
    a = digest_of(tmp_path, "int f(int x) {\n  return x + 1;  // one more\n}\n")
    b = digest_of(tmp_path, "// header\nint f(int x) {\n    /* body */ return x + 1;\n\n}\n")
    assert a == b


def test_code_edits_change_the_digest(tmp_path):
    a = digest_of(tmp_path, "int f(int x) { return x + 1; }\n")
    for edit in ("int f(int x) { return x + 2; }\n", "int f(int x) { return x - 1; }\n",
                 "int f(int y) { return y + 1; }\n"):
        assert digest_of(tmp_path, edit) != a


def test_record_names_existing_sources():
    rec = json.load(open(bench.TRAFFIC_RECORD))
    assert rec["code_sha256"]
    for path, digest in rec["code_sha256"].items():
        assert os.path.exists(os.path.join(ROOT, path)), path
        assert len(digest) == 64
    for name in ("ffd_scan_kernel", "ffd_refine_kernel", "lse_merge_kernel"):
        assert rec["kernels"][name]["hbm_bytes_per_launch"] > 0


def _tiny_case():
    from types import SimpleNamespace
    return SimpleNamespace(B=2, Hq=8, Hkv=2, G=4, D=128, seq_lens=np.array([130, 64]))


def test_algorithmic_bytes_of_a_hand_counted_step():
    """The roofline's numerator on a hand-counted case: 2 sequences (130 and 64 tokens), 8 query /
    2 KV heads. Kept (head, block): sequence 0, KV head 0: head 0 block 0 and head 2 block 2 (the
    last, partial block: 2 tokens), so the group union holds 64 + 2 tokens; KV head 1 keeps nothing.
    Sequence 1: head 1 block 0 (KV head 0) and head 5 block 0 (KV head 1), 64 tokens each; a bit set
    past the sequence's end (block 1) is not counted."""
    import bench
    case = _tiny_case()
    mask = np.zeros((2, 8, 4), dtype=bool)
    mask[0, 0, 0] = mask[0, 2, 2] = True
    mask[1, 1, 0] = mask[1, 5, 0] = True
    mask[1, 0, 1] = True
    nb = bench.algorithmic_bytes(case, mask, rows=3)
    assert nb["gather_tokens"] == 66 + 64 + 64
    assert nb["scan"] == 34 * (130 + 64) * 2                # 32 B of 2-bit codes + 2 B absmax
    assert nb["gather"] == (128 + 256) * 194                # int8 residual + bf16 values
    assert nb["io"] == 2 * 8 * (256 + 256 + 4)              # q in, out, lse
    assert nb["partials"] == 2 * 2 * 8 * 3 * 130 * 4        # m, l, acc[128] written and read
    assert nb["total"] == nb["scan"] + nb["gather"] + nb["io"] + nb["partials"]
    assert bench.algorithmic_bytes(case, mask, rows=3, bits=4)["scan"] == 66 * 194 * 2
    assert bench.algorithmic_bytes(case, mask, rows=0)["partials"] == 0


def test_dense_bytes_of_a_hand_counted_step():
    import bench
    case = _tiny_case()
    assert bench.dense_bytes(case, 2) == 512 * 194 * 2 + 2 * 8 * (512 + 4) + 2 * 2 * 8 * 2 * 130 * 4
