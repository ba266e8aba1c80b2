"""The traffic record's staleness check: a comment or whitespace edit to a kernel source keeps the
measured bytes, any change to the code voids them."""
import json
import os

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
