"""Host logic of bench.py: the key under which the HBM byte counters are
kept.  The counters describe compiled kernels, so the key must change with
the code and must not change with comments or layout."""

import os
import shutil

import bench


def test_code_tokens_drop_comments_and_layout():
    a = "int  f(int x) { // one\n  return x + 1; /* two\n three */ }\n"
    b = "int f(int x) {\n\treturn x + 1;\n}"
    assert bench.code_tokens(a) == bench.code_tokens(b)
    assert bench.code_tokens(a) != bench.code_tokens(a.replace("x + 1", "x + 2"))


def test_code_tokens_keep_literals():
    src = 'const char* s = "a // not a comment"; char c = \'"\'; const char* t = "/* nor this */";'
    out = bench.code_tokens(src)
    assert '"a // not a comment"' in out and '"/* nor this */"' in out and "'\"'" in out


def test_source_hash_follows_the_code_only(tmp_path, monkeypatch):
    src = os.path.join(os.path.dirname(bench.__file__), "paper_2602_18851_amd", "csrc")
    dst = tmp_path / "csrc"
    shutil.copytree(src, dst)
    monkeypatch.setattr(bench, "KERNEL_DIR", str(dst))
    base = bench.source_hash()
    f = dst / "sweeps.hip"
    text = f.read_text()
    f.write_text("// a comment added above everything\n" + text.replace("\n", "\n  ", 5))
    assert bench.source_hash() == base
    f.write_text(text.replace("kStreamPolicy", "kStreamPolicy + 0", 1))
    assert bench.source_hash() != base
