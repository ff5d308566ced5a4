"""Host-side logic of bench.py (no GPU): the source digest that ties the
committed HBM counters in profiles/traffic.txt to the kernel sources."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _write(tmp_path, name, text):
    p = tmp_path / name
    p.write_text(text)
    return str(p)


def test_digest_ignores_comments_and_blank_lines(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _write(tmp_path, "k.hip", "int f(int x) {\n  return x + 1;  // one\n}\n")
    _write(tmp_path, "b.py", "X = 1\n")
    d0 = bench.source_digest(["k.hip", "b.py"])
    _write(tmp_path, "k.hip", "// header\n/* block\n   comment */\nint f(int x) {\n\n"
                              "    return x + 1;\n}\n")
    _write(tmp_path, "b.py", "# note\nX = 1\n\n")
    assert bench.source_digest(["k.hip", "b.py"]) == d0


def test_digest_changes_with_code(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _write(tmp_path, "k.hip", "int f(int x) { return x + 1; }\n")
    d0 = bench.source_digest(["k.hip"])
    _write(tmp_path, "k.hip", "int f(int x) { return x + 2; }\n")
    assert bench.source_digest(["k.hip"]) != d0


def test_traffic_file_format():
    # kernel, workload, 16-hex digest, bytes per launch; a digest that no longer
    # matches the sources makes bench.py report traffic as null, not an error
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    for line in open(path):
        if not line.strip():
            continue
        kernel, workload, digest, nbytes = line.split()
        assert kernel in ("k_attn_prefill16", "k_attn_decode")
        assert len(digest) == 16 and int(digest, 16) >= 0
        assert float(nbytes) > 0
