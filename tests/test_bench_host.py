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


def test_valu_file_format():
    # kernel, workload, 16-hex digest, non-MFMA VALU instructions per launch
    path = os.path.join(ROOT, "profiles", "valu.txt")
    for line in open(path):
        if not line.strip():
            continue
        kernel, workload, digest, n = line.split()
        assert kernel == "k_attn_prefill16"
        assert len(digest) == 16 and int(digest, 16) >= 0
        assert int(n) > 0


def test_committed_counters_match_the_sources():
    # the counters in profiles/ were taken on the sources as committed: the
    # bench line reports them (a kernel change without new counters would make
    # them null, and this test would say so)
    assert bench.measured_traffic("k_attn_prefill16", "phi3m-prefill-4k") is not None
    assert bench.measured_traffic("k_attn_decode", "phi3m-decode-8k") is not None
    assert bench.measured_traffic("k_attn_decode", "long-decode-32k") is not None
    assert bench.measured_valu("k_attn_prefill16", "phi3m-prefill-4k") is not None


def test_valu_roofline_against_the_fp32_vector_peak(monkeypatch):
    # 157.3 TFLOP/s of fp32 FMAs = 64 lanes x 2 flops per wave64 instruction
    assert abs(bench.PEAK_VALU_GINST - 157.3e3 / 128) < 1e-9
    monkeypatch.setattr(bench, "measured_valu", lambda k, w: 1.0e9)
    r = bench.valu_roofline("k", "w", 2.0, {"valu_Ginst_per_s": 800.0})
    assert r["bound"] == "alu"
    assert abs(r["achieved"] - 500.0) < 1e-6          # 1e9 instructions in 2 ms
    assert abs(r["frac"] - 500.0 / bench.PEAK_VALU_GINST) < 1e-4
    assert abs(r["frac_of_measured_ceiling"] - 500.0 / 800.0) < 1e-4
    monkeypatch.setattr(bench, "measured_valu", lambda k, w: None)
    assert bench.valu_roofline("k", "w", 2.0, {"valu_Ginst_per_s": 800.0}) is None
