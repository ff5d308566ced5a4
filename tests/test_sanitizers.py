"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):

* the CPU oracle (oracle/turbo_oracle.c) driven through every routine on
  small ragged inputs (tests/sanitize/oracle_driver.c);
* the host side of the C ABI library (argument checks, sizing helpers, the
  Sec. 3.2 bit choice) called with valid, extreme and invalid arguments
  (tests/sanitize/abi_driver.cpp); the sanitizers instrument host code only.

Either driver exits non-zero on the first sanitizer report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all"]


def _run(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", *SAN, "-fno-omit-frame-pointer",
                           "-ffp-contract=off",
                           os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
                           os.path.join(ROOT, "oracle", "turbo_oracle.c"), "-o", exe, "-lm"])
    assert "ok" in _run(exe)


def test_abi_host_side_under_asan_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("no hipcc")
    host_san = [x for f in SAN + ["-fno-omit-frame-pointer"] for x in ("-Xarch_host", f)]
    inc = ["-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2412_08585_amd", "csrc")]
    api_o, prj_o, drv_o, exe = (str(tmp_path / n)
                                for n in ("api.o", "prj.o", "drv.o", "abi_driver"))
    for unit, obj in (("turbo_api.hip", api_o), ("qkv_project.hip", prj_o)):
        subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                               "-fPIC", *host_san, "-Xclang", "-target-feature", "-Xclang",
                               "-packed-fp32-ops", *inc, "-c",
                               os.path.join(ROOT, "paper_2412_08585_amd", "csrc", unit),
                               "-o", obj], stderr=subprocess.DEVNULL)
    subprocess.check_call([HIPCC, "-O1", "-g", "-std=c++17", *host_san, *inc, "-c",
                           os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp"), "-o",
                           drv_o], stderr=subprocess.DEVNULL)
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", *host_san, api_o, prj_o, drv_o, "-o", exe],
                          stderr=subprocess.DEVNULL)
    assert "ok" in _run(exe)
