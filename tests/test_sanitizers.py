"""AddressSanitizer + UndefinedBehaviorSanitizer runs of the host code (CPU).

The oracle (oracle/sanitize_check.c) and the library's host side
(tests/sanitize_host_check.cpp, with every library source; the sanitizers
apply to host code only) are built into throw-away executables and run on
seeded problems of every stage-type mode.  Any out-of-bounds access, leak or
undefined arithmetic fails the run."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=ENV)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_oracle_under_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "oracle_check")
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                        "-I", os.path.join(ROOT, "oracle"), "-o", exe,
                        os.path.join(ROOT, "oracle", "sanitize_check.c"),
                        os.path.join(ROOT, "oracle", "hapmoe_oracle.c"), "-lm"], check=True)
        out = _run(exe)
    assert out.count("dp = brute force") == 25


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc"), reason="hipcc missing")
def test_library_host_code_under_sanitizers():
    from paper_2609_39350_amd import build
    csrc = os.path.join(ROOT, "paper_2609_39350_amd", "csrc")
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "host_check")
        cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-ffp-contract=off",
               "-fno-fast-math", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
               "-Xarch_host", "-fno-omit-frame-pointer",
               "-I", os.path.join(ROOT, "include"), "-I", csrc, "-o", exe,
               os.path.join(ROOT, "tests", "sanitize_host_check.cpp"),
               *[os.path.join(csrc, s) for s in build.SOURCES]]
        subprocess.run(cmd, check=True, capture_output=True)
        out = _run(exe)
    assert out.count("candidates,") == 48 and "13 malformed problems refused" in out
