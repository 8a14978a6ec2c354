"""The host runtime (context, SHA-256 key chain, index, argument validation)
built with AddressSanitizer and UBSan and driven by a native self-test, on the
CPU. The paper ran its library under address sanitizers and other analysis
tools before release (Sec. 3, last paragraph of the sabotage testing)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_39358_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host compiler")
def test_host_runtime_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "host_selftest"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "native", "host_selftest.cpp"),
           os.path.join(CSRC, "ctx.cpp"), os.path.join(CSRC, "sha256.cpp"), os.path.join(CSRC, "file_io.cpp"),
           "-pthread", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    # the environment is passed through unchanged apart from the sanitizer options
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "host self-test ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
