"""The host graph compilers, the image validator and the model caches under
AddressSanitizer and UndefinedBehaviorSanitizer (CPU only; g++ builds
compiler.cpp, variative.cpp, cache.cpp, errors.cpp and
tests/sanitize/compiler_driver.cpp, no GPU code)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_21343_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_compiler_and_validator_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-pthread", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer",
           os.path.join(CSRC, "compiler.cpp"), os.path.join(CSRC, "variative.cpp"),
           os.path.join(CSRC, "cache.cpp"), os.path.join(CSRC, "errors.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "compiler_driver.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    # other preloaded libraries may precede the sanitizer runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, timeout=600,
                       env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-6000:]
    assert "ok" in r.stdout
