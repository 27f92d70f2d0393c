"""The host packer (csrc/pack.cpp) built with g++ under AddressSanitizer and
UndefinedBehaviorSanitizer, every report fatal, and driven through every host
entry point of the C ABI (tests/host/pack_sanitize.cpp): every configuration
family, ragged shapes, one and several threads, all-zero rows, ties, NaN
input, short and NULL buffers.  CPU only; no GPU code is built here."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2406_13868_amd", "csrc")


@pytest.mark.slow
def test_packer_under_asan_and_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / "pack_sanitize")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(HERE, "host", "pack_sanitize.cpp"), os.path.join(CSRC, "pack.cpp"),
           "-lpthread", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and "packer sanitized run ok" in r.stdout, (r.stdout + r.stderr)[-4000:]
