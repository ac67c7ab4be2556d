"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

tests/c/host_fuzz.cpp is built with g++ together with the plain C++ sources of the
library (mask layouts and tables, tile plans and mask bits, tile orders, argument
validation and the host-only entry points) and run on a seeded stream of random and
corrupted layouts and argument sets; every derived quantity is checked against a
brute-force mask from the layout's definition.  Any sanitizer report fails the run.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_25473_amd", "csrc")
HOST_SOURCES = ["layout.cpp", "validate.cpp", "capi_host.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "c", "host_fuzz.cpp")] + [os.path.join(CSRC, s) for s in HOST_SOURCES]
    subprocess.run(cmd + ["-o", exe], check=True)
    # (verify_asan_link_order=0: the sanitizer runtime need not come first among the
    # libraries the environment preloads)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    out = subprocess.run([exe, "150"], capture_output=True, text=True, env=env, timeout=300)
    assert out.returncode == 0 and out.stdout.strip().endswith("OK"), out.stdout[-3000:] + out.stderr[-3000:]
