"""The host encoder and decoder under the compiler's sanitizers.

``encode.cpp`` is plain host C++ (offline packing, Section 3.2), so it is
built here with g++ alone, together with ``encoder_sanitize_driver.cpp``, once
with AddressSanitizer + UndefinedBehaviorSanitizer and once with
ThreadSanitizer (the encoder splits columns over worker threads).  The driver
round-trips seeded random matrices of many shapes, tile heights and densities
through ``celty_encode_plan`` / ``celty_encode`` / ``celty_decode`` at 1, 3
and all threads, checks that the encoding does not depend on the thread
count, and exercises the documented error returns.  Any sanitizer report
aborts the driver with a non-zero status.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [
    os.path.join(ROOT, "paper_2608_01536_amd", "csrc", "encode.cpp"),
    os.path.join(ROOT, "tests", "encoder_sanitize_driver.cpp"),
]

SANITIZERS = {
    "address,undefined": {
        "flags": ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"],
        "env": {"ASAN_OPTIONS": "detect_leaks=1:verify_asan_link_order=0", "UBSAN_OPTIONS": "print_stacktrace=1"},
    },
    "thread": {
        "flags": ["-fsanitize=thread"],
        "env": {"TSAN_OPTIONS": "halt_on_error=1"},
    },
}


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
@pytest.mark.parametrize("sanitizer", sorted(SANITIZERS))
def test_encoder_clean_under_sanitizer(sanitizer, tmp_path):
    spec = SANITIZERS[sanitizer]
    exe = tmp_path / "encoder_driver"
    build = subprocess.run(
        ["g++", "-std=c++17", "-O1", "-g", *spec["flags"], "-I", os.path.join(ROOT, "include"),
         *SOURCES, "-pthread", "-o", str(exe)],
        capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ)
    env.update(spec["env"])
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "encoder sanitize driver: ok" in run.stdout
    assert "runtime error" not in run.stderr and "WARNING: ThreadSanitizer" not in run.stderr
