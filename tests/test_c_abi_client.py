"""The boundary from plain C: ``tests/c_abi_client.c`` includes
``include/celty.h`` under ``-std=c99 -pedantic -Werror``, links against the
in-tree ``libcelty.so`` and drives the host entry points (size plan, encode,
decode, an argument error, status strings) on a hand-checked 2 x 3 matrix.
No device call is made, so it runs without a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2608_01536_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_header_is_c99_and_host_entry_points_work_from_c(tmp_path):
    exe = tmp_path / "c_abi_client"
    build = subprocess.run(
        ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", os.path.join(ROOT, "include"),
         os.path.join(ROOT, "tests", "c_abi_client.c"), "-L", LIBDIR, "-lcelty", f"-Wl,-rpath,{LIBDIR}",
         "-o", str(exe)],
        capture_output=True, text=True, timeout=120)
    assert build.returncode == 0, build.stderr[-4000:]
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, f"check {run.returncode} failed: {run.stdout}{run.stderr}"
    assert "c abi client: ok" in run.stdout
