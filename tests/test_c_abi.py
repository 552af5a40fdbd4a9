"""The C ABI from a plain C99 program (tests/c/abi_host.c): compiled with
gcc against include/crosspool.h, linked to the built library, run on a
host-only pool and the planner (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

from paper_2606_24506_amd import crosspool as cpl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_plain_c_program_uses_the_abi(tmp_path):
    libdir = os.path.dirname(cpl._LIB_PATH)
    exe = tmp_path / "abi_host"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_host.c"), "-o", str(exe), "-L", libdir, "-lcrosspool",
                    "-Wl,-rpath," + libdir], check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "ok"
