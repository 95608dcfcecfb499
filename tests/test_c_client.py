"""include/mep.h compiles as C11 with warnings as errors, and a C program
linked against libmep.so runs the host-only entry points without a GPU."""
import os
import shutil
import subprocess

import pytest

from paper_2512_22147_amd import mep

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_client_of_the_abi(tmp_path):
    mep.lib()  # the library is built
    libdir = os.path.dirname(mep.LIB_PATH)
    exe = str(tmp_path / "client")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "abi_c", "host_calls.c"), "-o", exe,
           f"-L{libdir}", "-l:libmep.so", f"-Wl,-rpath,{libdir}", "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
