"""include/nbsgd.h from plain C: the header compiles as strict C11 and the
host entry points work when called from C (no GPU)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2211_00889_amd")


def test_host_entry_points_from_c(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    exe = str(tmp_path / "abi_host")
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I",
           os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_host.c"), "-o", exe,
           "-L", LIB_DIR, "-lnbsgd", "-lm", f"-Wl,-rpath,{LIB_DIR}"]
    b = subprocess.run(cmd, capture_output=True, text=True)
    assert b.returncode == 0, b.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"
