"""The harness generator's C ABI (include/synth.h) from plain C
(tests/c/synth_fill.c, built by __graft_entry__.build()): argument errors
without a GPU; on the GPU, device values bit for bit against the program's
own transcription of the generator's definition.  Also: every symbol the
header declares is exported by libsynth.so."""

import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c", "synth_fill")


def test_synth_header_symbols_exported():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "synth.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(synth_[a-z_]+)\s*\(", text)))
    assert names == ["synth_fill", "synth_fill_normal"]
    lib = ctypes.CDLL(os.path.join(ROOT, "synth", "libsynth.so"))
    for name in names:
        assert hasattr(lib, name), name


def test_synth_argument_errors_from_c():
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is missing: __graft_entry__.build() compiles it")
    r = subprocess.run([EXE, "host"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"


@pytest.mark.gpu
def test_synth_device_values_from_c():
    print("[case] synth_fill_normal from C on the device", flush=True)
    r = subprocess.run([EXE, "device"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"
