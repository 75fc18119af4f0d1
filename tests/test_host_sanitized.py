"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
the host translation units of libnbsgd (schedule, mixing matrices, MATCHA,
the step planner, the MLP shape checks) are rebuilt with g++ and the
sanitizers, and two programs run on them: tests/c/abi_host.c (every host
entry point and its error paths, from plain C) and tests/c/plan_emulation.cpp
(the fused step's plan walked as the kernel walks it, over 20,000 random,
straggler-skewed, sparse and full masks up to 16 x 64)."""

import os
import shutil
import subprocess

import pytest

from paper_2211_00889_amd import build


@pytest.fixture(scope="module")
def programs(tmp_path_factory):
    if shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("no host compiler")
    return build.build_sanitized_host_tests(str(tmp_path_factory.mktemp("san")))


def _run(exe):
    # the environment is passed on unchanged apart from the sanitizer options;
    # verify_asan_link_order=0 lets the sanitizer runtime load after any
    # library the environment preloads
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    return subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)


def test_host_entry_points_under_sanitizers(programs):
    r = _run(programs[0])
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.strip() == "ok"


def test_step_plan_emulation_under_sanitizers(programs):
    r = _run(programs[1])
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.strip() == "ok"
