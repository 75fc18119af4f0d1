"""nbsgd_step_strided and nbsgd_step_server driven from a plain C program (tests/c/abi_step.c, built
by __graft_entry__.build()) on HIP-runtime device buffers, against the
oracle on the same seeded inputs."""

import os
import struct
import subprocess

import numpy as np
import pytest

import oracle
import synth
from synth import workloads
from tests._util import TOL, rel_err

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c", "abi_step")


@pytest.mark.parametrize("n,m,P,ld,order", [(4, 4, 1030, 1036, 0), (8, 8, 20002, 20008, 1),
                                            (5, 3, 4099, 4100, 0), (16, 2, 257, 260, 1),
                                            (8, 8, 20002, 20008, 2), (3, 5, 1031, 1036, 2)])
def test_strided_step_from_c(tmp_path, n, m, P, ld, order):
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is missing: __graft_entry__.build() compiles it")
    seed = 11 * n + P
    X0 = synth.normal_f32(seed, workloads.STREAM_X, np.arange(n * P), 1.0).reshape(n, P)
    G0 = synth.normal_f32(seed, workloads.STREAM_G, np.arange(n * m * P), 0.03).reshape(n, m, P)
    V0 = (0.1 * synth.normal_f32(seed + 1, workloads.STREAM_X, np.arange(n * P), 1.0)).reshape(n, P)
    s = oracle.schedule.sample_schedule(seed, 2, n, m, oracle.schedule.Delay(1, 1.0, 1.0))
    mask = s["mask"].astype(np.uint8)
    W = (oracle.mixing.w_ring(n) if n > 2 else oracle.mixing.w_uniform(n)).astype(np.float32)
    lr, mom = np.float32(0.1), np.float32(0.9)
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(struct.pack("<iiiqqff", n, m, order, P, ld, lr, mom))
        for a in (mask, W, X0, V0.astype(np.float32), G0):
            f.write(np.ascontiguousarray(a).tobytes())
    print(f"[case] C ABI step n={n} m={m} P={P} ld={ld} order={order} (2: server form)", flush=True)
    r = subprocess.run([EXE, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"
    out = np.fromfile(dst, dtype=np.float32)
    assert out.size == 2 * n * P
    Xg, Vg = out[:n * P].reshape(n, P), out[n * P:].reshape(n, P)
    V0d = V0.astype(np.float32).astype(np.float64)
    if order == 2:  # the server form: row 0 of X is the model, the other rows stay as they were
        xo, Vo = oracle.step.parameter_server_step(X0[0], V0d, G0, mask, float(lr), float(mom))
        assert rel_err(Vg, Vo) <= TOL
        assert rel_err(Xg[0], xo) <= TOL
        assert (Xg[1:] == X0[1:]).all()
        return
    o = oracle.step.MIX_THEN_STEP if order == 0 else oracle.step.STEP_THEN_MIX
    Xo, Vo = oracle.step.step(X0, V0d, G0, mask, W.astype(np.float64), lr, mom, o)
    assert rel_err(Vg, Vo) <= TOL
    assert rel_err(Xg, Xo) <= TOL
