"""GPU parity of the end-to-end MLP workload (bf16 MFMA GEMMs, fp32
accumulation) against the oracle (bf16-rounded GEMM inputs, fp64 arithmetic),
through the C ABI.  The bar is relative error 1e-2 (bf16 GEMM inputs); the
sample indices, masks and counts must match exactly."""

import dataclasses
import os

import numpy as np
import pytest

import oracle
from oracle.mlp import BF16, Shape
from paper_2211_00889_amd import _lib, runner
from synth import mlp_data, workloads
from tests._util import mlp_blocks, pad_cols, rel_err_blocks

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL_BF16 = 1e-2  # per parameter block (W1, b1, W2, b2), each against its own rms
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mlp_trajectory.npz")


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _data(wl):
    A = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(wl.seed, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    return A, y, x0


@pytest.fixture(scope="module")
def tiny():
    wl = workloads.MLP_TINY
    return (wl, *_data(wl))


def test_grad_small_shape_every_entry(tiny):
    wl, A, y, x0 = tiny
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    rng = np.random.default_rng(0)
    X = (x0[None, :] + 0.05 * rng.standard_normal((wl.n, s.n_params))).astype(np.float32)
    mask = (rng.random((wl.n, wl.m)) < 0.6).astype(np.uint8)
    mask[1] = 0  # a learner with nothing finished: its rows stay untouched
    idx = rng.integers(0, wl.n_samples, size=(wl.n, wl.m, wl.batch)).astype(np.int32)
    _say(f"mlp grad small n={wl.n} m={wl.m} finished={int(mask.sum())}")
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    Xd = torch.from_numpy(pad_cols(X, r.P)).to(DEV)
    r.G.fill_(7.0)
    r.losses.fill_(-1.0)
    _lib.mlp_grad(Xd, wl.m, r.dims, r.data, r.labels, idx, mask, r.G, r.losses, r.workspace)
    torch.cuda.synchronize()
    G = r.G.cpu().numpy()
    L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
    for i in range(wl.n):
        for j in range(wl.m):
            if mask[i, j]:
                g, loss = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
                assert rel_err_blocks(G[i, j], g, mlp_blocks(*r.dims)) <= TOL_BF16, (i, j)
                assert (G[i, j, s.n_params:] == 0).all()  # the padding
                assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)
            else:
                assert (G[i, j] == 7.0).all() and L[i, j] == -1.0


@pytest.mark.parametrize("d_in,hidden,classes", [(384, 192, 10), (640, 320, 16), (256, 512, 2),
                                                  (128, 64, 16)])
def test_grad_and_loss_odd_shapes_every_entry(d_in, hidden, classes):
    """Shapes whose d_in splits into 3 or 2 slices (d_in / 64 = 6 or 10) and
    whose hidden units leave a half-filled 128-unit block (192, 320), two and
    sixteen classes; three learners with 1-5 finished mini-batches each, so
    the forward's 4-mini-batch groups come in every size; every finished
    entry and the evaluation losses against the oracle."""
    n, m, n_samples = 3, 5, 300
    s = Shape(d_in, hidden, classes, 32)
    A = mlp_data.inputs(7, n_samples, d_in)
    y = mlp_data.teacher_labels(7, A, hidden, classes)
    x0 = mlp_data.student_init(7, d_in, hidden, classes)
    rng = np.random.default_rng(d_in + hidden + classes)
    X = (x0[None, :] + 0.05 * rng.standard_normal((n, s.n_params))).astype(np.float32)
    mask = np.zeros((n, m), np.uint8)
    for i, c in enumerate((1, 5, 3)):
        mask[i, rng.permutation(m)[:c]] = 1  # not a prefix
    idx = rng.integers(0, n_samples, size=(n, m, 32)).astype(np.int32)
    _say(f"mlp grad shape d_in={d_in} hidden={hidden} classes={classes}")
    dims = (d_in, hidden, classes)
    P = _lib.mlp_param_count(*dims)
    Xd = torch.from_numpy(pad_cols(X, P)).to(DEV)
    data = torch.from_numpy(A).to(DEV)
    labels = torch.from_numpy(y.astype(np.int32)).to(DEV)
    G = torch.full((n, m, P), 7.0, dtype=torch.float32, device=DEV)
    losses = torch.full((n * m,), -1.0, dtype=torch.float32, device=DEV)
    rows = max(n * m * 32, 160)
    ws = torch.empty((_lib.mlp_workspace_bytes(*dims, rows) + 15) // 16 * 4, dtype=torch.float32,
                     device=DEV)
    _lib.mlp_grad(Xd, m, dims, data, labels, idx, mask, G, losses, ws)
    ev_idx = rng.integers(0, n_samples, size=160).astype(np.int32)
    ev = torch.full((5,), -1.0, dtype=torch.float32, device=DEV)
    _lib.mlp_loss(Xd[2], dims, data, labels, ev_idx, ev, ws)
    torch.cuda.synchronize()
    Gh, Lh = G.cpu().numpy(), losses.cpu().numpy().reshape(n, m)
    for i in range(n):
        for j in range(m):
            if mask[i, j]:
                g, loss = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
                assert rel_err_blocks(Gh[i, j], g, mlp_blocks(*dims)) <= TOL_BF16, (i, j)
                assert (Gh[i, j, s.n_params:] == 0).all()
                assert abs(Lh[i, j] - loss) <= TOL_BF16 * abs(loss)
            else:
                assert (Gh[i, j] == 7.0).all() and Lh[i, j] == -1.0
    evh = ev.cpu().numpy()
    for k in range(5):
        b = ev_idx[32 * k:32 * k + 32]
        _, loss = oracle.mlp.grad(X[2], A[b], y[b], s, BF16)
        assert abs(evh[k] - loss) <= TOL_BF16 * abs(loss), k


def test_grad_full_shape_sampled_entries():
    """The full shape in the runner's launch configuration: padded rows
    (row_stride(P) = 2^21 floats apart) through nbsgd_mlp_grad_strided."""
    wl = workloads.MLP
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    assert r.ld == 1 << 21 and r.ld > r.P
    mask, counts, _, _ = r.schedule.mask(0)
    idx = _lib.minibatch_indices(wl.seed, 0, wl.n, wl.m, wl.batch, wl.shard)
    _say(f"mlp grad full shape finished={int(mask.sum())} ld={r.ld}")
    r.Grows.fill_(7.0)
    _lib.mlp_grad_strided(r.Xrows, wl.m, r.dims, r.data, r.labels, idx, mask, r.Grows, r.losses,
                          r.workspace)
    torch.cuda.synchronize()
    L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
    finished = list(zip(*np.nonzero(mask)))
    for (i, j) in [finished[0], finished[len(finished) // 2], finished[-1]]:
        g, loss = oracle.mlp.grad(x0, A[idx[i, j]], y[idx[i, j]], s, BF16)
        assert rel_err_blocks(r.G[i, j].cpu().numpy(), g, mlp_blocks(*r.dims)) <= TOL_BF16
        assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)
    # every finished row: the layout padding inside P is zero, the row
    # padding beyond P untouched; unfinished rows untouched
    tail = r.Grows[:, :, s.n_params:].cpu().numpy()
    for i in range(wl.n):
        for j in range(wl.m):
            if mask[i, j]:
                assert (tail[i, j, :r.P - s.n_params] == 0).all()
                assert (tail[i, j, r.P - s.n_params:] == 7.0).all()
            else:
                assert (tail[i, j] == 7.0).all() and (r.G[i, j, :64] == 7.0).all()


def test_grad_strided_rows_match_contiguous_small_shape(tiny):
    """nbsgd_mlp_grad_strided on rows 36 floats longer than P: the same bits
    as nbsgd_mlp_grad on contiguous rows, the row padding never read (NaN in
    X) nor written (sentinel in G)."""
    wl, A, y, x0 = tiny
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    rng = np.random.default_rng(7)
    X = (x0[None, :] + 0.05 * rng.standard_normal((wl.n, s.n_params))).astype(np.float32)
    mask = (rng.random((wl.n, wl.m)) < 0.7).astype(np.uint8)
    mask[2] = 0
    mask[0, 0] = 1
    idx = rng.integers(0, wl.n_samples, size=(wl.n, wl.m, wl.batch)).astype(np.int32)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    P, ld = r.P, r.P + 36
    Xc = torch.from_numpy(pad_cols(X, P)).to(DEV)
    Gc = torch.full((wl.n, wl.m, P), 7.0, dtype=torch.float32, device=DEV)
    Lc = torch.full((wl.n * wl.m,), -1.0, dtype=torch.float32, device=DEV)
    Xs = torch.full((wl.n, ld), float("nan"), dtype=torch.float32, device=DEV)
    Xs[:, :P] = Xc
    Gs = torch.full((wl.n, wl.m, ld), 7.0, dtype=torch.float32, device=DEV)
    Ls = torch.full((wl.n * wl.m,), -1.0, dtype=torch.float32, device=DEV)
    _say(f"mlp grad strided ld={ld} P={P} finished={int(mask.sum())}")
    _lib.mlp_grad(Xc, wl.m, r.dims, r.data, r.labels, idx, mask, Gc, Lc, r.workspace)
    _lib.mlp_grad_strided(Xs, wl.m, r.dims, r.data, r.labels, idx, mask, Gs, Ls, r.workspace)
    torch.cuda.synchronize()
    assert torch.equal(Gs[:, :, :P], Gc) and torch.equal(Ls, Lc)
    assert (Gs[:, :, P:] == 7.0).all()
    Gn = Gc.cpu().numpy()
    for (i, j) in list(zip(*np.nonzero(mask)))[:3]:
        g, _ = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
        assert rel_err_blocks(Gn[i, j], g, mlp_blocks(*r.dims)) <= TOL_BF16, (i, j)


def test_training_small_shape_matches_oracle(tiny):
    wl, A, y, x0 = tiny
    _say(f"mlp training {wl.name} steps={wl.steps}")
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    step_loss, counts = [], []
    for k in range(wl.steps):
        mask, c, _ = r.step(k)
        L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
        step_loss.append(np.mean([L[i][mask[i] > 0].mean() for i in range(wl.n)]))
        counts.append(c)
    ev = float(r.evaluate().mean().cpu())
    torch.cuda.synchronize()
    ref = oracle.mlp.train(wl, A, y, x0, wl.steps)
    assert np.array_equal(np.array(counts), np.array(ref["counts"]))
    np.testing.assert_allclose(step_loss, ref["step_loss"], rtol=TOL_BF16)
    assert abs(ev - ref["eval_loss"][-1]) <= TOL_BF16 * ref["eval_loss"][-1]
    blocks = mlp_blocks(*r.dims)
    assert rel_err_blocks(r.X.cpu().numpy(), ref["X"], blocks) <= TOL_BF16
    assert rel_err_blocks(r.V.cpu().numpy(), ref["V"], blocks) <= TOL_BF16


def test_eval_loss_of_average_replica(tiny):
    wl, A, y, x0 = tiny
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    rng = np.random.default_rng(1)
    X = (x0[None, :] + 0.1 * rng.standard_normal((wl.n, s.n_params))).astype(np.float32)
    r.X.copy_(torch.from_numpy(pad_cols(X, r.P)))
    _say("mlp eval of the average replica")
    got = r.evaluate().cpu().numpy()
    ev = wl.eval_indices()
    xbar = X.astype(np.float64).mean(axis=0)
    want = [oracle.mlp.forward(xbar, A[ev[k:k + 32]], y[ev[k:k + 32]], s, BF16)[0]
            for k in range(0, len(ev), 32)]
    np.testing.assert_allclose(got, want, rtol=TOL_BF16)


def test_full_workload_trajectory_matches_golden():
    """200 iterations of the 8-learner MLP workload against the oracle's stored
    run (tests/golden/mlp_trajectory.npz, written by make_mlp_golden.py)."""
    ref = np.load(GOLDEN, allow_pickle=False)
    wl = workloads.MLP
    A, y, x0 = _data(wl)
    assert np.array_equal(np.bincount(y, minlength=wl.classes), ref["label_counts"])
    assert float(np.sum(x0, dtype=np.float64)) == float(ref["x0_sum"])
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    _say(f"mlp full workload, {wl.steps} steps")
    step_loss, counts, ev_loss = [], [], []
    for k in range(wl.steps):
        if k % wl.eval_every == 0:
            ev_loss.append(float(r.evaluate().mean().cpu()))
        mask, c, _ = r.step(k)
        L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
        step_loss.append(np.mean([L[i][mask[i] > 0].mean() for i in range(wl.n)]))
        counts.append(c)
        if k % 50 == 0:
            print(f"step {k} loss {step_loss[-1]:.5f} (oracle {ref['step_loss'][k]:.5f})", flush=True)
    ev_loss.append(float(r.evaluate().mean().cpu()))
    pos = torch.from_numpy(ref["positions"]).to(DEV)
    Xs = r.X.index_select(1, pos).cpu().numpy()
    Vs = r.V.index_select(1, pos).cpu().numpy()
    assert np.array_equal(np.array(counts), ref["counts"])
    np.testing.assert_allclose(step_loss, ref["step_loss"], rtol=TOL_BF16)
    np.testing.assert_allclose(ev_loss, ref["eval_loss"], rtol=TOL_BF16)
    assert ref["step_loss"][-1] < 0.8 * ref["step_loss"][0]  # it trains
    # Final parameters.  First-layer pre-activations within fp32 accumulation
    # error (~1e-6) of zero take different ReLU decisions on the matrix cores
    # (fp32 sums) and in the oracle (fp64 sums), a few per iteration, so the
    # 200-step parameter trajectories are not unique at the element level.
    # What must hold: the two runs end far closer to each other than to where
    # training started, block by block.
    x0s = x0[ref["positions"]][None, :].astype(np.float64)
    for name, a, b in mlp_blocks(*r.dims):
        sel = (ref["positions"] >= a) & (ref["positions"] < b)
        if sel.sum() < 2:
            continue
        gap = np.sqrt(np.mean((Xs[:, sel] - ref["X"][:, sel]) ** 2))
        moved = np.sqrt(np.mean((ref["X"][:, sel] - x0s[:, sel]) ** 2))
        print(f"final X block {name}: gpu-oracle rms {gap:.3e}, training displacement rms {moved:.3e}")
        assert gap <= 0.1 * moved, name


def test_blocking_baseline_small_shape_matches_oracle(tiny):
    """The D-PSGD baseline (every mini-batch finished, iteration time T_sync)
    on the same kernels, against the oracle's blocking run."""
    wl, A, y, x0 = tiny
    wl = dataclasses.replace(wl, delay=workloads.DelaySpec("const", 1.0, 0.0, slow_learner=-2,
                                                           slow_factor=2.0, slow_prob=0.5))
    _say(f"mlp blocking baseline {wl.name}")
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    secs, step_loss = [], []
    for k in range(wl.steps):
        mask, c, t = r.step(k, blocking=True)
        assert mask.all() and (c == wl.m).all()
        L = r.losses.cpu().numpy()
        step_loss.append(np.mean([L[i * wl.m:(i + 1) * wl.m].mean() for i in range(wl.n)]))
        secs.append(t)
    torch.cuda.synchronize()
    ref = oracle.mlp.train(wl, A, y, x0, wl.steps, blocking=True)
    assert secs == ref["seconds"]  # bitwise: same fp64 schedule on both sides
    np.testing.assert_allclose(step_loss, ref["step_loss"], rtol=TOL_BF16)
    blocks = mlp_blocks(*r.dims)
    assert rel_err_blocks(r.X.cpu().numpy(), ref["X"], blocks) <= TOL_BF16
    # the non-blocking schedule of the same iterations is never slower
    nb_secs = [runner.Schedule(wl).mask(k)[3][2] for k in range(wl.steps)]
    assert all(a <= b for a, b in zip(nb_secs, secs))


def test_grad_two_launch_groups_and_wide_indices():
    """1,024 mini-batches (16 learners x 64), more than one launch's list, on
    a data set of 70,000 samples (indices above 65,535 travel as 32-bit
    words).  Sampled entries around the group boundary and at both ends."""
    wl = dataclasses.replace(workloads.MLP_TINY, n=16, m=64, n_samples=70_000)
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    rng = np.random.default_rng(5)
    X = (x0[None, :] + 0.05 * rng.standard_normal((wl.n, s.n_params))).astype(np.float32)
    mask = np.ones((wl.n, wl.m), np.uint8)
    mask[3, 10:] = 0
    mask[15, 1:] = 0
    idx = rng.integers(0, wl.n_samples, size=(wl.n, wl.m, wl.batch)).astype(np.int32)
    idx[0, 0, :] = wl.n_samples - 1 - np.arange(wl.batch)  # the largest indices
    _say(f"mlp grad n={wl.n} m={wl.m} finished={int(mask.sum())} n_samples={wl.n_samples}")
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    Xd = torch.from_numpy(pad_cols(X, r.P)).to(DEV)
    r.G.fill_(7.0)
    _lib.mlp_grad(Xd, wl.m, r.dims, r.data, r.labels, idx, mask, r.G, r.losses, r.workspace)
    torch.cuda.synchronize()
    L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
    finished = list(zip(*np.nonzero(mask)))
    picks = [0, 1, 894, 895, 896, 897, len(finished) - 1]
    for k in picks:
        i, j = finished[k]
        g, loss = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
        assert rel_err_blocks(r.G[i, j].cpu().numpy(), g, mlp_blocks(*r.dims)) <= TOL_BF16, (k, i, j)
        assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)
    assert (r.G[3, 10:] == 7.0).all() and (r.G[15, 1:] == 7.0).all()


@pytest.mark.parametrize("dims", [(256, 128, 10), (3072, 512, 10)])
@pytest.mark.parametrize("finished", [56, 57])
def test_grad_indices_in_arguments_match_indices_through_workspace(finished, dims):
    """Up to 56 finished mini-batches travel with their sample indices in the
    forward kernel's arguments; more go through the workspace first.  Every
    mini-batch's gradient and loss depend only on its own samples and
    replica, so a call with 56 (or 57) finished and one with all 64 agree bit
    for bit on the common entries; the 64-entry call is also checked against
    the oracle on sampled entries."""
    n, m, n_samples = 8, 8, 300
    s = Shape(*dims, 32)
    A = mlp_data.inputs(11, n_samples, dims[0])
    y = mlp_data.teacher_labels(11, A, dims[1], dims[2])
    x0 = mlp_data.student_init(11, *dims)
    rng = np.random.default_rng(finished)
    X = (x0[None, :] + 0.05 * rng.standard_normal((n, s.n_params))).astype(np.float32)
    idx = rng.integers(0, n_samples, size=(n, m, 32)).astype(np.int32)
    part = np.zeros(n * m, np.uint8)
    part[rng.permutation(n * m)[:finished]] = 1
    part = part.reshape(n, m)
    full = np.ones((n, m), np.uint8)
    _say(f"mlp grad indices in arguments / workspace, dims={dims} finished={finished} and 64")
    P = _lib.mlp_param_count(*dims)
    Xd = torch.from_numpy(pad_cols(X, P)).to(DEV)
    data = torch.from_numpy(A).to(DEV)
    labels = torch.from_numpy(y.astype(np.int32)).to(DEV)
    ws = torch.empty((_lib.mlp_workspace_bytes(*dims, n * m * 32) + 15) // 16 * 4,
                     dtype=torch.float32, device=DEV)
    out = {}
    for name, mask in (("part", part), ("full", full)):
        G = torch.full((n, m, P), 7.0, dtype=torch.float32, device=DEV)
        losses = torch.full((n * m,), -1.0, dtype=torch.float32, device=DEV)
        _lib.mlp_grad(Xd, m, dims, data, labels, idx, mask, G, losses, ws)
        torch.cuda.synchronize()
        out[name] = (G.cpu().numpy(), losses.cpu().numpy().reshape(n, m))
    Gp, Lp = out["part"]
    Gf, Lf = out["full"]
    done = part.astype(bool)
    assert np.array_equal(Gp[done], Gf[done]) and np.array_equal(Lp[done], Lf[done])
    assert (Gp[~done] == 7.0).all() and (Lp[~done] == -1.0).all()
    for i, j in ((0, 0), (3, 5), (7, 7)):
        g, loss = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
        assert rel_err_blocks(Gf[i, j], g, mlp_blocks(*dims)) <= TOL_BF16, (i, j)
        assert abs(Lf[i, j] - loss) <= TOL_BF16 * abs(loss)


def test_grad_largest_16_bit_sample_index():
    """65,536 samples: every index fits 16 bits, so the indices ride in the
    forward kernel's arguments, the largest one (65,535) included."""
    wl = dataclasses.replace(workloads.MLP_TINY, n_samples=65_536)
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    rng = np.random.default_rng(9)
    X = (x0[None, :] + 0.05 * rng.standard_normal((wl.n, s.n_params))).astype(np.float32)
    mask = np.ones((wl.n, wl.m), np.uint8)
    idx = rng.integers(0, wl.n_samples, size=(wl.n, wl.m, wl.batch)).astype(np.int32)
    idx[2, 3, :] = wl.n_samples - 1 - np.arange(wl.batch)
    _say(f"mlp grad n_samples={wl.n_samples} largest index {wl.n_samples - 1}")
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    Xd = torch.from_numpy(pad_cols(X, r.P)).to(DEV)
    _lib.mlp_grad(Xd, wl.m, r.dims, r.data, r.labels, idx, mask, r.G, r.losses, r.workspace)
    torch.cuda.synchronize()
    L = r.losses.cpu().numpy().reshape(wl.n, wl.m)
    for i, j in ((2, 3), (0, 0), (wl.n - 1, wl.m - 1)):
        g, loss = oracle.mlp.grad(X[i], A[idx[i, j]], y[idx[i, j]], s, BF16)
        assert rel_err_blocks(r.G[i, j].cpu().numpy(), g, mlp_blocks(*r.dims)) <= TOL_BF16, (i, j)
        assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)


def test_loss_odd_batch_count(tiny):
    """Three batches: the forward pairs two of them in one tile and leaves
    the third alone."""
    wl, A, y, x0 = tiny
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    idx = np.random.default_rng(2).integers(0, wl.n_samples, size=3 * 32).astype(np.int32)
    out = torch.zeros(3, dtype=torch.float32, device=DEV)
    _say("mlp loss, 3 batches")
    _lib.mlp_loss(r.X[1], r.dims, r.data, r.labels, idx, out, r.workspace)
    got = out.cpu().numpy()
    want = [oracle.mlp.forward(x0, A[idx[k:k + 32]], y[idx[k:k + 32]], s, BF16)[0] for k in (0, 32, 64)]
    np.testing.assert_allclose(got, want, rtol=TOL_BF16)
