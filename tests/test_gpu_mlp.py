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
from tests._util import mlp_blocks, pad_cols

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
                assert _grad_ok(G[i, j], X[i], A[idx[i, j]], y[idx[i, j]], s, r.dims), (i, j)
                assert (G[i, j, s.n_params:] == 0).all()  # the padding
                assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)
            else:
                assert (G[i, j] == 7.0).all() and L[i, j] == -1.0


@pytest.mark.parametrize("d_in,hidden,classes", [(384, 192, 10), (640, 320, 16), (256, 512, 2),
                                                  (128, 64, 16), (768, 128, 10), (1024, 64, 5)])
def test_grad_and_loss_odd_shapes_every_entry(d_in, hidden, classes):
    """Shapes whose d_in splits into 3 or 2 slices (d_in / 64 = 6 or 10), or
    into four slices of 1, 3 or 4 chunks of 64 (d_in = 256, 768, 1024: the
    forward's pipeline tail alone; d_in = 640 and the full shape also run its
    steady loop), and
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
                assert _grad_ok(Gh[i, j], X[i], A[idx[i, j]], y[idx[i, j]], s, dims), (i, j)
                assert (Gh[i, j, s.n_params:] == 0).all()
                assert abs(Lh[i, j] - loss) <= TOL_BF16 * abs(loss)
            else:
                assert (Gh[i, j] == 7.0).all() and Lh[i, j] == -1.0
    evh = ev.cpu().numpy()
    for k in range(5):
        b = ev_idx[32 * k:32 * k + 32]
        _, loss = oracle.mlp.grad(X[2], A[b], y[b], s, BF16)
        assert abs(evh[k] - loss) <= TOL_BF16 * abs(loss), k


# Decisions taken from floating point.  Both sides multiply the same bf16
# operands exactly; the matrix cores add the products in fp32 (the forward in
# four d_in slices), the oracle in fp64, and the sums differ by about 1e-7 to
# 1e-6 at these shapes.  Where a value lies that close to a boundary, the two
# sides may decide differently:
# * the ReLU of a first-layer pre-activation within AMBIGUOUS of zero;
# * the bf16 rounding of H = relu(Z1) (within AMBIGUOUS of a rounding
#   midpoint), of dZ2 and of dZ1 (within BF16_WINDOW, relative, of one).
# The thresholds keep a twenty-fold margin over the measured differences.  A
# different decision moves the gradient entries that the value feeds by one
# sample's share (ReLU) or one bf16 step of it (rounding); those entries get
# that amount as an allowance on top of the 1e-2 bar, every other entry is
# held to the bar alone.
AMBIGUOUS = 2e-5
BF16_WINDOW = 1e-5


def _bf16_near_midpoint(v, window_rel):
    """(mask, bf16 step): entries of v whose fp32 value lies within
    window_rel * |v| of a bf16 rounding midpoint, and the bf16 spacing at v."""
    f = np.asarray(v, np.float64).astype(np.float32)
    low = (f.view(np.uint32) & np.uint32(0xFFFF)).astype(np.float64)
    fulp = np.spacing(np.abs(f)).astype(np.float64)  # fp32 spacing at v
    near = np.abs(low - 32768.0) * fulp <= window_rel * np.abs(f.astype(np.float64))
    step = fulp * 65536.0
    return near & (f != 0), step


def _flip_allowance(params, Ab, yb, s):
    """(allowance per parameter, decisions): the gradient entries each
    undetermined decision of the mini-batch feeds, with the amount a
    different decision moves them, from the oracle's own intermediates."""
    q = oracle.mlp.bf16_round
    W1, b1, W2, b2 = oracle.mlp.unpack(params, s)
    Aq, W1q, W2q = q(Ab), q(W1), q(W2)
    Z1 = Aq @ W1q + b1
    act = Z1 > 0.0
    H = np.maximum(Z1, 0.0)
    Hq = q(H)
    Z2 = Hq @ W2q + b2
    P = np.exp(Z2 - Z2.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    P[np.arange(len(yb)), yb] -= 1.0
    dZ2 = P / len(yb)
    dZ2q = q(dZ2)
    dH = dZ2q @ W2q.T
    dZ1 = dH * act
    w1, o_b1, o_w2, o_b2 = s.offsets()
    allow = np.zeros(s.n_params)
    aW1 = allow[:o_b1].reshape(s.d_in, s.hidden)
    aW2 = allow[o_w2:o_b2].reshape(s.hidden, s.classes)
    ab1 = allow[o_b1:o_w2]
    absA = np.abs(Aq)
    count = 0
    # ReLU decisions
    for r, h in zip(*np.nonzero(np.abs(Z1) < AMBIGUOUS)):
        aW1[:, h] += absA[r] * abs(dH[r, h])
        ab1[h] += abs(dH[r, h])
        aW2[h, :] += AMBIGUOUS * np.abs(dZ2q[r])
        count += 1
    # bf16 rounding of H (absolute window, the error of Z1)
    nearH, stepH = _bf16_near_midpoint(H, AMBIGUOUS / np.maximum(H, 1e-30))
    for r, h in zip(*np.nonzero(nearH)):
        aW2[h, :] += stepH[r, h] * np.abs(dZ2q[r])
        count += 1
    # bf16 rounding of dZ2
    # (dZ2 = softmax - onehot cancels for a confident class: its fp32 error is
    # absolute, about 1e-9 after the 1/b scale, so the window has that floor)
    nearZ, stepZ = _bf16_near_midpoint(dZ2, np.maximum(BF16_WINDOW, 2e-8 / np.maximum(np.abs(dZ2), 1e-30)))
    for r, c in zip(*np.nonzero(nearZ)):
        aW2[:, c] += stepZ[r, c] * Hq[r]
        feed = stepZ[r, c] * np.abs(W2q[:, c]) * act[r]  # dH[r, :] moves by this
        aW1 += np.outer(absA[r], feed)
        ab1 += feed
        count += 1
    # bf16 rounding of dZ1
    nearD, stepD = _bf16_near_midpoint(dZ1, BF16_WINDOW)
    for r, h in zip(*np.nonzero(nearD)):
        aW1[:, h] += absA[r] * stepD[r, h]
        count += 1
    allow *= 1.01
    return allow, count


def _allowance_is_the_exception(allow, want, blocks, hidden):
    """Few of each block's entries get an allowance larger than the bar
    itself: at most 1% of them, or two hidden units' worth (a ReLU decision
    covers a unit's whole dW1 column)."""
    for _, a, b in blocks:
        w = want[..., a:b]
        rms = float(np.sqrt(np.mean(w * w))) or 1.0
        assert float(np.mean(allow[..., a:b] > TOL_BF16 * rms)) <= max(0.01, 2.0 / hidden)


def _within(got, want, blocks, allow=None):
    """Element-wise bar: |got - want| <= 1e-2 * max(|want|, rms of want's
    block) + allowance, for every element of every block."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    worst = 0.0
    for _, a, b in blocks:
        w = want[..., a:b]
        rms = float(np.sqrt(np.mean(w * w))) or 1.0
        excess = np.abs(got[..., a:b] - w) - (0.0 if allow is None else allow[..., a:b])
        worst = max(worst, float(np.max(excess / np.maximum(np.abs(w), rms))))
    return worst <= TOL_BF16, worst


def _grad_ok(got, params, Ab, yb, s, dims):
    """One mini-batch gradient against the oracle's at the same parameters:
    element-wise at 1e-2 per block, with the undetermined decisions'
    allowances."""
    g, _ = oracle.mlp.grad(params, Ab, yb, s, BF16)
    allow, _ = _flip_allowance(params, Ab, yb, s)
    _allowance_is_the_exception(allow, g, mlp_blocks(*dims), s.hidden)
    ok, worst = _within(np.asarray(got)[:s.n_params], g, mlp_blocks(*dims), allow)
    return ok


def test_grad_full_shape_every_entry():
    """The full shape in the runner's launch configuration (padded rows,
    row_stride(P) = 2^21 floats apart, nbsgd_mlp_grad_strided): every
    finished mini-batch's gradient, element by element, and its loss against
    the oracle."""
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
    G = r.G.cpu().numpy()
    blocks = mlp_blocks(*r.dims)
    for i, j in zip(*np.nonzero(mask)):
        g, loss = oracle.mlp.grad(x0, A[idx[i, j]], y[idx[i, j]], s, BF16)
        allow, _ = _flip_allowance(x0, A[idx[i, j]], y[idx[i, j]], s)
        _allowance_is_the_exception(allow, g, blocks, wl.hidden)
        ok, worst = _within(G[i, j, :s.n_params], g, blocks, allow)
        assert ok, (i, j, worst)
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
                assert (tail[i, j] == 7.0).all() and (G[i, j, :64] == 7.0).all()


def _iteration_from_common_state(wl, k, A, y, x0):
    """One whole iteration of an MLP workload (gradients of every finished
    mini-batch on the matrix cores, then the fused step) from a state both
    sides share: the initial replicas (k = 0) or the oracle's own state after
    k iterations, rounded to fp32 and given to both.  Every finished G row and
    loss, and X and V, element by element against one oracle iteration, with
    the allowances of the undetermined decisions (_flip_allowance) carried
    through the step."""
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    if k == 0:
        X = np.tile(x0.astype(np.float64), (wl.n, 1))
        V = np.zeros_like(X)
    else:
        ref = oracle.mlp.train(wl, A, y, x0, k, evaluate=False)
        X, V = ref["X"], ref["V"]
    X32, V32 = X.astype(np.float32), V.astype(np.float32)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    r.X[:, :s.n_params] = torch.from_numpy(X32).to(DEV)
    r.V[:, :s.n_params] = torch.from_numpy(V32).to(DEV)
    mask, counts, _ = r.step(k)
    torch.cuda.synchronize()
    G = r.G.cpu().numpy()
    Xg, Vg = r.X.cpu().numpy(), r.V.cpu().numpy()
    L = r.losses.cpu().numpy().reshape(wl.n, wl.m)

    sch = oracle.schedule.sample_schedule(wl.seed, k, wl.n, wl.m, oracle.workload.delay(wl))
    assert np.array_equal(sch["mask"], mask)
    shuf = oracle.mlp.Shuffler(wl.seed, wl.shard, wl.m, wl.batch)
    Xs, Vs = X32.astype(np.float64), V32.astype(np.float64)
    Go = np.zeros((wl.n, wl.m, s.n_params))
    allow_v = np.zeros((wl.n, s.n_params))
    blocks = mlp_blocks(*r.dims)
    for i in range(wl.n):
        rows = shuf.indices(k, i)
        for j in range(wl.m):
            if not mask[i, j]:
                continue
            Go[i, j], loss = oracle.mlp.grad(Xs[i], A[rows[j]], y[rows[j]], s, BF16)
            allow, _ = _flip_allowance(Xs[i], A[rows[j]], y[rows[j]], s)
            _allowance_is_the_exception(allow, Go[i, j], blocks, wl.hidden)
            ok, worst = _within(G[i, j, :s.n_params], Go[i, j], blocks, allow)
            assert ok, ("G", i, j, worst)
            assert abs(L[i, j] - loss) <= TOL_BF16 * abs(loss)
            allow_v[i] += allow / counts[i]
    W = oracle.workload.mixer(wl).w(k)
    lr, mu = float(np.float32(wl.lr)), float(np.float32(wl.momentum))
    order = oracle.workload.order(wl)
    Xo, Vo = oracle.step.step(Xs, Vs, Go, mask, W, lr, mu, order)
    ok, worst = _within(Vg[:, :s.n_params], Vo, blocks, allow_v)
    assert ok, ("V", worst)
    eta_allow = (lr * counts / wl.m)[:, None] * allow_v
    if order == oracle.step.STEP_THEN_MIX:  # the stepped rows are mixed
        eta_allow = np.abs(W) @ eta_allow
    ok, worst = _within(Xg[:, :s.n_params], Xo, blocks, eta_allow)
    assert ok, ("X", worst)
    assert (Xg[:, s.n_params:] == 0).all() and (Vg[:, s.n_params:] == 0).all()


@pytest.mark.parametrize("k", [0, 12])
def test_full_shape_iteration_from_common_state(k):
    """The full workload (D-PSGD ring), from its initial replicas and from the
    oracle's state after 12 iterations."""
    wl = workloads.MLP
    _say(f"mlp full-shape iteration {k} from a common state")
    _iteration_from_common_state(wl, k, *_data(wl))


@pytest.mark.parametrize("kind", ["ring", "matcha", "uniform"])
@pytest.mark.parametrize("k", [0, 7, 11])
def test_small_shape_iteration_from_common_state(tiny, kind, k):
    """Each mixing kind (D-PSGD ring, MATCHA, all-reduce with uniform W) on
    the small workload, from the oracle's own states along its run."""
    wl, A, y, x0 = tiny
    wl = workloads.mlp_with_mixing(wl, kind)
    _say(f"mlp {wl.name} iteration {k} from a common state")
    _iteration_from_common_state(wl, k, A, y, x0)


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
        assert _grad_ok(Gn[i, j], X[i], A[idx[i, j]], y[idx[i, j]], s, r.dims), (i, j)


@pytest.mark.parametrize("kind", ["ring", "matcha", "uniform"])
def test_training_small_shape_matches_oracle(tiny, kind):
    """Non-blocking training under each mixing kind (D-PSGD ring, MATCHA,
    all-reduce with uniform W) against the oracle's run of the same
    workload."""
    wl, A, y, x0 = tiny
    wl = workloads.mlp_with_mixing(wl, kind)
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
    # Over a trajectory the element-level parameters are not unique: a ReLU
    # or bf16 rounding decision taken differently (see AMBIGUOUS) moves a
    # unit's parameters, which moves that unit's pre-activations of later
    # samples, and a unit whose pre-activations hover near zero amplifies
    # that from step to step.  The element-wise bar is held one iteration at
    # a time from common states (test_small_shape_iteration_from_common_state);
    # here X and V are compared block by block by their rms gap, at 1e-2 of
    # the parameters (X) and 5% of the momentum (V).
    for name, a, b in mlp_blocks(*r.dims):
        for got, want, bar in ((r.X.cpu().numpy()[:, a:b], ref["X"][:, a:b], TOL_BF16),
                               (r.V.cpu().numpy()[:, a:b], ref["V"][:, a:b], 0.05)):
            gap = np.sqrt(np.mean((got - want) ** 2))
            assert gap <= bar * np.sqrt(np.mean(want ** 2)), (name, gap)


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


@pytest.mark.parametrize("kind", ["ring", "matcha", "uniform"])
def test_blocking_baseline_small_shape_matches_oracle(tiny, kind):
    """The synchronous baselines (D-PSGD, MATCHA, all-reduce: every
    mini-batch finished, iteration time T_sync) on the same kernels, against
    the oracle's blocking run."""
    wl, A, y, x0 = tiny
    wl = dataclasses.replace(workloads.mlp_with_mixing(wl, kind),
                             delay=workloads.DelaySpec("const", 1.0, 0.0, slow_learner=-2,
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
    # parameters by their rms gap per block (the trajectory is not unique at
    # the element level, see test_training_small_shape_matches_oracle)
    for name, a, b in mlp_blocks(*r.dims):
        got, want = r.X.cpu().numpy()[:, a:b], ref["X"][:, a:b]
        assert np.sqrt(np.mean((got - want) ** 2)) <= TOL_BF16 * np.sqrt(np.mean(want ** 2)), name
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
        assert _grad_ok(r.G[i, j].cpu().numpy(), X[i], A[idx[i, j]], y[idx[i, j]], s, r.dims), (k, i, j)
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
        assert _grad_ok(Gf[i, j], X[i], A[idx[i, j]], y[idx[i, j]], s, dims), (i, j)
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
        assert _grad_ok(r.G[i, j].cpu().numpy(), X[i], A[idx[i, j]], y[idx[i, j]], s, r.dims), (i, j)
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
