"""nbsgd_mlp_grad_noalloc (the gradient call whose workspace is the library's
static device buffer) against nbsgd_mlp_grad_strided with a caller workspace,
through the C ABI: bit for bit on every finished row and loss, unfinished
rows untouched, over consecutive calls (the full MLP shape, then a smaller
shape and mask, then the full shape again with another mask), and the
rejection of a request that needs more workspace than the buffer holds."""

import numpy as np
import pytest

from paper_2211_00889_amd import _lib, runner
from synth import mlp_data, workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _inputs(wl, noise_seed):
    A = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(wl.seed, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    rng = np.random.default_rng(noise_seed)
    X = (x0[None, :] + 0.05 * rng.standard_normal((wl.n, x0.size))).astype(np.float32)
    return A, y, x0, X


def _both(r, X, mask, idx):
    """(G, losses) of the workspace call and of the allocation-free call on
    the same inputs, each into sentinel-filled buffers in the runner's
    row-strided layout."""
    wl = r.wl
    P, ld = r.P, r.ld
    Xd = torch.zeros((wl.n, ld), dtype=torch.float32, device=DEV)
    Xd[:, :X.shape[1]] = torch.from_numpy(X).to(DEV)
    out = []
    for call in ("workspace", "noalloc"):
        G = torch.full((wl.n, wl.m, ld), 7.0, dtype=torch.float32, device=DEV)
        L = torch.full((wl.n * wl.m,), -1.0, dtype=torch.float32, device=DEV)
        if call == "workspace":
            _lib.mlp_grad_strided(Xd, wl.m, r.dims, r.data, r.labels, idx, mask, G, L, r.workspace)
        else:
            _lib.mlp_grad_noalloc(Xd, wl.m, r.dims, r.data, r.labels, idx, mask, G, L)
        torch.cuda.synchronize()
        out.append((G[:, :, :P].cpu().numpy(), G[:, :, P:].cpu().numpy(), L.cpu().numpy()))
    return out


def _check(out, mask):
    (Gw, Tw, Lw), (Gn, Tn, Ln) = out
    done = mask.astype(bool)
    assert np.array_equal(Gn[done], Gw[done]), "finished rows differ from the workspace call"
    assert np.array_equal(Ln.reshape(mask.shape)[done], Lw.reshape(mask.shape)[done])
    assert (Gn[~done] == 7.0).all() and (Ln.reshape(mask.shape)[~done] == -1.0).all()
    assert (Tn == 7.0).all() and (Tw == 7.0).all()  # row padding beyond P never written


def test_noalloc_matches_workspace_call_on_consecutive_calls():
    full = workloads.MLP
    A, y, x0, X = _inputs(full, 1)
    r = runner.MlpRunner(full, DEV, A, y, x0)
    sched = runner.Schedule(full)
    mask, _, _, _ = sched.mask(0)
    idx = _lib.minibatch_indices(full.seed, 0, full.n, full.m, full.batch, full.shard)
    _say(f"noalloc call 1: full shape, finished={int(mask.sum())}")
    _check(_both(r, X, mask, idx), mask)

    tiny = workloads.MLP_TINY
    At, yt, x0t, Xt = _inputs(tiny, 2)
    rt = runner.MlpRunner(tiny, DEV, At, yt, x0t)
    rng = np.random.default_rng(3)
    mask_t = (rng.random((tiny.n, tiny.m)) < 0.5).astype(np.uint8)
    mask_t[0, 2] = 1
    idx_t = rng.integers(0, tiny.n_samples, size=(tiny.n, tiny.m, tiny.batch)).astype(np.int32)
    _say(f"noalloc call 2: shape {tiny.d_in}x{tiny.hidden}x{tiny.classes}, "
         f"finished={int(mask_t.sum())}")
    _check(_both(rt, Xt, mask_t, idx_t), mask_t)

    mask3 = np.ones((full.n, full.m), np.uint8)
    mask3[5, 3:] = 0
    idx3 = _lib.minibatch_indices(full.seed, 1, full.n, full.m, full.batch, full.shard)
    _say(f"noalloc call 3: full shape, finished={int(mask3.sum())}")
    _check(_both(r, X, mask3, idx3), mask3)


def test_noalloc_rejects_more_than_its_buffer_holds():
    """128 finished mini-batches of a 512-unit hidden layer need more than
    the 32 MiB buffer: refused before anything is enqueued."""
    wl = workloads.MlpWorkload("noalloc_limit", n=16, m=8, d_in=128, hidden=512, classes=10,
                               n_samples=16 * 256)
    A, y, x0, X = _inputs(wl, 4)
    r = runner.MlpRunner(wl, DEV, A, y, x0)
    need = _lib.mlp_workspace_bytes(wl.d_in, wl.hidden, wl.classes, 128 * 32)
    assert need > _lib.MLP_SCRATCH_BYTES
    mask = np.ones((wl.n, wl.m), np.uint8)
    idx = np.zeros((wl.n, wl.m, 32), np.int32)
    r.Grows.fill_(7.0)
    _say("noalloc: request above the static buffer")
    with pytest.raises(_lib.NbsgdError) as e:
        _lib.mlp_grad_noalloc(r.Xrows, wl.m, r.dims, r.data, r.labels, idx, mask, r.Grows, r.losses)
    assert e.value.status == _lib.E_UNSUPPORTED and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (r.Grows == 7.0).all()
    # 113 finished fit the buffer and match the workspace call
    mask[:] = 0
    mask.reshape(-1)[:113] = 1
    idx = np.random.default_rng(6).integers(0, wl.n_samples, size=(wl.n, wl.m, 32)).astype(np.int32)
    _say("noalloc: 113 finished mini-batches, hidden 512")
    _check(_both(r, X, mask, idx), mask)
