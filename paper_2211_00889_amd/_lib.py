"""ctypes binding of libnbsgd.so: argument marshalling only.

Every computation happens in the library (host C++ for the schedule and the
mixing matrices, gfx950 kernels for the step).  Device arrays are PyTorch CUDA
tensors used as plain device memory; the stream defaults to torch's current
stream on the tensor's device.  A missing library raises at import time of the
first call, never falls back to anything else.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnbsgd.so")

OK, E_ARG, E_SHAPE, E_ALIGN, E_MASK, E_W, E_HIP, E_UNSUPPORTED = range(8)
MIX_THEN_STEP, STEP_THEN_MIX = 0, 1
DELAY_CONST, DELAY_EXP, DELAY_LOMAX = 0, 1, 2
MAX_LEARNERS, MAX_MINIBATCHES = 16, 64
SLOW_NONE, SLOW_RANDOM = -1, -2

EXPORTS = ("nbsgd_sample_mask", "nbsgd_iteration_accounting", "nbsgd_accumulate", "nbsgd_mix", "nbsgd_update", "nbsgd_step",
           "nbsgd_step_strided", "nbsgd_step_server", "nbsgd_row_stride",
           "nbsgd_w_allreduce", "nbsgd_w_ring", "nbsgd_matcha_create", "nbsgd_matcha_w",
           "nbsgd_matcha_matchings", "nbsgd_matcha_set", "nbsgd_matcha_get", "nbsgd_matcha_optimize",
           "nbsgd_matcha_destroy", "nbsgd_mlp_param_count",
           "nbsgd_mlp_workspace_bytes", "nbsgd_minibatch_indices", "nbsgd_mlp_grad",
           "nbsgd_mlp_grad_strided", "nbsgd_mlp_grad_noalloc", "nbsgd_mlp_loss",
           "nbsgd_last_error")


class NbsgdError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"nbsgd status {status}: {message}")
        self.status = status


class MlpShape(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("hidden", ctypes.c_int32), ("classes", ctypes.c_int32),
                ("batch", ctypes.c_int32)]


class Delay(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("base", ctypes.c_double), ("param", ctypes.c_double),
                ("slow_learner", ctypes.c_int32), ("slow_factor", ctypes.c_double),
                ("slow_prob", ctypes.c_double)]


class Accounting(ctypes.Structure):
    _fields_ = [(k, ctypes.c_double) for k in ("x_first", "x_last", "y", "throughput",
                                                 "throughput_sync", "data", "ratio")]


_c_void_p, _i32, _i64, _u64, _f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                     ctypes.c_uint64, ctypes.c_float)
_lib = None


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "nbsgd_sample_mask": [_u64, _u64, _i32, _i32, ctypes.POINTER(Delay), _c_void_p, _c_void_p,
                              _c_void_p, _c_void_p],
        "nbsgd_iteration_accounting": [_c_void_p, _i32, _i32, ctypes.POINTER(Accounting)],
        "nbsgd_accumulate": [_c_void_p, _c_void_p, _i32, _i32, _i64, _c_void_p, _c_void_p],
        "nbsgd_mix": [_c_void_p, _c_void_p, _i32, _i64, _c_void_p, _c_void_p],
        "nbsgd_update": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _i32, _i32, _i64, _f32, _f32,
                         _c_void_p],
        "nbsgd_step": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _i32, _i32, _i64,
                       _f32, _f32, _i32, _c_void_p],
        "nbsgd_step_strided": [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _c_void_p, _i32, _i32,
                               _i64, _f32, _f32, _i32, _c_void_p],
        "nbsgd_step_server": [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _i32, _i32, _i64, _f32,
                              _f32, _c_void_p],
        "nbsgd_row_stride": [_i64, ctypes.POINTER(_i64)],
        "nbsgd_w_allreduce": [_i32, _c_void_p],
        "nbsgd_w_ring": [_i32, _c_void_p],
        "nbsgd_matcha_create": [_u64, _i32, _i32, ctypes.POINTER(_c_void_p)],
        "nbsgd_matcha_w": [_c_void_p, _u64, _c_void_p, _c_void_p],
        "nbsgd_matcha_matchings": [_c_void_p, _c_void_p, _c_void_p, _c_void_p],
        "nbsgd_matcha_set": [_c_void_p, _c_void_p, ctypes.c_double],
        "nbsgd_matcha_get": [_c_void_p, _c_void_p, _c_void_p],
        "nbsgd_matcha_optimize": [_c_void_p, ctypes.c_double, _i32, _c_void_p, _c_void_p],
        "nbsgd_mlp_param_count": [ctypes.POINTER(MlpShape), ctypes.POINTER(_i64)],
        "nbsgd_mlp_workspace_bytes": [ctypes.POINTER(MlpShape), _i64, ctypes.POINTER(ctypes.c_size_t)],
        "nbsgd_minibatch_indices": [_u64, _u64, _i32, _i32, _i32, _i32, _c_void_p],
        "nbsgd_mlp_grad": [_c_void_p, _i32, _i32, ctypes.POINTER(MlpShape), _c_void_p, _c_void_p, _i64,
                           _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, ctypes.c_size_t,
                           _c_void_p],
        "nbsgd_mlp_grad_strided": [_c_void_p, _i64, _i32, _i32, ctypes.POINTER(MlpShape), _c_void_p,
                                   _c_void_p, _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                   _c_void_p, ctypes.c_size_t, _c_void_p],
        "nbsgd_mlp_grad_noalloc": [_c_void_p, _i64, _i32, _i32, ctypes.POINTER(MlpShape), _c_void_p,
                                   _c_void_p, _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                   _c_void_p],
        "nbsgd_mlp_loss": [_c_void_p, ctypes.POINTER(MlpShape), _c_void_p, _c_void_p, _i64, _c_void_p,
                           _i32, _c_void_p, _c_void_p, ctypes.c_size_t, _c_void_p],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.nbsgd_matcha_destroy.argtypes = [_c_void_p]
    lib.nbsgd_matcha_destroy.restype = None
    lib.nbsgd_last_error.argtypes = []
    lib.nbsgd_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != OK:
        raise NbsgdError(status, load().nbsgd_last_error().decode())


def _host_ptr(a: np.ndarray):
    return a.ctypes.data_as(_c_void_p)


def _dev(t, name):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous float32")
    return _c_void_p(t.data_ptr())


def _stream(t, stream):
    import torch

    if stream is None:
        return _c_void_p(torch.cuda.current_stream(t.device).cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return _c_void_p(stream.cuda_stream)
    return _c_void_p(int(stream))


def _u8(a, shape):
    a = np.ascontiguousarray(np.asarray(a), dtype=np.uint8)
    if a.shape != shape:
        raise ValueError(f"expected shape {shape}, got {a.shape}")
    return a


def _w32(W, n):
    W = np.ascontiguousarray(np.asarray(W), dtype=np.float32)
    if W.shape != (n, n):
        raise ValueError(f"W must be {n}x{n}")
    return W


# ------------------------------------------------------------------ host calls
def sample_mask(seed: int, step: int, n: int, m: int, kind: int, base: float = 1.0,
                param: float = 1.0, slow_learner: int = -1, slow_factor: float = 1.0,
                slow_prob: float = 0.0):
    """Returns (mask uint8[n, m], counts int32[n], times f64[n, m], timing f64[3])."""
    d = Delay(kind, base, param, slow_learner, slow_factor, slow_prob)
    mask = np.zeros((max(n, 0), max(m, 0)), np.uint8)
    counts = np.zeros(max(n, 0), np.int32)
    times = np.zeros((max(n, 0), max(m, 0)), np.float64)
    timing = np.zeros(3, np.float64)
    _check(load().nbsgd_sample_mask(seed, step, n, m, ctypes.byref(d), _host_ptr(mask),
                                    _host_ptr(counts), _host_ptr(times), _host_ptr(timing)))
    return mask, counts, times, timing


def iteration_accounting(times) -> dict:
    """Sec. 4.3 accounting (Thm 3-5, Cor. 1) of one iteration's per-mini-batch
    times [n, m]; returns the fields of nbsgd_accounting as a dict."""
    times = np.ascontiguousarray(np.asarray(times), dtype=np.float64)
    if times.ndim != 2:
        raise ValueError("times must be [n, m]")
    n, m = times.shape
    a = Accounting()
    _check(load().nbsgd_iteration_accounting(_host_ptr(times), n, m, ctypes.byref(a)))
    return {k: getattr(a, k) for k, _ in Accounting._fields_}


def w_allreduce(n: int) -> np.ndarray:
    W = np.zeros((max(n, 0), max(n, 0)), np.float32)
    _check(load().nbsgd_w_allreduce(n, _host_ptr(W)))
    return W


def w_ring(n: int) -> np.ndarray:
    W = np.zeros((max(n, 0), max(n, 0)), np.float32)
    _check(load().nbsgd_w_ring(n, _host_ptr(W)))
    return W


class Matcha:
    """Owner of an nbsgd_matcha handle."""

    def __init__(self, seed: int, n: int, degree: int):
        self.n = n
        h = _c_void_p()
        _check(load().nbsgd_matcha_create(seed, n, degree, ctypes.byref(h)))
        self._h = h

    def w(self, step: int):
        W = np.zeros((self.n, self.n), np.float32)
        active = ctypes.c_int32(0)
        _check(load().nbsgd_matcha_w(self._h, step, _host_ptr(W), ctypes.byref(active)))
        return W, active.value

    def matchings(self):
        E, M = ctypes.c_int32(0), ctypes.c_int32(0)
        _check(load().nbsgd_matcha_matchings(self._h, None, ctypes.byref(E), ctypes.byref(M)))
        buf = np.zeros((E.value, 3), np.int32)
        _check(load().nbsgd_matcha_matchings(self._h, _host_ptr(buf), ctypes.byref(E),
                                             ctypes.byref(M)))
        return buf, M.value

    def set(self, probs, alpha: float):
        probs = np.ascontiguousarray(np.asarray(probs), dtype=np.float64)
        _check(load().nbsgd_matcha_set(self._h, _host_ptr(probs), float(alpha)))

    def get(self):
        _, M = self.matchings()
        probs = np.zeros(M, np.float64)
        alpha = ctypes.c_double(0.0)
        _check(load().nbsgd_matcha_get(self._h, _host_ptr(probs), ctypes.byref(alpha)))
        return probs, alpha.value

    def optimize(self, budget: float, iterations: int = 2000):
        """MATCHA's own activation probabilities and alpha; returns
        (lambda_2, spectral norm) attained."""
        l2, rho = ctypes.c_double(0.0), ctypes.c_double(0.0)
        _check(load().nbsgd_matcha_optimize(self._h, budget, iterations, ctypes.byref(l2),
                                            ctypes.byref(rho)))
        return l2.value, rho.value

    def close(self):
        if getattr(self, "_h", None):
            load().nbsgd_matcha_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()


# ---------------------------------------------------------------- device calls
def accumulate(G, mask, Gbar, stream=None):
    n, m, P = G.shape
    mask = _u8(mask, (n, m))
    if tuple(Gbar.shape) != (n, P):
        raise ValueError("Gbar must be [n, P]")
    _check(load().nbsgd_accumulate(_dev(G, "G"), _host_ptr(mask), n, m, P, _dev(Gbar, "Gbar"),
                                   _stream(G, stream)))


def mix(X, W, Y, stream=None):
    n, P = X.shape
    W = _w32(W, n)
    if tuple(Y.shape) != (n, P):
        raise ValueError("Y must be [n, P]")
    _check(load().nbsgd_mix(_dev(X, "X"), _host_ptr(W), n, P, _dev(Y, "Y"), _stream(X, stream)))


def update(X, V, Gbar, counts, m: int, lr: float, momentum: float, stream=None):
    n, P = X.shape
    counts = np.ascontiguousarray(np.asarray(counts), dtype=np.int32)
    if counts.shape != (n,) or tuple(V.shape) != (n, P) or tuple(Gbar.shape) != (n, P):
        raise ValueError("shape mismatch")
    _check(load().nbsgd_update(_dev(X, "X"), _dev(V, "V"), _dev(Gbar, "Gbar"), _host_ptr(counts),
                               n, m, P, lr, momentum, _stream(X, stream)))


def step(X, V, G, mask, W, lr: float, momentum: float, order: int, stream=None):
    n, m, P = G.shape
    if tuple(X.shape) != (n, P) or tuple(V.shape) != (n, P):
        raise ValueError("X and V must be [n, P] with G [n, m, P]")
    mask = _u8(mask, (n, m))
    W = _w32(W, n)
    _check(load().nbsgd_step(_dev(X, "X"), _dev(V, "V"), _dev(G, "G"), _host_ptr(mask),
                             _host_ptr(W), n, m, P, lr, momentum, order, _stream(X, stream)))


def step_strided(X, V, G, P: int, mask, W, lr: float, momentum: float, order: int, stream=None):
    """nbsgd_step on padded rows: X, V [n, ld], G [n, m, ld]; the first P
    columns of each row are the parameters."""
    n, m, ld = G.shape
    if tuple(X.shape) != (n, ld) or tuple(V.shape) != (n, ld):
        raise ValueError("X and V must be [n, ld] with G [n, m, ld]")
    mask = _u8(mask, (n, m))
    W = _w32(W, n)
    _check(load().nbsgd_step_strided(_dev(X, "X"), _dev(V, "V"), _dev(G, "G"), ld, _host_ptr(mask),
                                     _host_ptr(W), n, m, P, lr, momentum, order, _stream(X, stream)))


def step_server(x, V, G, P: int, mask, lr: float, momentum: float, stream=None):
    """nbsgd_step_server: x [ld] or [P] (the server model), V [n, ld],
    G [n, m, ld]; the first P columns of each row are the parameters."""
    n, m, ld = G.shape
    if tuple(V.shape) != (n, ld) or x.dim() != 1 or x.shape[0] < P:
        raise ValueError("V must be [n, ld] and x hold P floats, with G [n, m, ld]")
    mask = _u8(mask, (n, m))
    _check(load().nbsgd_step_server(_dev(x, "x"), _dev(V, "V"), _dev(G, "G"), ld, _host_ptr(mask), n, m,
                                    P, lr, momentum, _stream(x, stream)))


def row_stride(P: int) -> int:
    ld = _i64(0)
    _check(load().nbsgd_row_stride(P, ctypes.byref(ld)))
    return ld.value


# ------------------------------------------------------------ MLP workload
def _shape(d_in, hidden, classes, batch=32):
    return MlpShape(d_in, hidden, classes, batch)


def mlp_param_count(d_in: int, hidden: int, classes: int, batch: int = 32) -> int:
    P = _i64(0)
    _check(load().nbsgd_mlp_param_count(ctypes.byref(_shape(d_in, hidden, classes, batch)),
                                        ctypes.byref(P)))
    return P.value


def mlp_workspace_bytes(d_in: int, hidden: int, classes: int, rows: int, batch: int = 32) -> int:
    b = ctypes.c_size_t(0)
    _check(load().nbsgd_mlp_workspace_bytes(ctypes.byref(_shape(d_in, hidden, classes, batch)), rows,
                                            ctypes.byref(b)))
    return b.value


def minibatch_indices(seed: int, step: int, n: int, m: int, b: int, shard: int) -> np.ndarray:
    idx = np.zeros((max(n, 0), max(m, 0), max(b, 0)), np.int32)
    _check(load().nbsgd_minibatch_indices(seed, step, n, m, b, shard, _host_ptr(idx)))
    return idx


def _i32_dev(t, name):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.int32 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous int32 CUDA tensor")
    return _c_void_p(t.data_ptr())


def _ws(t):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise TypeError("workspace must be a contiguous CUDA tensor")
    return _c_void_p(t.data_ptr()), t.numel() * t.element_size()


def _mlp_grad_args(X, m, dims, data, labels, idx, mask, G, losses, ld):
    n = X.shape[0]
    if X.dim() != 2 or X.shape[1] != ld or tuple(G.shape) != (n, m, ld):
        raise ValueError(f"X must be [n, {ld}] and G [n, m, {ld}]")
    if losses.numel() < n * m:
        raise ValueError("losses must hold n*m entries")
    idx = np.ascontiguousarray(np.asarray(idx), dtype=np.int32)
    if idx.size != n * m * 32:
        raise ValueError("idx must hold n*m*32 sample indices")
    if data.dim() != 2 or data.shape[1] != dims[0] or labels.numel() < data.shape[0]:
        raise ValueError("data must be [n_samples, d_in] with a label per sample")
    return n, idx, _u8(mask, (n, m))


def mlp_grad(X, m: int, dims, data, labels, idx, mask, G, losses, workspace, stream=None):
    """dims = (d_in, hidden, classes); X [n, P]; G [n, m, P]; idx host int32
    [n, m, 32]; mask host [n, m]."""
    n, idx, mask = _mlp_grad_args(X, m, dims, data, labels, idx, mask, G, losses,
                                  mlp_param_count(*dims))
    ws, ws_bytes = _ws(workspace)
    _check(load().nbsgd_mlp_grad(_dev(X, "X"), n, m, ctypes.byref(_shape(*dims)), _dev(data, "data"),
                                 _i32_dev(labels, "labels"), data.shape[0], _host_ptr(idx),
                                 _host_ptr(mask), _dev(G, "G"), _dev(losses, "losses"), ws, ws_bytes,
                                 _stream(X, stream)))


def mlp_grad_strided(X, m: int, dims, data, labels, idx, mask, G, losses, workspace, stream=None):
    """nbsgd_mlp_grad on padded rows: X [n, ld], G [n, m, ld] (the layout of
    step_strided); the first P columns of each row are the parameters."""
    ld = X.shape[-1]
    n, idx, mask = _mlp_grad_args(X, m, dims, data, labels, idx, mask, G, losses, ld)
    ws, ws_bytes = _ws(workspace)
    _check(load().nbsgd_mlp_grad_strided(_dev(X, "X"), ld, n, m, ctypes.byref(_shape(*dims)),
                                         _dev(data, "data"), _i32_dev(labels, "labels"),
                                         data.shape[0], _host_ptr(idx), _host_ptr(mask), _dev(G, "G"),
                                         _dev(losses, "losses"), ws, ws_bytes, _stream(X, stream)))


def mlp_grad_noalloc(X, m: int, dims, data, labels, idx, mask, G, losses, stream=None):
    """nbsgd_mlp_grad_noalloc: mlp_grad_strided with the library's static
    device scratch buffer as the workspace (no workspace argument)."""
    ld = X.shape[-1]
    n, idx, mask = _mlp_grad_args(X, m, dims, data, labels, idx, mask, G, losses, ld)
    _check(load().nbsgd_mlp_grad_noalloc(_dev(X, "X"), ld, n, m, ctypes.byref(_shape(*dims)),
                                         _dev(data, "data"), _i32_dev(labels, "labels"),
                                         data.shape[0], _host_ptr(idx), _host_ptr(mask), _dev(G, "G"),
                                         _dev(losses, "losses"), _stream(X, stream)))


MLP_SCRATCH_BYTES = 32 * 1024 * 1024


def mlp_loss(params, dims, data, labels, idx, losses, workspace, stream=None):
    """Mean loss of ``params`` on the samples ``idx`` (host int32), per 32."""
    idx = np.ascontiguousarray(np.asarray(idx), dtype=np.int32).reshape(-1)
    ws, ws_bytes = _ws(workspace)
    _check(load().nbsgd_mlp_loss(_dev(params, "params"), ctypes.byref(_shape(*dims)), _dev(data, "data"),
                                 _i32_dev(labels, "labels"), data.shape[0], _host_ptr(idx), idx.size,
                                 _dev(losses, "losses"), ws, ws_bytes, _stream(params, stream)))
