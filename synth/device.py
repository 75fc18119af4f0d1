"""ctypes binding of ``libsynth.so`` (built from ``fill.hip``): fills device
tensors in place with exactly the values ``gen.normal_f32`` / ``gen.uniform_f32``
return for the same (seed, stream, flat index)."""

from __future__ import annotations

import ctypes
import os

from .gen import normal_scale, splitmix_key, uniform_scale

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(LIB_PATH)
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64,
                                   ctypes.c_float, ctypes.c_int, ctypes.c_void_p]
        _lib = lib
    return _lib


def _fill(t, seed, stream, scale, kind, first, stream_handle):
    import torch

    if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
        raise ValueError("expected a contiguous float32 CUDA tensor")
    if stream_handle is None:
        stream_handle = torch.cuda.current_stream(t.device).cuda_stream
    rc = _load().synth_fill(ctypes.c_void_p(t.data_ptr()), t.numel(), first,
                            splitmix_key(seed, stream), float(scale), kind,
                            ctypes.c_void_p(stream_handle))
    if rc != 0:
        raise RuntimeError(f"synth_fill failed with hipError {rc}")
    return t


def fill_normal(t, seed: int, stream: int, std: float, first: int = 0, stream_handle=None):
    return _fill(t, seed, stream, normal_scale(std), 0, first, stream_handle)


def fill_uniform(t, seed: int, stream: int, half_width: float, first: int = 0, stream_handle=None):
    return _fill(t, seed, stream, uniform_scale(half_width), 1, first, stream_handle)
