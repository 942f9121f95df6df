"""Binding of the device input generator and copy kernel (synth/synth.hip)."""
from __future__ import annotations

import ctypes
import os

import torch  # before libsynth.so: share PyTorch's HIP runtime

from . import gen

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth.so")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run "
                          "`python -m paper_2607_21224_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, i64, u64, u32, f = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                               ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float)
    lib.synth_fill_normal.argtypes = [vp, i, i64, i64, u64, i, i64, f, u32, f, vp]
    lib.synth_fill_normal.restype = i
    lib.synth_copy_f32.argtypes = [vp, vp, i64, vp]
    lib.synth_copy_f32.restype = i
    return lib


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = _load()
    return _lib


def _check_f32_device(x, name: str) -> None:
    """The kernels write through the raw address: only a contiguous fp32
    tensor on the GPU may reach them."""
    if x.dtype != torch.float32 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")


def _stream(s):
    if s is None:
        return None
    return s if isinstance(s, int) else int(s.cuda_stream)


def fill_normal(out, P: int, seed: int, kind: int, t: int, sigma: float,
                outlier_rate: float = 0.0, outlier_scale: float = 100.0,
                stream=None) -> None:
    """Fill out[:, :P] (a contiguous (rows, ld) fp32 CUDA tensor) with stream
    key(seed, kind, t, row) draws."""
    _check_f32_device(out, "out")
    if out.dim() not in (1, 2):
        raise ValueError("out must be a (ld,) or (rows, ld) tensor")
    rows, ld = (out.shape[0], out.shape[1]) if out.dim() == 2 else (1, out.shape[0])
    if not 0 <= P <= ld:
        raise ValueError(f"P = {P} does not fit rows of {ld}")
    r = lib().synth_fill_normal(out.data_ptr(), rows, P, ld, seed, kind, t, sigma,
                                gen.outlier_threshold(outlier_rate), outlier_scale,
                                _stream(stream))
    if r != 0:
        raise RuntimeError(f"synth_fill_normal failed ({r})")


def fill_theta0(out, P: int, seed: int, sigma: float = 0.02, stream=None) -> None:
    fill_normal(out, P, seed, gen.KIND_THETA0, 0, sigma, stream=stream)


def fill_grads(out, P: int, seed: int, step: int, sigma: float = 1e-3,
               outlier_rate: float = 0.0, outlier_scale: float = 100.0,
               stream=None) -> None:
    fill_normal(out, P, seed, gen.KIND_GRAD, step, sigma, outlier_rate,
                outlier_scale, stream)


def copy_f32(dst, src, n: int, stream=None) -> None:
    _check_f32_device(dst, "dst")
    _check_f32_device(src, "src")
    if not 0 <= n <= min(dst.numel(), src.numel()):
        raise ValueError(f"copy of {n} elements between tensors of {src.numel()} and "
                         f"{dst.numel()}")
    r = lib().synth_copy_f32(dst.data_ptr(), src.data_ptr(), n, _stream(stream))
    if r != 0:
        raise RuntimeError(f"synth_copy_f32 failed ({r})")
