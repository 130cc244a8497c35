"""Python binding of libmpq.so (the HIP C ABI declared in include/mpq.h).

Argument marshalling only: torch tensors on a ROCm device provide the device
memory and the current stream; every step of the fit, the output error and
the reconstruction runs in the library's HIP kernels.  There is no CPU
fallback: if the library is missing, every call raises.

The library is loaded after torch, so it binds to the HIP runtime that torch
already loaded (both carry the soname libamdhip64.so.7) and the stream
handles and device pointers torch hands out are valid in it.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmpq.so")

MPQ_OK = 0
MPQ_ERR_INVALID_ARG = -1
MPQ_ERR_SHAPE = -2
MPQ_ERR_HIP = -3
MPQ_ERR_NOMEM = -4
MAX_POINTS = 64
MAX_GRID = 4096

EXPORTS = ("mpq_fit_layer", "mpq_fit_layer_dense", "mpq_fit_max_dim", "mpq_output_error",
           "mpq_reconstruct", "mpq_last_error")

_lib = None


class MPQError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"mpq status {status}: {message}")
        self.status = status


def load(path: str = LIB_PATH):
    """Load libmpq.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing; build it with `python -m paper_2002_09049_amd.build`")
    lib = ctypes.CDLL(path)
    P, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    for name in ("mpq_fit_layer", "mpq_fit_layer_dense"):
        getattr(lib, name).argtypes = [P, i64, i64, i32, i32, P, i32, f32, P, P, P, P, P]
        getattr(lib, name).restype = i32
    lib.mpq_fit_max_dim.argtypes = [i32]
    lib.mpq_fit_max_dim.restype = i64
    lib.mpq_output_error.argtypes = [P, P, P, P, i64, i64, i32, P, i64, P, P, P]
    lib.mpq_output_error.restype = i32
    lib.mpq_reconstruct.argtypes = [P, P, P, i64, i64, i32, P, P]
    lib.mpq_reconstruct.restype = i32
    lib.mpq_last_error.argtypes = []
    lib.mpq_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return load().mpq_last_error().decode()


def _check(rc: int):
    if rc != MPQ_OK:
        raise MPQError(rc, last_error())


def _dev(x: torch.Tensor, dtype, name: str) -> int:
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise ValueError(f"{name} must be a ROCm device tensor")
    if x.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {x.dtype})")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return x.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def fit_layer(W: torch.Tensor, bits: int, max_points: int, n_grid: int, tol: float,
              grid=None, with_err: bool = True, stream=None, out=None, dense: bool = False):
    """mpq_fit_layer (mpq_fit_layer_dense with dense=True).  W: [C, d] fp32 on the device.

    Returns (codes [C, P, d] int8, scales [C, P] fp32, counts [C] int32,
    err [C, P] fp32 or None).  ``grid`` is an optional host sequence of
    n_grid multipliers in (0, 1].  ``out`` may hold preallocated
    (codes, scales, counts, err) tensors."""
    if W.dim() != 2:
        raise ValueError("W must be 2-D [C_out, d]")
    C, d = W.shape
    dev = W.device
    if out is None:
        codes = torch.empty((C, max_points, d), dtype=torch.int8, device=dev)
        scales = torch.empty((C, max_points), dtype=torch.float32, device=dev)
        counts = torch.empty((C,), dtype=torch.int32, device=dev)
        err = torch.empty((C, max_points), dtype=torch.float32, device=dev) if with_err else None
    else:
        codes, scales, counts, err = out
    gbuf = None
    if grid is not None:
        import numpy as np
        g = np.ascontiguousarray(grid, dtype=np.float32)
        if g.shape != (n_grid,):
            raise ValueError("grid must have n_grid entries")
        gbuf = g
    lib = load()
    fn = lib.mpq_fit_layer_dense if dense else lib.mpq_fit_layer
    rc = fn(_dev(W, torch.float32, "W"), C, d, bits, max_points,
                           None if gbuf is None else gbuf.ctypes.data_as(ctypes.c_void_p),
                           n_grid, float(tol), _dev(codes, torch.int8, "codes"),
                           _dev(scales, torch.float32, "scales"),
                           _dev(counts, torch.int32, "counts"),
                           None if err is None else _dev(err, torch.float32, "err"),
                           _stream(stream))
    _check(rc)
    return codes, scales, counts, err


def fit_max_dim(n_grid: int) -> int:
    v = load().mpq_fit_max_dim(n_grid)
    if v < 0:
        raise MPQError(int(v), last_error())
    return int(v)


def output_error(W: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor, counts: torch.Tensor,
                 X: torch.Tensor, with_ref: bool = False, stream=None,
                 out: Optional[Tuple[torch.Tensor, Optional[torch.Tensor]]] = None):
    """mpq_output_error.  X: [d, n] fp32.  Returns (err [C], ref [C] or None)."""
    C, d = W.shape
    P = codes.shape[1]
    if codes.shape != (C, P, d) or scales.shape != (C, P) or counts.shape != (C,):
        raise ValueError("codes/scales/counts do not match W")
    if X.dim() != 2 or X.shape[0] != d:
        raise ValueError("X must be [d, n]")
    n = X.shape[1]
    if out is None:
        err = torch.empty((C,), dtype=torch.float32, device=W.device)
        ref = torch.empty((C,), dtype=torch.float32, device=W.device) if with_ref else None
    else:
        err, ref = out
    rc = load().mpq_output_error(_dev(W, torch.float32, "W"), _dev(codes, torch.int8, "codes"),
                                 _dev(scales, torch.float32, "scales"),
                                 _dev(counts, torch.int32, "counts"), C, d, P,
                                 _dev(X, torch.float32, "X"), n, _dev(err, torch.float32, "err"),
                                 None if ref is None else _dev(ref, torch.float32, "ref"),
                                 _stream(stream))
    _check(rc)
    return err, ref


def reconstruct(codes: torch.Tensor, scales: torch.Tensor, counts: torch.Tensor, stream=None,
                out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """mpq_reconstruct.  Returns W_hat [C, d] fp32."""
    C, P, d = codes.shape
    W_hat = torch.empty((C, d), dtype=torch.float32, device=codes.device) if out is None else out
    rc = load().mpq_reconstruct(_dev(codes, torch.int8, "codes"), _dev(scales, torch.float32, "scales"),
                                _dev(counts, torch.int32, "counts"), C, d, P,
                                _dev(W_hat, torch.float32, "W_hat"), _stream(stream))
    _check(rc)
    return W_hat
