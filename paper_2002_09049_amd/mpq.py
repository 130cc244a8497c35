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

EXPORTS = ("mpq_fit_layer", "mpq_fit_layer_dense", "mpq_fit_layers", "mpq_fit_max_dim",
           "mpq_output_error", "mpq_output_error_layers", "mpq_reconstruct",
           "mpq_reconstruct_layers", "mpq_last_error", "mpq_timing_enable", "mpq_timing_only", "mpq_timing_read",
           "mpq_fit_kernel_of", "mpq_quantize_layers", "mpq_fit_layer_calib",
           "mpq_fit_layers_calib", "mpq_integer_scales", "mpq_integer_forward",
           "mpq_integer_forward_layers", "mpq_fit_layers_ex", "mpq_output_error_noalloc")


class Layer(ctypes.Structure):
    """struct mpq_layer (include/mpq.h)."""
    _fields_ = [("W", ctypes.c_void_p), ("c_out", ctypes.c_int64), ("d", ctypes.c_int64),
                ("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("fit_err", ctypes.c_void_p),
                ("X", ctypes.c_void_p), ("n", ctypes.c_int64), ("out_err", ctypes.c_void_p),
                ("out_ref", ctypes.c_void_p), ("W_hat", ctypes.c_void_p),
                ("fit_xerr", ctypes.c_void_p), ("offsets", ctypes.c_void_p)]



class FitOptions(ctypes.Structure):
    """struct mpq_fit_options (include/mpq.h)."""
    _fields_ = [("refit", ctypes.c_int), ("calib", ctypes.c_int), ("eps", ctypes.c_float),
                ("relative", ctypes.c_int), ("clip_grid", ctypes.c_int),
                ("paper_eta", ctypes.c_float), ("asym", ctypes.c_int), ("gate", ctypes.c_int)]


class IntLayer(ctypes.Structure):
    """struct mpq_int_layer (include/mpq.h)."""
    _fields_ = [("codes", ctypes.c_void_p), ("A", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("c_out", ctypes.c_int64), ("d", ctypes.c_int64), ("X", ctypes.c_void_p),
                ("n", ctypes.c_int64), ("Y", ctypes.c_void_p)]


_lib = None


class KernelTime(ctypes.Structure):
    """struct mpq_kernel_time (include/mpq.h)."""
    _fields_ = [("name", ctypes.c_char * 64), ("ms", ctypes.c_float)]


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
    lib.mpq_fit_layer_calib.argtypes = [P, i64, i64, i32, i32, P, i32, P, i64, f32, i32, P, P, P, P,
                                         P, P]
    lib.mpq_fit_layer_calib.restype = i32
    lib.mpq_fit_layers_calib.argtypes = [P, i32, i32, i32, P, i32, f32, i32, P]
    lib.mpq_fit_layers_calib.restype = i32
    lib.mpq_integer_scales.argtypes = [P, P, i64, i32, i32, P, P, P]
    lib.mpq_integer_scales.restype = i32
    lib.mpq_integer_forward.argtypes = [P, P, P, i64, i64, i32, P, i64, i32, P, P]
    lib.mpq_integer_forward.restype = i32
    lib.mpq_integer_forward_layers.argtypes = [P, i32, i32, i32, P]
    lib.mpq_integer_forward_layers.restype = i32
    lib.mpq_fit_layers_ex.argtypes = [P, i32, i32, i32, P, i32, f32, P, P]
    lib.mpq_fit_layers_ex.restype = i32
    lib.mpq_fit_max_dim.argtypes = [i32]
    lib.mpq_fit_max_dim.restype = i64
    lib.mpq_output_error.argtypes = [P, P, P, P, i64, i64, i32, P, i64, P, P, P]
    lib.mpq_output_error.restype = i32
    lib.mpq_output_error_noalloc.argtypes = [P, P, P, P, i64, i64, i32, P, i64, P, P, P]
    lib.mpq_output_error_noalloc.restype = i32
    lib.mpq_reconstruct.argtypes = [P, P, P, i64, i64, i32, P, P]
    lib.mpq_reconstruct.restype = i32
    lib.mpq_fit_layers.argtypes = [P, i32, i32, i32, P, i32, f32, P]
    lib.mpq_fit_layers.restype = i32
    lib.mpq_quantize_layers.argtypes = [P, i32, i32, i32, P, i32, f32, P]
    lib.mpq_quantize_layers.restype = i32
    lib.mpq_output_error_layers.argtypes = [P, i32, i32, P]
    lib.mpq_output_error_layers.restype = i32
    lib.mpq_reconstruct_layers.argtypes = [P, i32, i32, P]
    lib.mpq_reconstruct_layers.restype = i32
    lib.mpq_last_error.argtypes = []
    lib.mpq_last_error.restype = ctypes.c_char_p
    lib.mpq_timing_enable.argtypes = [i32]
    lib.mpq_timing_enable.restype = i32
    lib.mpq_timing_only.argtypes = [ctypes.c_char_p]
    lib.mpq_timing_only.restype = i32
    lib.mpq_timing_read.argtypes = [P, i32]
    lib.mpq_timing_read.restype = i32
    lib.mpq_fit_kernel_of.argtypes = [i64, i32, i32, i32, ctypes.c_char_p, i32]
    lib.mpq_fit_kernel_of.restype = i32
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


def fit_layer_calib(W: torch.Tensor, bits: int, max_points: int, n_grid: int, X: torch.Tensor,
                    eps: float, relative: bool = True, grid=None, with_err: bool = True,
                    stream=None, out=None):
    """mpq_fit_layer_calib: the fit with Algorithm 2's stopping rule on the
    calibration batch X [d, n] fp32.  Returns (codes, scales, counts, err or
    None, xerr [C, P]).  ``out`` may hold preallocated (codes, scales,
    counts, err, xerr)."""
    if W.dim() != 2:
        raise ValueError("W must be 2-D [C_out, d]")
    C, d = W.shape
    if X.dim() != 2 or X.shape[0] != d:
        raise ValueError("X must be [d, n]")
    dev = W.device
    if out is None:
        codes = torch.empty((C, max_points, d), dtype=torch.int8, device=dev)
        scales = torch.empty((C, max_points), dtype=torch.float32, device=dev)
        counts = torch.empty((C,), dtype=torch.int32, device=dev)
        err = torch.empty((C, max_points), dtype=torch.float32, device=dev) if with_err else None
        xerr = torch.empty((C, max_points), dtype=torch.float32, device=dev)
    else:
        codes, scales, counts, err, xerr = out
    g = LayerSet._grid(grid, n_grid)
    rc = load().mpq_fit_layer_calib(
        _dev(W, torch.float32, "W"), C, d, bits, max_points,
        None if g is None else g.ctypes.data_as(ctypes.c_void_p), n_grid,
        _dev(X, torch.float32, "X"), X.shape[1], float(eps), 1 if relative else 0,
        _dev(codes, torch.int8, "codes"), _dev(scales, torch.float32, "scales"),
        _dev(counts, torch.int32, "counts"), None if err is None else _dev(err, torch.float32, "err"),
        _dev(xerr, torch.float32, "xerr"), _stream(stream))
    _check(rc)
    return codes, scales, counts, err, xerr


def fit_max_dim(n_grid: int) -> int:
    v = load().mpq_fit_max_dim(n_grid)
    if v < 0:
        raise MPQError(int(v), last_error())
    return int(v)


def output_error(W: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor, counts: torch.Tensor,
                 X: torch.Tensor, with_ref: bool = False, stream=None,
                 out: Optional[Tuple[torch.Tensor, Optional[torch.Tensor]]] = None,
                 noalloc: bool = False):
    """mpq_output_error (noalloc: mpq_output_error_noalloc, whose workspace is
    the library's fixed per-device array; pass `out` to allocate nothing on
    the Python side either).  X: [d, n] fp32.  Returns (err [C], ref [C] or
    None)."""
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
    lib = load()
    fn = lib.mpq_output_error_noalloc if noalloc else lib.mpq_output_error
    rc = fn(_dev(W, torch.float32, "W"), _dev(codes, torch.int8, "codes"),
            _dev(scales, torch.float32, "scales"), _dev(counts, torch.int32, "counts"), C, d, P,
            _dev(X, torch.float32, "X"), n, _dev(err, torch.float32, "err"),
            None if ref is None else _dev(ref, torch.float32, "ref"), _stream(stream))
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


def integer_scales(scales: torch.Tensor, counts: torch.Tensor, p: int, stream=None,
                   out: Optional[torch.Tensor] = None, count_clamped: bool = True):
    """mpq_integer_scales (Eq. (14)).  Returns (A [C, P] int32, number of
    clamped values as a 1-element uint64 device tensor (int64 view) or None)."""
    C, P = scales.shape
    A = torch.empty((C, P), dtype=torch.int32, device=scales.device) if out is None else out
    cl = torch.zeros((1,), dtype=torch.int64, device=scales.device) if count_clamped else None
    _check(load().mpq_integer_scales(_dev(scales, torch.float32, "scales"),
                                     _dev(counts, torch.int32, "counts"), C, P, int(p),
                                     _dev(A, torch.int32, "A"),
                                     None if cl is None else cl.data_ptr(), _stream(stream)))
    return A, cl


def integer_forward(codes: torch.Tensor, A: torch.Tensor, counts: torch.Tensor, X: torch.Tensor,
                    p: int, stream=None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """mpq_integer_forward (Eq. (15), Steps 1-3).  X [n, d] int8.  Returns Y [C, n] int64."""
    C, P, d = codes.shape
    if X.dim() != 2 or X.shape[1] != d:
        raise ValueError("X must be [n, d]")
    n = X.shape[0]
    Y = torch.empty((C, n), dtype=torch.int64, device=codes.device) if out is None else out
    _check(load().mpq_integer_forward(_dev(codes, torch.int8, "codes"), _dev(A, torch.int32, "A"),
                                      _dev(counts, torch.int32, "counts"), C, d, P,
                                      _dev(X, torch.int8, "X"), n, int(p), _dev(Y, torch.int64, "Y"),
                                      _stream(stream)))
    return Y


def integer_forward_layers(layers, max_points: int, p: int, stream=None):
    """mpq_integer_forward_layers.  layers: list of (codes, A, counts, X, Y) device tensors."""
    arr = (IntLayer * max(len(layers), 1))()
    for i, (codes, A, counts, X, Y) in enumerate(layers):
        C, P, d = codes.shape
        if P != max_points or X.shape[1] != d or Y.shape != (C, X.shape[0]):
            raise ValueError(f"layer {i}: shapes do not match")
        L = arr[i]
        L.codes, L.A = _dev(codes, torch.int8, "codes"), _dev(A, torch.int32, "A")
        L.counts, L.X = _dev(counts, torch.int32, "counts"), _dev(X, torch.int8, "X")
        L.Y = _dev(Y, torch.int64, "Y")
        L.c_out, L.d, L.n = C, d, X.shape[0]
    _check(load().mpq_integer_forward_layers(ctypes.addressof(arr), len(layers), max_points, int(p),
                                             _stream(stream)))


def timing_enable(on: bool = True):
    """mpq_timing_enable: drop earlier records; record (or stop recording)
    HIP events around every kernel launch, on the launch's own stream."""
    _check(load().mpq_timing_enable(1 if on else 0))


def timing_only(name=None):
    """mpq_timing_only: time only the launches of the kernel ``name`` (None:
    every launch)."""
    _check(load().mpq_timing_only(None if name is None else name.encode()))


def timing_read():
    """mpq_timing_read: [(kernel name, ms)] in launch order (waits for the
    recorded events)."""
    lib = load()
    n = lib.mpq_timing_read(None, 0)
    if n < 0:
        _check(n)
    buf = (KernelTime * max(n, 1))()
    n = lib.mpq_timing_read(ctypes.addressof(buf), n)
    return [(buf[i].name.decode(), float(buf[i].ms)) for i in range(n)]


def fit_kernel_of(d: int, bits: int, n_grid: int, default_grid: bool = True) -> str:
    """mpq_fit_kernel_of: the kernel name that fits channels of length d."""
    buf = ctypes.create_string_buffer(64)
    _check(load().mpq_fit_kernel_of(d, bits, n_grid, 1 if default_grid else 0, buf, 64))
    return buf.value.decode()


class LayerSet:
    """The layers of a network for the batched calls (mpq_fit_layers,
    mpq_output_error_layers, mpq_reconstruct_layers).

    Allocates the outputs of every layer once on the weights' device and
    keeps the descriptor array, so each batched call is one C call.
    ``weights``: list of [C, d] fp32 device tensors; ``calib``: optional list
    of [d, n] fp32 device tensors (one per layer)."""

    def __init__(self, weights, max_points: int, calib=None, with_fit_err: bool = True,
                 with_ref: bool = False):
        self.max_points = max_points
        self.W = list(weights)
        self.X = list(calib) if calib is not None else None
        n = len(self.W)
        self.arr = (Layer * max(n, 1))()
        self.codes, self.scales, self.counts, self.fit_err = [], [], [], []
        self.err, self.ref, self.W_hat, self.xerr, self.offsets = [], [], [], [], []
        for i, W in enumerate(self.W):
            C, d = W.shape
            dev = W.device
            codes = torch.empty((C, max_points, d), dtype=torch.int8, device=dev)
            scales = torch.empty((C, max_points), dtype=torch.float32, device=dev)
            counts = torch.empty((C,), dtype=torch.int32, device=dev)
            ferr = torch.empty((C, max_points), dtype=torch.float32, device=dev) if with_fit_err else None
            err = torch.empty((C,), dtype=torch.float32, device=dev)
            ref = torch.empty((C,), dtype=torch.float32, device=dev) if with_ref else None
            what = torch.empty((C, d), dtype=torch.float32, device=dev)
            xerr = torch.empty((C, max_points), dtype=torch.float32, device=dev) if calib is not None else None
            self.xerr.append(xerr)
            self.offsets.append(torch.zeros((C,), dtype=torch.float32, device=dev))
            self.codes.append(codes)
            self.scales.append(scales)
            self.counts.append(counts)
            self.fit_err.append(ferr)
            self.err.append(err)
            self.ref.append(ref)
            self.W_hat.append(what)
            L = self.arr[i]
            L.W = _dev(W, torch.float32, "W")
            L.c_out, L.d = C, d
            L.codes, L.scales, L.counts = codes.data_ptr(), scales.data_ptr(), counts.data_ptr()
            L.fit_err = None if ferr is None else ferr.data_ptr()
            if self.X is not None:
                X = self.X[i]
                if X.dim() != 2 or X.shape[0] != d:
                    raise ValueError(f"calib[{i}] must be [d, n]")
                L.X = _dev(X, torch.float32, "X")
                L.n = X.shape[1]
            L.out_err = err.data_ptr() if self.X is not None else None
            L.out_ref = None if ref is None else ref.data_ptr()
            L.W_hat = what.data_ptr()
            L.fit_xerr = None if xerr is None else xerr.data_ptr()
        self.n = n

    @staticmethod
    def _grid(grid, n_grid):
        if grid is None:
            return None
        import numpy as np
        g = np.ascontiguousarray(grid, dtype=np.float32)
        if g.shape != (n_grid,):
            raise ValueError("grid must have n_grid entries")
        return g

    def fit_ex(self, bits: int, n_grid: int, tol: float = 0.0, refit: bool = False,
               calib: bool = False, eps: float = 0.0, relative: bool = True, clip_grid: int = 0,
               paper_eta: float = 0.0, asym: bool = False, gate: bool = False, grid=None,
               stream=None):
        """mpq_fit_layers_ex: the fit with options (refit: reading A2; calib:
        Algorithm 2's stopping rule on the calibration batches; clip_grid:
        point 1 from the clipping of Eq. (13) with that many factors;
        paper_eta: the paper's own grid of Eq. (11) with that maximal step;
        gate: Algorithm 2's naive first point, reading F1)."""
        if (calib or clip_grid) and self.X is None:
            raise ValueError("LayerSet was built without calibration batches")
        g = self._grid(grid, n_grid)
        opt = FitOptions(1 if refit else 0, 1 if calib else 0, float(eps), 1 if relative else 0,
                         int(clip_grid), float(paper_eta), 1 if asym else 0, 1 if gate else 0)
        # the offsets take part in the fit and, afterwards, in the layer's
        # output error and reconstruction only when the fit is asymmetric
        for i in range(self.n):
            self.arr[i].offsets = self.offsets[i].data_ptr() if asym and self.offsets[i] is not None else None
        _check(load().mpq_fit_layers_ex(ctypes.addressof(self.arr), self.n, bits, self.max_points,
                                        None if g is None else g.ctypes.data_as(ctypes.c_void_p),
                                        n_grid, float(tol), ctypes.addressof(opt), _stream(stream)))

    def _symmetric(self):
        """A symmetric fit follows: the layers' output error and
        reconstruction take no offsets."""
        for i in range(self.n):
            self.arr[i].offsets = None

    def fit(self, bits: int, n_grid: int, tol: float, grid=None, stream=None):
        self._symmetric()
        g = self._grid(grid, n_grid)
        _check(load().mpq_fit_layers(ctypes.addressof(self.arr), self.n, bits, self.max_points,
                                     None if g is None else g.ctypes.data_as(ctypes.c_void_p),
                                     n_grid, float(tol), _stream(stream)))

    def quantize(self, bits: int, n_grid: int, tol: float, grid=None, stream=None):
        """mpq_quantize_layers: fit, output error (when calibration batches
        were given) and reconstruction of every layer in one call."""
        self._symmetric()
        g = self._grid(grid, n_grid)
        _check(load().mpq_quantize_layers(ctypes.addressof(self.arr), self.n, bits, self.max_points,
                                          None if g is None else g.ctypes.data_as(ctypes.c_void_p),
                                          n_grid, float(tol), _stream(stream)))

    def fit_calib(self, bits: int, n_grid: int, eps: float, relative: bool = True, grid=None,
                  stream=None):
        """mpq_fit_layers_calib: the fit of every layer with Algorithm 2's
        stopping rule on its calibration batch; xerr [C, P] per layer."""
        if self.X is None:
            raise ValueError("LayerSet was built without calibration batches")
        self._symmetric()
        g = self._grid(grid, n_grid)
        _check(load().mpq_fit_layers_calib(ctypes.addressof(self.arr), self.n, bits, self.max_points,
                                           None if g is None else g.ctypes.data_as(ctypes.c_void_p),
                                           n_grid, float(eps), 1 if relative else 0, _stream(stream)))

    def output_error(self, stream=None):
        if self.X is None:
            raise ValueError("LayerSet was built without calibration batches")
        _check(load().mpq_output_error_layers(ctypes.addressof(self.arr), self.n, self.max_points,
                                              _stream(stream)))

    def reconstruct(self, stream=None):
        _check(load().mpq_reconstruct_layers(ctypes.addressof(self.arr), self.n, self.max_points,
                                             _stream(stream)))
