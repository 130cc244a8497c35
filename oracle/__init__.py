"""Oracle for the multipoint fit: a plain fp64 CPU implementation in C.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP library (``paper_2002_09049_amd``); the only module both
sides use is the seeded input generator ``paper_2002_09049_amd.workloads``,
which holds none of the method's arithmetic.

The arithmetic lives in ``mpq_oracle.c`` (see its header for the paper
passages and readings it follows); this module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "mpq_oracle.c")
LIB = os.path.join(_HERE, "libmpq_oracle.so")
_default = None


def build(force: bool = True, src: str = SRC, out: str = LIB) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math, no FP contraction)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-fno-fast-math", "-ffp-contract=off", src, "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


def _declare(lib):
    P = ctypes.c_void_p
    i64, i32, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_double
    lib.oracle_fit.argtypes = [P, i64, i64, i32, i32, P, i32, f64, P, P, P, P, i32]
    lib.oracle_fit.restype = i32
    lib.oracle_verify.argtypes = [P, i64, i64, i32, i32, P, i32, f64, P, P, P, P,
                                  P, i64, P, P, P, P, P, i32]
    lib.oracle_verify.restype = i32
    lib.oracle_fit_calib.argtypes = [P, i64, i64, i32, i32, P, i32, P, i64, f64, i32, P, P, P, P,
                                     P, i32]
    lib.oracle_fit_calib.restype = i32
    lib.oracle_verify_calib.argtypes = [P, i64, i64, i32, i32, P, i32, P, i64, f64, i32, P, P, P,
                                        P, P, P, i64, P, P, P, P, P, i32]
    lib.oracle_verify_calib.restype = i32
    lib.oracle_output_error.argtypes = [P, P, P, P, i64, i64, i32, P, i64, P, i64,
                                        P, P, i32]
    lib.oracle_output_error.restype = i32
    lib.oracle_reconstruct.argtypes = [P, P, P, i64, i64, i32, P]
    lib.oracle_reconstruct.restype = None
    lib.oracle_candidate_scales.argtypes = [P, i64, i32, P, i32, P]
    lib.oracle_candidate_scales.restype = None
    lib.oracle_codes.argtypes = [P, i64, f64, i32, P]
    lib.oracle_codes.restype = None
    lib.oracle_scale_error.argtypes = [P, i64, f64, i32]
    lib.oracle_scale_error.restype = f64
    lib.oracle_levels.argtypes = [i32]
    lib.oracle_levels.restype = i32
    lib.oracle_default_grid.argtypes = [i32, P]
    lib.oracle_default_grid.restype = None
    lib.oracle_fit_ex.argtypes = [P, i64, i64, i32, i32, P, i32, f64, P, i64, i32, f64, i32, i32,
                                  i32, f64, i32, P, P, P, P, P, P, i32]
    lib.oracle_fit_ex.restype = i32
    lib.oracle_verify_ex.argtypes = [P, i64, i64, i32, i32, P, i32, f64, P, i64, i32, f64, i32, i32,
                                     i32, f64, i32, P, P, P, P, P, P, P, i64, P, P, P, P, P, i32]
    lib.oracle_output_error_ex.argtypes = [P, P, P, P, P, i64, i64, i32, P, i64, P, i64, P, P, i32]
    lib.oracle_output_error_ex.restype = i32
    lib.oracle_reconstruct_ex.argtypes = [P, P, P, P, i64, i64, i32, P]
    lib.oracle_reconstruct_ex.restype = None
    lib.oracle_min_gap.argtypes = [P, i64, P]
    lib.oracle_min_gap.restype = f64
    lib.oracle_paper_grid.argtypes = [P, i64, i32, f64, P, P, P]
    lib.oracle_paper_grid.restype = None
    lib.oracle_paper_grid_search.argtypes = [P, i64, i32, f64, i64, P]
    lib.oracle_paper_grid_search.restype = i64
    lib.oracle_verify_ex.restype = i32
    lib.oracle_integer_scales.argtypes = [P, P, i64, i32, i32, P]
    lib.oracle_integer_scales.restype = i64
    lib.oracle_integer_forward.argtypes = [P, P, P, i64, i64, i32, P, i64, i32, P]
    lib.oracle_integer_forward.restype = i32
    return lib


def load(path: Optional[str] = None) -> "Oracle":
    """Oracle bound to a compiled library (default: the built one)."""
    global _default
    if path is not None:
        return Oracle(_declare(ctypes.CDLL(path)))
    if _default is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build(force=True)
        _default = Oracle(_declare(ctypes.CDLL(LIB)))
    return _default


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _grid(grid, G):
    if grid is None:
        return None
    g = np.ascontiguousarray(grid, dtype=np.float32)
    assert g.shape == (G,)
    return g


class Oracle:
    """numpy front end of one compiled oracle library."""

    def __init__(self, lib):
        self.lib = lib

    def levels(self, bits: int) -> int:
        return self.lib.oracle_levels(bits)

    def default_grid(self, G: int) -> np.ndarray:
        c = np.empty(G, np.float32)
        self.lib.oracle_default_grid(G, _p(c))
        return c

    def candidate_scales(self, r: np.ndarray, bits: int, grid: np.ndarray) -> np.ndarray:
        r = np.ascontiguousarray(r, dtype=np.float64)
        g = np.ascontiguousarray(grid, dtype=np.float32)
        a = np.empty(g.shape[0], np.float32)
        self.lib.oracle_candidate_scales(_p(r), r.size, self.levels(bits), _p(g), g.size, _p(a))
        return a

    def codes(self, r: np.ndarray, a: float, bits: int) -> np.ndarray:
        r = np.ascontiguousarray(r, dtype=np.float64)
        q = np.empty(r.size, np.int8)
        self.lib.oracle_codes(_p(r), r.size, float(a), self.levels(bits), _p(q))
        return q

    def scale_error(self, r: np.ndarray, a: float, bits: int) -> float:
        r = np.ascontiguousarray(r, dtype=np.float64)
        return self.lib.oracle_scale_error(_p(r), r.size, float(a), self.levels(bits))

    def fit(self, W: np.ndarray, bits: int, max_points: int, n_grid: int, tol: float,
            grid: Optional[np.ndarray] = None, n_threads: int = 0, refit: bool = False,
            gate: bool = False):
        """Free-running greedy fit (refit: reading A2; gate: Algorithm 2's naive
        first point, reading F1). Returns (codes[C,P,d] i8, scales[C,P] f32,
        counts[C] i32, err[C,P] f64)."""
        return self._fit(W, bits, max_points, n_grid, tol, None, 0.0, False, refit, grid,
                         n_threads, gate=gate)[:4]

    def fit_clip(self, W, bits: int, max_points: int, n_grid: int, X, tol: float = 0.0,
                 calib: bool = False, eps: float = 0.0, relative: bool = True, clip_grid: int = 20,
                 grid=None, n_threads: int = 0):
        """Fit whose first point is the clipping of Eq. (13) on X (reading C1),
        then Algorithm 1 with the stopping rule S1 (tol) or, with calib, S4.
        Returns (codes, scales, counts, err, xerr)."""
        return self._fit(W, bits, max_points, n_grid, tol, X, eps, relative, False, grid,
                         n_threads, calib=calib, clip_grid=clip_grid)

    def fit_paper(self, W, bits: int, max_points: int, tol: float, eta: float = 2.0 ** -10,
                  n_threads: int = 0):
        """Greedy fit on the paper's own grid, Eq. (11) (readings D1, G3).
        Returns (codes, scales, counts, err)."""
        return self._fit(W, bits, max_points, 1, tol, None, 0.0, False, False, None, n_threads,
                         eta=eta)[:4]

    def min_gap(self, r) -> float:
        r = np.ascontiguousarray(r, dtype=np.float64)
        return self.lib.oracle_min_gap(_p(r), r.size, _p(np.empty(r.size)))

    def paper_grid(self, r, bits: int, eta: float = 2.0 ** -10):
        """(gamma, number of grid points) of Eq. (11) for the residual r."""
        r = np.ascontiguousarray(r, dtype=np.float64)
        g = ctypes.c_double()
        n = ctypes.c_int64()
        self.lib.oracle_paper_grid(_p(r), r.size, self.levels(bits), float(eta), _p(np.empty(r.size)),
                                   ctypes.byref(g), ctypes.byref(n))
        return g.value, n.value

    def paper_grid_search(self, r, bits: int, gamma: float, count: int):
        """(g, E) of the grid argmin of Eq. (9) over g gamma, 1 <= g <= count."""
        r = np.ascontiguousarray(r, dtype=np.float64)
        E = ctypes.c_double()
        g = self.lib.oracle_paper_grid_search(_p(r), r.size, self.levels(bits), float(gamma),
                                              int(count), ctypes.byref(E))
        return int(g), E.value

    def fit_asym(self, W, bits: int, max_points: int, n_grid: int, tol: float = 0.0, X=None,
                 calib: bool = False, eps: float = 0.0, relative: bool = True, refit: bool = False,
                 grid=None, n_threads: int = 0, gate: bool = False):
        """Fit with the per-channel offset of reading B2 (the asymmetric set of
        Eq. (1)).  Returns (codes, scales, counts, err, xerr, offsets[C] f32)."""
        return self._fit(W, bits, max_points, n_grid, tol, X, eps, relative, refit, grid, n_threads,
                         calib=calib, asym=True, gate=gate)

    def _fit(self, W, bits, P, n_grid, tol, X, eps, relative, refit, grid, n_threads, calib=None,
             clip_grid=0, eta=0.0, asym=False, gate=False):
        calib = (X is not None) if calib is None else calib
        W = np.ascontiguousarray(W, dtype=np.float32)
        C, d = W.shape
        if X is not None:
            X = np.ascontiguousarray(X, dtype=np.float32)
            assert X.shape[0] == d
        codes_ = np.zeros((C, P, d), np.int8)
        scales = np.zeros((C, P), np.float32)
        counts = np.zeros(C, np.int32)
        err = np.zeros((C, P), np.float64)
        xerr = np.zeros((C, P), np.float64)
        offsets = np.zeros(C, np.float32) if asym else None
        g = _grid(grid, n_grid)
        rc = self.lib.oracle_fit_ex(_p(W), C, d, bits, P, _p(g), n_grid, float(tol), _p(X),
                                    0 if X is None else X.shape[1], 1 if calib else 0, float(eps),
                                    1 if relative else 0, 1 if refit else 0, int(clip_grid),
                                    float(eta), 1 if gate else 0, _p(offsets), _p(codes_),
                                    _p(scales), _p(counts), _p(err), _p(xerr), n_threads)
        if rc != 0:
            raise MemoryError("oracle_fit_ex failed")
        return (codes_, scales, counts, err, xerr) + ((offsets,) if asym else ())

    def verify(self, W, bits, max_points, n_grid, tol, codes_, scales, counts, err=None,
               grid=None, channels=None, n_threads: int = 0, refit: bool = False,
               gate: bool = False):
        """Lockstep check of another implementation's fit output (rules V1-V4;
        refit: reading A2; gate: reading F1, status 10 for a wrong naive-point
        decision).

        Returns a dict of per-channel arrays: status, cand_ties, code_ties,
        stop_ties, err_relmax, and the checked channel indices.
        """
        return self._verify(W, bits, max_points, n_grid, tol, None, 0.0, False, refit, codes_,
                            scales, counts, err, None, grid, channels, n_threads, gate=gate)

    def verify_clip(self, W, bits, max_points, n_grid, X, codes_, scales, counts, err=None,
                    xerr=None, tol: float = 0.0, calib: bool = False, eps: float = 0.0,
                    relative: bool = True, clip_grid: int = 20, grid=None, channels=None,
                    n_threads: int = 0):
        """Lockstep check of a fit whose first point is the clipping of reading C1."""
        return self._verify(W, bits, max_points, n_grid, tol, X, eps, relative, False, codes_,
                            scales, counts, err, xerr, grid, channels, n_threads, calib=calib,
                            clip_grid=clip_grid)

    def verify_paper(self, W, bits, max_points, tol, codes_, scales, counts, err=None,
                     eta: float = 2.0 ** -10, channels=None, n_threads: int = 0):
        """Lockstep check of a fit on the paper's grid (readings D1, G3)."""
        return self._verify(W, bits, max_points, 1, tol, None, 0.0, False, False, codes_, scales,
                            counts, err, None, None, channels, n_threads, eta=eta)

    def verify_asym(self, W, bits, max_points, n_grid, codes_, scales, counts, offsets, err=None,
                    xerr=None, tol: float = 0.0, X=None, calib: bool = False, eps: float = 0.0,
                    relative: bool = True, refit: bool = False, grid=None, channels=None,
                    n_threads: int = 0, gate: bool = False):
        """Lockstep check of a fit with the per-channel offset of reading B2
        (status 9: an offset that is not the fp32 midpoint)."""
        return self._verify(W, bits, max_points, n_grid, tol, X, eps, relative, refit, codes_,
                            scales, counts, err, xerr, grid, channels, n_threads, calib=calib,
                            offsets=offsets, gate=gate)

    def _verify(self, W, bits, P, n_grid, tol, X, eps, relative, refit, codes_, scales, counts,
                err, xerr, grid, channels, n_threads, calib=None, clip_grid=0, eta=0.0, offsets=None,
                gate=False):
        calib = (X is not None) if calib is None else calib
        if offsets is not None:
            offsets = np.ascontiguousarray(offsets, dtype=np.float32)
        W = np.ascontiguousarray(W, dtype=np.float32)
        C, d = W.shape
        if X is not None:
            X = np.ascontiguousarray(X, dtype=np.float32)
        codes_ = np.ascontiguousarray(codes_, dtype=np.int8)
        scales = np.ascontiguousarray(scales, dtype=np.float32)
        counts = np.ascontiguousarray(counts, dtype=np.int32)
        assert codes_.shape == (C, P, d) and scales.shape == (C, P)
        assert counts.shape == (C,)
        e = None if err is None else np.ascontiguousarray(err, dtype=np.float32)
        xe = None if xerr is None else np.ascontiguousarray(xerr, dtype=np.float32)
        chan = np.arange(C, dtype=np.int64) if channels is None else \
            np.ascontiguousarray(channels, dtype=np.int64)
        n = chan.size
        out = {k: np.zeros(n, np.int32) for k in ("status", "cand_ties", "code_ties", "stop_ties")}
        out["err_relmax"] = np.zeros(n, np.float64)
        g = _grid(grid, n_grid)
        rc = self.lib.oracle_verify_ex(
            _p(W), C, d, bits, P, _p(g), n_grid, float(tol), _p(X), 0 if X is None else X.shape[1],
            1 if calib else 0, float(eps), 1 if relative else 0, 1 if refit else 0, int(clip_grid),
            float(eta), 1 if gate else 0, _p(offsets), _p(codes_), _p(scales),
            _p(counts), _p(e), _p(xe), _p(chan), n, _p(out["status"]), _p(out["cand_ties"]),
            _p(out["code_ties"]), _p(out["stop_ties"]), _p(out["err_relmax"]), n_threads)
        if rc != 0:
            raise MemoryError("oracle_verify_ex failed")
        out["channels"] = chan
        return out

    def fit_calib(self, W: np.ndarray, bits: int, max_points: int, n_grid: int, X: np.ndarray,
                  eps: float, relative: bool, grid: Optional[np.ndarray] = None, n_threads: int = 0,
                  refit: bool = False, gate: bool = False):
        """Free-running fit with Algorithm 2's stopping rule on the calibration
        batch X [d, N] (reading S4; refit: reading A2; gate: Algorithm 2's
        naive first point, reading F1).  Returns (codes, scales, counts, err,
        xerr[C,P] f64: the output error after each point)."""
        return self._fit(W, bits, max_points, n_grid, 0.0, X, eps, relative, refit, grid, n_threads,
                         gate=gate)

    def verify_calib(self, W, bits, max_points, n_grid, X, eps, relative, codes_, scales, counts,
                     err=None, xerr=None, grid=None, channels=None, n_threads: int = 0,
                     refit: bool = False, gate: bool = False):
        """Lockstep check (V1, V2, V4, V4x and S4's stop decision) of another
        implementation's fit with Algorithm 2's stopping rule (gate: reading F1)."""
        return self._verify(W, bits, max_points, n_grid, 0.0, X, eps, relative, refit, codes_,
                            scales, counts, err, xerr, grid, channels, n_threads, gate=gate)

    def output_error(self, W, codes_, scales, counts, X, channels=None, with_ref=True, n_threads: int = 0,
                     offsets=None):
        """Eq. (12) in fp64 (offsets: reading B2). Returns (err, ref) for the listed channels."""
        W = np.ascontiguousarray(W, dtype=np.float32)
        C, d = W.shape
        P = codes_.shape[1]
        X = np.ascontiguousarray(X, dtype=np.float32)
        assert X.shape[0] == d
        N = X.shape[1]
        chan = None if channels is None else np.ascontiguousarray(channels, dtype=np.int64)
        n = C if chan is None else chan.size
        err = np.zeros(n, np.float64)
        ref = np.zeros(n, np.float64) if with_ref else None
        off = None if offsets is None else np.ascontiguousarray(offsets, dtype=np.float32)
        rc = self.lib.oracle_output_error_ex(
            _p(W), _p(off), _p(np.ascontiguousarray(codes_, dtype=np.int8)),
            _p(np.ascontiguousarray(scales, dtype=np.float32)),
            _p(np.ascontiguousarray(counts, dtype=np.int32)), C, d, P, _p(X), N,
            _p(chan), 0 if chan is None else chan.size, _p(err), _p(ref), n_threads)
        if rc != 0:
            raise MemoryError("oracle_output_error failed")
        return err, ref

    def reconstruct(self, codes_, scales, counts, offsets=None) -> np.ndarray:
        codes_ = np.ascontiguousarray(codes_, dtype=np.int8)
        C, P, d = codes_.shape
        out = np.zeros((C, d), np.float32)
        off = None if offsets is None else np.ascontiguousarray(offsets, dtype=np.float32)
        self.lib.oracle_reconstruct_ex(_p(off), _p(codes_),
                                      _p(np.ascontiguousarray(scales, dtype=np.float32)),
                                      _p(np.ascontiguousarray(counts, dtype=np.int32)), C, d, P,
                                      _p(out))
        return out

    def integer_scales(self, scales, counts, p: int):
        """Eq. (14) (reading I1). Returns (A [C,P] int32, number clamped)."""
        scales = np.ascontiguousarray(scales, dtype=np.float32)
        counts = np.ascontiguousarray(counts, dtype=np.int32)
        C, P = scales.shape
        A = np.zeros((C, P), np.int32)
        n = self.lib.oracle_integer_scales(_p(scales), _p(counts), C, P, int(p), _p(A))
        return A, int(n)

    def integer_forward(self, codes_, A, counts, X, p: int):
        """Eq. (15), Steps 1-3 (readings B1, I2).  codes [C,P,d] int8, A [C,P]
        int32, X [N,d] int8.  Returns Y [C,N] int64."""
        codes_ = np.ascontiguousarray(codes_, dtype=np.int8)
        C, P, d = codes_.shape
        X = np.ascontiguousarray(X, dtype=np.int8)
        assert X.shape[1] == d
        N = X.shape[0]
        Y = np.zeros((C, N), np.int64)
        rc = self.lib.oracle_integer_forward(
            _p(codes_), _p(np.ascontiguousarray(A, dtype=np.int32)),
            _p(np.ascontiguousarray(counts, dtype=np.int32)), C, d, P, _p(X), N, int(p), _p(Y))
        if rc != 0:
            raise OverflowError("oracle_integer_forward: a sum left its integer range")
        return Y


def _delegate(name):
    def f(*args, **kw):
        return getattr(load(), name)(*args, **kw)
    f.__name__ = name
    f.__doc__ = getattr(Oracle, name).__doc__
    return f


for _n in ("levels", "default_grid", "candidate_scales", "codes", "scale_error", "fit",
           "verify", "fit_calib", "verify_calib", "output_error", "reconstruct",
           "integer_scales", "integer_forward", "fit_clip", "verify_clip", "fit_paper",
           "verify_paper", "min_gap", "paper_grid", "paper_grid_search", "fit_asym",
           "verify_asym"):
    globals()[_n] = _delegate(_n)
