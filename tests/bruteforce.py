"""Brute-force and closed-form references that pin the oracle.

None of this imports the oracle's arithmetic; each function computes its
answer a different way (exhaustive enumeration, least squares, exact
piecewise-quadratic minimisation), so a mistake in the oracle shows up as a
disagreement.
"""
from __future__ import annotations

import itertools

import numpy as np


def all_code_vectors(d: int, M: int) -> np.ndarray:
    """Every vector of {-M..M}^d, shape ((2M+1)^d, d)."""
    levels = np.arange(-M, M + 1, dtype=np.int64)
    return np.array(list(itertools.product(levels, repeat=d)), dtype=np.float64)


def best_code_vector(r: np.ndarray, a: float, M: int):
    """argmin over all code vectors q of ||r - a q||^2 (Eq. (8) by enumeration).

    Returns (q, E_min, n_minimisers) where n_minimisers counts vectors whose
    error is within 1e-12 relative of the minimum (ties)."""
    Q = all_code_vectors(r.size, M)
    E = ((r[None, :] - a * Q) ** 2).sum(axis=1)
    i = int(np.argmin(E))
    n_min = int(np.sum(E <= E[i] * (1 + 1e-12) + 1e-300))
    return Q[i].astype(np.int64), float(E[i]), n_min


def global_single_point_optimum(r: np.ndarray, M: int) -> float:
    """min over all nonzero q and all real a of ||r - a q||^2 (least squares)."""
    Q = all_code_vectors(r.size, M)
    qq = (Q * Q).sum(axis=1)
    rq = Q @ r
    keep = qq > 0
    return float(r @ r - np.max(rq[keep] ** 2 / qq[keep]))


def range_single_point_optimum(r: np.ndarray, M: int, amax: float) -> float:
    """min over all q and a in (0, amax] of ||r - a q||^2 (enumeration + LS)."""
    Q = all_code_vectors(r.size, M)
    qq = (Q * Q).sum(axis=1)
    rq = Q @ r
    a = np.where(qq > 0, np.clip(rq / np.maximum(qq, 1.0), 0.0, amax), 0.0)
    E = r @ r - 2.0 * a * rq + a * a * qq
    return float(E.min())


def continuum_scale_optimum(r: np.ndarray, M: int, amax: float) -> float:
    """Exact min of E(a) = ||r - a [r/a]_Q||^2 over a in (0, amax].

    E is continuous and quadratic in a between the breakpoints |r_j|/(k+1/2)
    where an element changes code.  On each piece the codes are fixed, so
    the piece's minimum is the clipped least-squares scale.  No code vectors
    are enumerated, so this is independent of ``range_single_point_optimum``.
    """
    x = np.abs(r.astype(np.float64))
    bps = [x[j] / (k + 0.5) for j in range(x.size) for k in range(M) if x[j] > 0]
    pts = sorted({b for b in bps if 0 < b < amax} | {amax})
    lo = 0.0
    best = float(x @ x)               # the a -> 0+ limit (all codes clipped... or zero)
    for hi in pts:
        mid = 0.5 * (lo + hi)
        q = np.clip(np.rint(x / mid), 0, M)
        sqq = float(q @ q)
        srq = float(q @ x)
        if sqq > 0:
            a = min(max(srq / sqq, lo), hi)
            if a > 0:
                best = min(best, float(x @ x - 2 * a * srq + a * a * sqq))
        lo = hi
    return best


def joint_two_point_optimum(r: np.ndarray, M: int) -> float:
    """min over (q1, q2, a1, a2) of ||r - a1 q1 - a2 q2||^2 (Eq. (5), n = 2)."""
    Q = all_code_vectors(r.size, M)
    Q = Q[(Q * Q).sum(axis=1) > 0]
    best = float(r @ r)
    G = Q @ Q.T
    b = Q @ r
    diag = np.diag(G)
    best = min(best, float(r @ r - np.max(b * b / diag)))
    for i in range(Q.shape[0]):
        g11 = diag[i]
        g12 = G[i]
        g22 = diag
        det = g11 * g22 - g12 * g12
        ok = det > 1e-12
        b1, b2 = b[i], b
        # projection energy b^T G^-1 b for the 2x2 system
        proj = np.where(ok, (g22 * b1 * b1 - 2 * g12 * b1 * b2 + g11 * b2 * b2) /
                        np.where(ok, det, 1.0), 0.0)
        best = min(best, float(r @ r - proj.max()))
    return best


def residual_chain(w: np.ndarray, codes: np.ndarray, scales: np.ndarray, n: int):
    """Residuals r_1 = w, r_{i+1} = r_i - a_i q_i in fp64 (Eq. (7))."""
    r = [w.astype(np.float64)]
    for i in range(n):
        r.append(r[-1] - np.float64(scales[i]) * codes[i].astype(np.float64))
    return r


def hadamard(n: int) -> np.ndarray:
    """Sylvester Hadamard matrix of order n (a power of two); H H^T = n I."""
    H = np.array([[1.0]])
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    return H
