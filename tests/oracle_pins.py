"""Pins of the oracle: each check compares it with something other than itself.

Every ``check_*`` takes an ``oracle.Oracle`` and raises AssertionError when
the oracle disagrees with the paper, a closed form, brute force or a library
routine.  ``test_oracle_pins.py`` runs them on the oracle;
``test_oracle_mutants.py`` runs them on deliberately broken copies of the
oracle and requires every copy to fail at least one check.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _golden(name):
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    return next(c for c in cases if c["name"] == name)


def _fl32(x):
    return float(np.float32(x))


# ---------------------------------------------------------------- Eq. (1)-(3)
def check_levels(orc):
    """Eq. (1): [-1 : eps_b : 1] with eps_b = 1/(2^(b-1)-1) has 2M+1 points."""
    for b in range(2, 9):
        eps = 1.0 / (2 ** (b - 1) - 1)
        n_points = int(round(2.0 / eps)) + 1
        assert 2 * orc.levels(b) + 1 == n_points, b


def check_rounding_ties(orc):
    """Eq. (2) at exact half-way points against numpy's round-half-even."""
    g = _golden("rounding_half_ties_to_even")
    r = np.array(g["r"], np.float64)
    q = orc.codes(r, g["a"], g["bits"])
    M = 2 ** (g["bits"] - 1) - 1
    lib = np.clip(np.round(r / g["a"]), -M, M).astype(np.int64)   # numpy rounds half to even
    assert q.tolist() == g["expect_codes"] == lib.tolist(), (q, lib)


def check_codes_bruteforce(orc):
    """P-a: [r/a]_Q (Eq. (8)) equals the minimiser over all (2M+1)^d code vectors."""
    rng = np.random.default_rng(11)
    for bits, d in ((2, 6), (3, 4), (4, 3), (4, 4)):
        M = 2 ** (bits - 1) - 1
        for _ in range(6):
            r = rng.standard_normal(d)
            m = np.abs(r).max()
            a = float(rng.uniform(0.05, 1.0) * m / M) if rng.random() < 0.7 \
                else float(rng.uniform(0.02, 0.3) * m)
            q = orc.codes(r, a, bits)
            qb, Eb, nmin = bf.best_code_vector(r, a, M)
            assert nmin == 1
            assert q.tolist() == qb.tolist(), (bits, r, a, q, qb)
            assert abs(orc.scale_error(r, a, bits) - Eb) <= 1e-12 * max(Eb, 1e-300)


def _first_step(orc, r, bits, G, grid=None):
    """Error and scale after one point of the oracle's fit (P=1, tol=0)."""
    W = np.asarray(r, np.float32)[None, :]
    codes, scales, counts, err = orc.fit(W, bits, 1, G, 0.0, grid=grid)
    return float(err[0, 0]), float(scales[0, 0]), codes[0, 0], int(counts[0])


def check_grid_search_bruteforce(orc):
    """Eq. (9): the chosen scale minimises, over the candidates of reading G2,
    the brute-force error min_q ||r - a q||^2; the tie rule picks the first."""
    rng = np.random.default_rng(12)
    for bits, d, G in ((2, 5, 16), (3, 4, 8), (4, 3, 32)):
        M = 2 ** (bits - 1) - 1
        for _ in range(4):
            r = rng.standard_normal(d).astype(np.float32).astype(np.float64)
            m = _fl32(np.abs(r).max())
            cands = [_fl32(m * _fl32((g + 1) / G) / M) for g in range(G)]
            Eb = [bf.best_code_vector(r, a, M)[1] for a in cands]
            gbest = int(np.argmin(Eb))
            e0, a0, q0, n0 = _first_step(orc, r, bits, G)
            assert n0 == 1
            assert a0 == cands[gbest], (a0, cands[gbest])
            assert abs(e0 - Eb[gbest]) <= 1e-12 * Eb[gbest]
            assert q0.tolist() == bf.best_code_vector(r, a0, M)[0].tolist()


def check_grid_search_bounds(orc):
    """P-b: the grid-search error is bounded below by the continuum optimum
    over the range (0, max|r|/M], which is bounded below by the global
    single-point optimum; refining a nested grid never hurts and converges."""
    rng = np.random.default_rng(13)
    for bits, d in ((2, 6), (3, 4), (4, 3)):
        M = 2 ** (bits - 1) - 1
        for _ in range(3):
            r = rng.standard_normal(d).astype(np.float32).astype(np.float64)
            amax = _fl32(_fl32(np.abs(r).max()) / M)       # largest candidate (c_G = 1)
            e_cont = bf.continuum_scale_optimum(r, M, amax)
            e_range = bf.range_single_point_optimum(r, M, amax)
            e_glob = bf.global_single_point_optimum(r, M)
            assert abs(e_cont - e_range) <= 1e-9 * max(e_range, 1e-12), (e_cont, e_range)
            assert e_glob <= e_range * (1 + 1e-12)
            gaps = []
            for G in (16, 256, 4096):
                e, *_ = _first_step(orc, r, bits, G)
                assert e >= e_range * (1 - 1e-9), (G, e, e_range)
                gaps.append(e - e_range)
            assert gaps[2] <= gaps[1] + 1e-15 and gaps[1] <= gaps[0] + 1e-15, gaps
            assert gaps[2] <= 2e-3 * (r @ r), gaps


def check_two_point_joint(orc):
    """P-b: the greedy two-point error is no better than the joint optimum of Eq. (5)."""
    rng = np.random.default_rng(14)
    for bits, d in ((2, 4), (3, 3)):
        M = 2 ** (bits - 1) - 1
        for _ in range(3):
            r = rng.standard_normal(d).astype(np.float32)
            codes, scales, counts, err = orc.fit(r[None, :], bits, 2, 64, 0.0)
            if counts[0] < 2:
                continue
            ej = bf.joint_two_point_optimum(r.astype(np.float64), M)
            assert err[0, 1] >= ej * (1 - 1e-9) - 1e-15, (err[0, 1], ej)


def check_naive_quantizer(orc):
    """P-c: one candidate (grid {1}) and one point is ordinary symmetric
    per-channel max-abs quantization; compared with torch's fake quantizer."""
    import torch
    rng = np.random.default_rng(15)
    for bits in (3, 4, 8):
        M = 2 ** (bits - 1) - 1
        W = (rng.standard_normal((16, 200)) * np.exp(rng.standard_normal((16, 1)))).astype(np.float32)
        codes, scales, counts, err = orc.fit(W, bits, 1, 1, 0.0, grid=np.array([1.0], np.float32))
        wt = torch.from_numpy(W)
        s = wt.abs().amax(dim=1) / M                       # fp32 scale max|w|/M
        assert np.array_equal(scales[:, 0], s.numpy()), bits
        fq = torch.fake_quantize_per_channel_affine(wt, s, torch.zeros(16, dtype=torch.int32),
                                                    0, -M, M)
        qt = torch.round(fq / s[:, None]).to(torch.int64).numpy()
        t = W.astype(np.float64) / s.numpy().astype(np.float64)[:, None]
        near_half = np.abs(np.abs(t - np.floor(t)) - 0.5) < 1e-5
        ok = (codes[:, 0, :] == qt) | near_half
        assert ok.all(), bits
        assert (counts == 1).all()


def check_equal_magnitudes(orc):
    """P-d: all |w_j| equal (and d = 1): one point, codes sign(w)*M, scale fl32(m/M)."""
    for bits in (2, 3, 4, 8):
        M = 2 ** (bits - 1) - 1
        for w in ([0.3, -0.3, 0.3, 0.3, -0.3], [-1.7]):
            W = np.array([w], np.float32)
            codes, scales, counts, err = orc.fit(W, bits, 4, 64, 1e-3)
            m = float(np.float32(abs(w[0])))
            assert counts[0] == 1, (bits, counts)
            assert scales[0, 0] == np.float32(m / M)
            assert codes[0, 0].tolist() == [int(np.sign(x)) * M for x in w]


def check_worked_examples(orc):
    """P-e and the stop-boundary case, derived by hand (tests/golden)."""
    g = _golden("two_elements_exact_tie")
    W = np.array([g["w"]], np.float32)
    codes, scales, counts, err = orc.fit(W, g["bits"], g["max_points"], g["n_grid"], g["tol"])
    e = g["expect"]
    assert counts[0] == e["count"]
    assert scales[0].tolist() == e["scales"]
    assert codes[0].tolist() == e["codes"]
    assert err[0].tolist() == e["err"]
    g = _golden("stop_exactly_at_tolerance")
    W = np.array([g["w"]], np.float32)
    for v in g["variants"]:
        codes, scales, counts, err = orc.fit(W, g["bits"], g["max_points"], g["n_grid"],
                                             float(np.float32(v["tol"])))
        assert counts[0] == v["count"], v
        assert scales[0].tolist() == v["scales"]
        assert err[0].tolist() == v["err"]
        assert codes[0, 0].tolist() == v["codes_point0"]
        if "codes_point1" in v:
            assert codes[0, 1].tolist() == v["codes_point1"]


def check_monotone_decrease(orc):
    """P-f: ||r_{i+1}||^2 <= ||r_i||^2 - max|r_i|^2 (+1e-6 ||r_i||^2 slack);
    err[i] is ||r_{i+1}||^2 of the residual chain of Eq. (7)."""
    rng = np.random.default_rng(16)
    for bits, G in ((2, 64), (3, 128), (4, 256), (8, 64)):
        W = (rng.standard_normal((12, 97)) * np.exp(0.5 * rng.standard_normal((12, 1)))).astype(np.float32)
        W[3, :50] = 0.0
        codes, scales, counts, err = orc.fit(W, bits, 5, G, 0.0)
        for k in range(W.shape[0]):
            n = int(counts[k])
            rs = bf.residual_chain(W[k], codes[k], scales[k], n)
            for i in range(n):
                e0 = float(rs[i] @ rs[i])
                e1 = float(rs[i + 1] @ rs[i + 1])
                m = float(np.abs(rs[i]).max())
                assert e1 <= e0 - m * m + 1e-6 * e0, (bits, k, i, e0, e1, m)
                assert abs(err[k, i] - e1) <= 1e-12 * max(e0, 1e-300)


def check_reconstruct(orc):
    """P-g: reconstruct = sum_i a_i q_i (Eq. (4)); ||w - w~||^2 equals the last err."""
    rng = np.random.default_rng(17)
    W = (rng.standard_normal((10, 77)) * 0.1).astype(np.float32)
    codes, scales, counts, err = orc.fit(W, 4, 4, 128, 1e-4)
    Wh = orc.reconstruct(codes, scales, counts)
    ref = np.einsum("kp,kpj->kj", scales.astype(np.float64) *
                    (np.arange(4)[None, :] < counts[:, None]), codes.astype(np.float64))
    assert np.array_equal(Wh, ref.astype(np.float32))
    for k in range(10):
        n = counts[k]
        e = float(((W[k].astype(np.float64) - Wh[k].astype(np.float64)) ** 2).sum())
        assert abs(e - err[k, n - 1]) <= 1e-5 * err[k, n - 1] + 1e-12 * float(W[k] @ W[k])


def check_invariances(orc):
    """P-h: w -> -w negates codes; w -> 2^k w scales the scales by 2^k;
    permuting elements permutes codes."""
    rng = np.random.default_rng(18)
    W = (rng.standard_normal((8, 60)) * 0.2).astype(np.float32)
    base = orc.fit(W, 4, 4, 128, 1e-3)
    neg = orc.fit(-W, 4, 4, 128, 1e-3)
    assert np.array_equal(neg[0], -base[0]) and np.array_equal(neg[1], base[1])
    assert np.array_equal(neg[2], base[2])
    for k in (-3, 5):
        sc = orc.fit((W * np.float32(2.0 ** k)).astype(np.float32), 4, 4, 128, 1e-3)
        assert np.array_equal(sc[0], base[0]) and np.array_equal(sc[2], base[2])
        assert np.array_equal(sc[1], (base[1] * np.float32(2.0 ** k)).astype(np.float32))
    perm = rng.permutation(60)
    pe = orc.fit(np.ascontiguousarray(W[:, perm]), 4, 4, 128, 1e-3)
    assert np.array_equal(pe[2], base[2])
    assert np.array_equal(pe[0], base[0][:, :, perm])
    assert np.array_equal(pe[1], base[1])


def check_output_error(orc):
    """P-i: with X X^T = N I the output error equals ||w - w~||^2; for random X
    it equals a numpy fp64 matmul (Eq. (12), mean over the batch)."""
    rng = np.random.default_rng(19)
    d, N = 24, 64
    W = (rng.standard_normal((6, d)) * 0.3).astype(np.float32)
    codes, scales, counts, err = orc.fit(W, 3, 3, 64, 1e-2)
    H = bf.hadamard(N)[:d].astype(np.float32)          # rows orthogonal, norm^2 = N
    e, r = orc.output_error(W, codes, scales, counts, H)
    for k in range(6):
        n = counts[k]
        assert abs(e[k] - err[k, n - 1]) <= 1e-10 * err[k, n - 1]
        assert abs(r[k] - float(W[k].astype(np.float64) @ W[k].astype(np.float64))) <= 1e-10 * r[k]
    X = rng.standard_normal((d, 37)).astype(np.float32)
    e, r = orc.output_error(W, codes, scales, counts, X)
    Wh = np.einsum("kp,kpj->kj", scales.astype(np.float64) * (np.arange(3)[None, :] < counts[:, None]),
                   codes.astype(np.float64))
    D = W.astype(np.float64) - Wh
    ye = D @ X.astype(np.float64)
    yr = W.astype(np.float64) @ X.astype(np.float64)
    assert np.allclose(e, (ye ** 2).mean(axis=1), rtol=1e-9, atol=0)
    assert np.allclose(r, (yr ** 2).mean(axis=1), rtol=1e-9, atol=0)
    sub = np.array([4, 1], np.int64)
    e2, r2 = orc.output_error(W, codes, scales, counts, X, channels=sub)
    assert np.array_equal(e2, e[sub]) and np.array_equal(r2, r[sub])


def check_stop_rule(orc):
    """S1-S3: tol >= 1 gives one point; a zero channel gets none; tol = 0 runs
    to the cap unless the residual vanishes."""
    rng = np.random.default_rng(20)
    W = (rng.standard_normal((5, 40)) * 0.2).astype(np.float32)
    W[2] = 0.0
    c1 = orc.fit(W, 4, 6, 64, 1.0)[2]
    assert c1.tolist() == [1, 1, 0, 1, 1]
    c0 = orc.fit(W, 4, 6, 64, 0.0)[2]
    assert c0.tolist() == [6, 6, 0, 6, 6]
    # every candidate scale of a channel at the bottom of the fp32 range
    # rounds to zero (max|w| / 7 is below half the smallest subnormal): no point
    tiny = np.array([[1e-45, 0.0, -1e-45]], np.float32)
    assert orc.fit(tiny, 4, 6, 64, 0.0)[2].tolist() == [0]
    # with bits = 2 (M = 1) the largest candidate equals max|w| and is nonzero
    c, s, n, e = orc.fit(tiny, 2, 6, 64, 0.0)
    assert n.tolist() == [1] and s[0, 0] == np.float32(1e-45) and c[0, 0].tolist() == [1, 0, -1]


def check_exponential_decay(orc):
    """Theorem 1 (qualitative): log ||r_i|| falls roughly linearly in i.
    Parity unpinned for the rate: the constants are not given."""
    rng = np.random.default_rng(21)
    W = rng.standard_normal((4, 256)).astype(np.float32)
    codes, scales, counts, err = orc.fit(W, 2, 8, 1024, 0.0)
    for k in range(4):
        e = np.concatenate([[float(W[k].astype(np.float64) @ W[k].astype(np.float64))], err[k]])
        ratios = e[1:] / e[:-1]
        assert (ratios < 0.9).all(), ratios


def check_verifier(orc):
    """The lockstep verifier accepts the oracle's own output and flags
    planted mistakes (wrong count, off-grid scale, worse candidate, wrong
    code, dirty unused slot, wrong err)."""
    rng = np.random.default_rng(22)
    W = (rng.standard_normal((6, 50)) * np.exp(0.5 * rng.standard_normal((6, 1)))).astype(np.float32)
    bits, P, G, tol = 4, 4, 64, 1e-3
    codes, scales, counts, err = orc.fit(W, bits, P, G, tol)
    ok = orc.verify(W, bits, P, G, tol, codes, scales, counts, err.astype(np.float32))
    assert (ok["status"] == 0).all() and ok["cand_ties"].sum() == 0 and ok["code_ties"].sum() == 0
    assert (ok["err_relmax"] < 1e-6).all()

    def status(c, s, n, e):
        return orc.verify(W, bits, P, G, tol, c, s, n, e)["status"][0]

    e32 = err.astype(np.float32)
    n2 = counts.copy(); n2[0] = n2[0] + 1 if n2[0] < P else n2[0] - 1
    assert status(codes, scales, n2, None) != 0
    s2 = scales.copy(); s2[0, 0] = np.nextafter(s2[0, 0], np.float32(1))
    assert status(codes, s2, counts, None) == 2
    r = W[0].astype(np.float64)
    m = _fl32(np.abs(r).max())
    cands = np.array([_fl32(m * _fl32((g + 1) / G) / 7) for g in range(G)], np.float32)
    E = [orc.scale_error(r, float(a), bits) for a in cands]
    worst = int(np.argmax(E))
    s3 = scales.copy(); s3[0, 0] = cands[worst]
    c3 = codes.copy(); c3[0, 0] = orc.codes(r, float(cands[worst]), bits)
    assert status(c3, s3, counts, None) == 3
    c4 = codes.copy(); c4[0, 0, 7] += 1 if c4[0, 0, 7] < 7 else -1
    assert status(c4, scales, counts, None) == 4
    c5 = codes.copy(); c5[0, P - 1, 3] = 1
    if counts[0] < P:
        assert status(c5, scales, counts, None) == 5
    e6 = e32.copy(); e6[0, 0] *= 1.001
    assert status(codes, scales, counts, e6) == 6


# ------------------------------------------- S4: Algorithm 2 on a batch X
def _calib_case(seed=21, C=10, d=24, N=40):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((C, d)) * np.exp(0.5 * rng.standard_normal((C, 1)))).astype(np.float32)
    W[C - 1] = 0.0                                   # an all-zero channel
    # correlated, non-isotropic inputs (ReLU of mixed Gaussians), d != N
    X = np.maximum(rng.standard_normal((d, N)) + 0.5 * rng.standard_normal((1, N)), 0.0)
    return W, X.astype(np.float32)


def _numpy_output_errors(W, X, codes, scales, counts):
    """e_n of Eq. (12) for n = 1..count, from the outputs, in numpy fp64."""
    out = []
    Xd = X.astype(np.float64)
    for k in range(W.shape[0]):
        D = W[k].astype(np.float64)
        es = []
        for i in range(counts[k]):
            D = D - float(scales[k, i]) * codes[k, i].astype(np.float64)
            es.append(float(np.mean((D @ Xd) ** 2)))
        out.append(es)
    return out


def check_calib_hadamard_is_isotropic(orc):
    """S4 with X X^T = N I: e_n = ||r_n||^2 and the relative threshold is
    eps ||w||^2, so the fit equals the isotropic rule S1 with tol = eps."""
    rng = np.random.default_rng(5)
    d, N = 48, 64
    X = bf.hadamard(N)[:d].astype(np.float32)
    W = rng.standard_normal((12, d)).astype(np.float32)
    for bits, P, G, eps in ((4, 6, 64, 1e-3), (3, 8, 32, 2e-3), (2, 5, 16, 0.05)):
        c1, s1, n1, e1, x1 = orc.fit_calib(W, bits, P, G, X, eps, True)
        c0, s0, n0, e0 = orc.fit(W, bits, P, G, eps)
        assert np.array_equal(n1, n0) and np.array_equal(s1, s0) and np.array_equal(c1, c0)
        assert np.allclose(x1, e0, rtol=1e-9, atol=0)


def check_calib_stop_definition(orc):
    """S4 against its definition: the reported output errors are Eq. (12)
    of the outputs (numpy fp64), the count is the first n >= 1 with
    e_n <= thr (else max_points), and the points are the isotropic fit's
    (Algorithm 1 does not see X)."""
    W, X = _calib_case()
    ref = np.mean((W.astype(np.float64) @ X.astype(np.float64)) ** 2, axis=1)
    for bits, P, G, eps, rel in ((4, 6, 64, 3e-3, True), (3, 8, 32, 1e-2, True),
                                 (4, 6, 64, 0.02 * float(np.median(ref)), False)):
        codes, scales, counts, err, xerr = orc.fit_calib(W, bits, P, G, X, eps, rel)
        es = _numpy_output_errors(W, X, codes, scales, counts)
        c0, s0, n0, _ = orc.fit(W, bits, P, G, 0.0)
        for k in range(W.shape[0]):
            thr = eps * ref[k] if rel else eps
            n = counts[k]
            assert np.allclose(xerr[k, :n], es[k], rtol=1e-10, atol=1e-300), k
            assert (xerr[k, n:] == 0).all()
            if not W[k].any():
                assert n == 0
                continue
            assert n >= 1
            assert all(e > thr for e in es[k][:-1]), (k, es[k], thr)
            assert n == P or es[k][-1] <= thr, (k, es[k], thr)
            assert np.array_equal(codes[k, :n], c0[k, :n]) and np.array_equal(scales[k, :n], s0[k, :n])


def check_calib_runs_to_cap(orc):
    """S4 with an absolute threshold of 0: no output error of a random
    channel reaches 0 within the cap, so every nonzero channel takes exactly
    max_points points, and a tiny cap binds before any threshold does."""
    W, X = _calib_case(seed=12)
    for P in (1, 2, 5):
        codes, scales, counts, err, xerr = orc.fit_calib(W, 4, P, 32, X, 0.0, False)
        assert (counts[:-1] == P).all() and counts[-1] == 0, (P, counts)
        assert (xerr[:-1, P - 1] > 0).all()


def check_calib_zero_batch(orc):
    """S4 with X = 0: every output error is 0 <= thr, so a nonzero channel
    stops after the one point S2 requires."""
    W, X = _calib_case(seed=8)
    X = np.zeros_like(X)
    for rel in (True, False):
        codes, scales, counts, err, xerr = orc.fit_calib(W, 4, 5, 32, X, 0.0, rel)
        assert (counts[:-1] == 1).all() and counts[-1] == 0, counts


def check_calib_scaling(orc):
    """S4 is invariant to X -> 2X with a relative threshold, and with an
    absolute one when eps -> 4 eps (e scales by 4)."""
    W, X = _calib_case(seed=9)
    a = orc.fit_calib(W, 4, 6, 64, X, 3e-3, True)
    b = orc.fit_calib(W, 4, 6, 64, 2 * X, 3e-3, True)
    assert all(np.array_equal(u, v) for u, v in zip(a[:3], b[:3]))
    eps = 0.01 * float(np.median(a[4][:, 0]))
    c = orc.fit_calib(W, 4, 6, 64, X, eps, False)
    e = orc.fit_calib(W, 4, 6, 64, 2 * X, 4 * eps, False)
    assert all(np.array_equal(u, v) for u, v in zip(c[:3], e[:3]))
    assert np.allclose(e[4], 4 * c[4], rtol=1e-12, atol=0)


def check_calib_verifier(orc):
    """The S4 verifier accepts the oracle's own fit and flags a wrong count
    and a wrong output-error value."""
    W, X = _calib_case(seed=10)
    P, G, eps = 6, 64, 3e-3
    codes, scales, counts, err, xerr = orc.fit_calib(W, 4, P, G, X, eps, True)
    e32, x32 = err.astype(np.float32), xerr.astype(np.float32)

    def status(c, s, n, e, x):
        v = orc.verify_calib(W, 4, P, G, X, eps, True, c, s, n, e, x)
        return int(v["status"].max())

    assert status(codes, scales, counts, e32, x32) == 0
    k = int(np.argmax((counts >= 1) & (counts < P)))
    n2 = counts.copy(); n2[k] += 1
    c2 = codes.copy(); s2 = scales.copy()
    c3, s3, _, _ = orc.fit(W, 4, P, G, 0.0)
    c2[k], s2[k] = c3[k], s3[k]          # one more genuine point, zero slots after it
    c2[k, n2[k]:] = 0; s2[k, n2[k]:] = 0
    assert status(c2, s2, n2, None, None) == 1
    x8 = x32.copy(); x8[k, 0] *= 1.001
    assert status(codes, scales, counts, e32, x8) == 8


def check_calib_verifier_fp32_evaluation(orc):
    """The S4 verifier accepts output errors evaluated as the GPU does (the
    difference rounded to fp32, fp32 products and sums: numpy float32
    matmul), also for one- and three-column batches whose outputs can nearly
    cancel, and still flags a 1e-4 relative change of a well-averaged one."""
    rng = np.random.default_rng(17)
    d, P = 300, 5
    W = rng.standard_normal((200, d)).astype(np.float32)
    for N in (1, 3, 512):
        X = rng.standard_normal((d, N)).astype(np.float32)
        codes, scales, counts, err, xerr = orc.fit_calib(W, 4, P, 64, X, 1e-3, True)
        x32 = np.zeros((W.shape[0], P), np.float32)
        for k in range(W.shape[0]):
            D = W[k].astype(np.float64)
            for i in range(counts[k]):
                D = D - float(scales[k, i]) * codes[k, i].astype(np.float64)
                y = D.astype(np.float32) @ X
                x32[k, i] = np.float32(np.mean(y.astype(np.float64) ** 2))
        v = orc.verify_calib(W, 4, P, 64, X, 1e-3, True, codes, scales, counts, None, x32)
        assert (v["status"] == 0).all(), (N, np.nonzero(v["status"])[0][:5])
        if N == 512:
            x32[:, 0] *= np.float32(1 + 1e-4)
            v = orc.verify_calib(W, 4, P, 64, X, 1e-3, True, codes, scales, counts, None, x32)
            assert (v["status"] == 8).all()


# ------------------------------------------- reading F1: Algorithm 2's naive first point
def _naive_point(w, bits):
    """The naive quantization [w]_Q of Algorithm 2 in numpy: code step
    fl32(fl32(max|w|) / M), codes rounded half to even and clipped."""
    M = 2 ** (bits - 1) - 1
    a = np.float32(np.float64(np.float32(np.abs(w).max())) / M)
    if a == 0:
        return a, np.zeros(w.shape, np.int8)
    q = np.clip(np.round(w.astype(np.float64) / np.float64(a)), -M, M)
    return a, q.astype(np.int8)


def check_gate_worked_example(orc):
    """Reading F1 on the hand-derived case (tests/golden): the naive point is
    kept when its output error passes, and discarded (Algorithm 1 from w)
    when it does not."""
    g = _golden("naive_first_gate")
    W = np.array([g["w"]], np.float32)
    for v in g["variants"]:
        X = np.array(v["X"], np.float32)
        for key, gate in (("gate", True), ("no_gate", False)):
            c, s, n, _, x = orc.fit_calib(W, g["bits"], g["max_points"], g["n_grid"], X,
                                          g["eps"], False, gate=gate)
            e = v[key]
            assert n[0] == e["count"], (key, v["X"], n)
            assert s[0].tolist() == e["scales"], (key, s)
            assert c[0].tolist() == e["codes"], (key, c)
            assert x[0].tolist() == e["xerr"], (key, x)


def _gate_threshold(values):
    """A threshold halfway between two well-separated sorted values, so that
    about half the channels pass and none sits near it."""
    v = np.sort(np.asarray(values, np.float64))
    gaps = np.diff(v) / np.maximum(v[1:], 1e-300)
    lo = len(v) // 4
    i = lo + int(np.argmax(gaps[lo:len(v) - lo]))
    return 0.5 * (v[i] + v[i + 1])


def check_gate_definition(orc):
    """Reading F1 against its definition, per channel, in numpy: the naive
    point of Algorithm 2 is kept (count 1) when its error under the rule in
    force is at most the threshold; otherwise the fit is exactly the fit
    without the gate (Algorithm 1 from w)."""
    W, X = _calib_case(seed=31, C=24, d=40, N=50)
    Xd = X.astype(np.float64)
    # P = 1: the cap bounds Algorithm 1 only, so a failing naive point still
    # gives way to Algorithm 1's first point
    for bits, P, G in ((4, 6, 64), (3, 5, 32), (4, 1, 64)):
        eN, EN = [], []
        for k in range(W.shape[0]):
            a, q = _naive_point(W[k], bits)
            R = W[k].astype(np.float64) - np.float64(a) * q
            eN.append(float(np.mean((R @ Xd) ** 2)))
            EN.append(float(R @ R))
        live = W.any(axis=1)
        # S4, absolute threshold
        eps = _gate_threshold(np.array(eN)[live])
        c1, s1, n1, _, x1 = orc.fit_calib(W, bits, P, G, X, eps, False, gate=True)
        c0, s0, n0, _, x0 = orc.fit_calib(W, bits, P, G, X, eps, False)
        kept = 0
        for k in range(W.shape[0]):
            if not live[k]:
                assert n1[k] == 0
                continue
            a, q = _naive_point(W[k], bits)
            if eN[k] <= eps:
                kept += 1
                assert n1[k] == 1 and s1[k, 0] == a and np.array_equal(c1[k, 0], q), k
                assert abs(x1[k, 0] - eN[k]) <= 1e-12 * eN[k] + 1e-300
            else:
                assert n1[k] == n0[k] and np.array_equal(s1[k], s0[k]) and np.array_equal(c1[k], c0[k])
        assert 0 < kept < live.sum()
        # S1 (isotropic), relative tolerance
        Ew = (W.astype(np.float64) ** 2).sum(axis=1)
        ratio = np.array(EN)[live] / Ew[live]
        tol = _gate_threshold(ratio)
        c1, s1, n1, _ = orc.fit(W, bits, P, G, tol, gate=True)
        c0, s0, n0, _ = orc.fit(W, bits, P, G, tol)
        for k in np.nonzero(live)[0]:
            a, q = _naive_point(W[k], bits)
            if EN[k] <= tol * Ew[k]:
                assert n1[k] == 1 and s1[k, 0] == a and np.array_equal(c1[k, 0], q), k
            else:
                assert n1[k] == n0[k] and np.array_equal(s1[k], s0[k]) and np.array_equal(c1[k], c0[k])


def check_gate_hadamard_is_isotropic(orc):
    """Reading F1 with X X^T = N I: the output error is ||r||^2 and the
    relative threshold eps ||w||^2, so the gated S4 fit equals the gated
    isotropic fit with tol = eps; the gate changes the first point of some
    channels (against the fit without it)."""
    rng = np.random.default_rng(8)
    d, N = 48, 64
    X = bf.hadamard(N)[:d].astype(np.float32)
    W = (rng.standard_normal((16, d)) * np.exp(0.3 * rng.standard_normal((16, 1)))).astype(np.float32)
    changed = 0
    for bits, P, G in ((4, 6, 64), (3, 8, 32)):
        ratio = []
        for k in range(W.shape[0]):
            a, q = _naive_point(W[k], bits)
            R = W[k].astype(np.float64) - np.float64(a) * q
            ratio.append(float(R @ R) / float(W[k].astype(np.float64) @ W[k].astype(np.float64)))
        eps = _gate_threshold(ratio)
        c1, s1, n1, e1, x1 = orc.fit_calib(W, bits, P, G, X, eps, True, gate=True)
        c0, s0, n0, e0 = orc.fit(W, bits, P, G, eps, gate=True)
        assert np.array_equal(n1, n0) and np.array_equal(s1, s0) and np.array_equal(c1, c0)
        assert np.allclose(x1, e0, rtol=1e-9, atol=0)
        cg, sg, ng, _ = orc.fit(W, bits, P, G, eps)
        changed += int(((sg[:, 0] != s0[:, 0]) & (n0 == 1)).sum())
    assert changed > 0


def check_gate_verifier(orc):
    """The verifier with reading F1 accepts gated fits (S1 and S4) and flags,
    with status 10, a fit that took Algorithm 1's point where the naive one
    passes."""
    W, X = _calib_case(seed=33, C=16, d=30, N=40)
    bits, P, G = 4, 6, 64
    eN = []
    for k in range(W.shape[0] - 1):
        a, q = _naive_point(W[k], bits)
        R = W[k].astype(np.float64) - np.float64(a) * q
        eN.append(float(np.mean((R @ X.astype(np.float64)) ** 2)))
    eps = _gate_threshold(eN)
    c1, s1, n1, e1, x1 = orc.fit_calib(W, bits, P, G, X, eps, False, gate=True)
    v = orc.verify_calib(W, bits, P, G, X, eps, False, c1, s1, n1, e1.astype(np.float32),
                         x1.astype(np.float32), gate=True)
    assert (v["status"] == 0).all(), v["status"]
    c0, s0, n0, e0, x0 = orc.fit_calib(W, bits, P, G, X, eps, False)
    v = orc.verify_calib(W, bits, P, G, X, eps, False, c0, s0, n0, None, None, gate=True)
    differs = (s0[:, 0] != s1[:, 0]) & (n1 == 1)
    assert differs.any()
    assert (v["status"][differs] == 10).all(), v["status"]
    tol = 1e-2
    c1, s1, n1, e1 = orc.fit(W, bits, P, G, tol, gate=True)
    v = orc.verify(W, bits, P, G, tol, c1, s1, n1, e1.astype(np.float32), gate=True)
    assert (v["status"] == 0).all(), v["status"]


# ------------------------------------------- reading A2: least-squares refit
def check_refit_one_point(orc):
    """One point: the codes are Eq. (10)'s at the searched scale (unchanged
    by the refit) and the scale is fl32(<w, q> / <q, q>) (numpy fp64); the
    error is never larger than without the refit."""
    rng = np.random.default_rng(31)
    W = (rng.standard_normal((60, 50)) * rng.uniform(0.1, 3, (60, 1))).astype(np.float32)
    for bits, G in ((4, 64), (2, 16), (3, 7)):
        c0, s0, n0, e0 = orc.fit(W, bits, 1, G, 0.0)
        c1, s1, n1, e1 = orc.fit(W, bits, 1, G, 0.0, refit=True)
        assert np.array_equal(c0, c1) and np.array_equal(n0, n1)
        w, q = W.astype(np.float64), c1[:, 0, :].astype(np.float64)
        a = np.float32((w * q).sum(1) / (q * q).sum(1))
        assert np.array_equal(s1[:, 0], a)
        assert (e1[:, 0] <= e0[:, 0] * (1 + 1e-15)).all()


def check_refit_residual_chain(orc):
    """Several points with the refit: the reported err equals ||w - sum a q||^2
    rebuilt from the outputs; each new residual is orthogonal to its codes up
    to the fp32 rounding of a; the error never increases."""
    rng = np.random.default_rng(32)
    W = rng.standard_normal((40, 90)).astype(np.float32)
    codes, scales, counts, err = orc.fit(W, 4, 5, 64, 0.0, refit=True)
    for k in range(40):
        r = W[k].astype(np.float64)
        prev = (r * r).sum()
        for i in range(counts[k]):
            q = codes[k, i].astype(np.float64)
            r = r - float(scales[k, i]) * q
            e = (r * r).sum()
            assert abs(e - err[k, i]) <= 1e-12 * max(err[k, i], 1e-300), (k, i)
            assert abs((r * q).sum()) <= 2.0 ** -23 * abs(float(scales[k, i])) * (q * q).sum() + 1e-300
            assert e <= prev
            prev = e


def check_refit_verifier(orc):
    """The refit verifier accepts the oracle's refit output and flags plain
    grid scales, a refit scale off by 1e-5, and (as the plain verifier) the
    refit output itself."""
    rng = np.random.default_rng(33)
    W = rng.standard_normal((30, 70)).astype(np.float32)
    codes, scales, counts, err = orc.fit(W, 4, 4, 64, 0.0, refit=True)
    e32 = err.astype(np.float32)
    v = orc.verify(W, 4, 4, 64, 0.0, codes, scales, counts, e32, refit=True)
    assert (v["status"] == 0).all()
    assert (orc.verify(W, 4, 4, 64, 0.0, codes, scales, counts, e32)["status"] == 2).all()
    c0, s0, n0, e0 = orc.fit(W, 4, 4, 64, 0.0)
    v = orc.verify(W, 4, 4, 64, 0.0, c0, s0, n0, None, refit=True)
    assert (v["status"] == 2).all()
    s2 = scales.copy()
    s2[:, 0] *= np.float32(1 + 1e-5)
    assert (orc.verify(W, 4, 4, 64, 0.0, codes, s2, counts, None, refit=True)["status"] == 2).all()


# ------------------------------------------- reading C1: clipping of Eq. (13)
def _clip_case(seed, C=25, d=40, N=30):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((C, d)) * np.exp(0.4 * rng.standard_normal((C, 1)))).astype(np.float32)
    # correlated inputs, so the output error ranks the candidates unlike ||w - a q||^2
    X = (rng.standard_normal((d, N)) + 2.0 * rng.standard_normal((1, N))).astype(np.float32)
    return W, X


def check_clip_bruteforce(orc):
    """The first point is the candidate of [0.05:0.05:1] * max|w| / M whose
    output error, in numpy fp64, is smallest (first minimum), with Eq. (10)'s
    codes at that scale."""
    W, X = _clip_case(41)
    c20 = orc.default_grid(20)
    for bits in (4, 3, 2):
        codes, scales, counts, err, _ = orc.fit_clip(W, bits, 1, 64, X)
        for k in range(W.shape[0]):
            w = W[k].astype(np.float64)
            a = orc.candidate_scales(w, bits, c20)
            e = []
            for aj in a:
                q = orc.codes(w, float(aj), bits).astype(np.float64)
                e.append(np.mean(((w - float(aj) * q) @ X.astype(np.float64)) ** 2))
            j = int(np.argmin(e))
            assert scales[k, 0] == a[j], (bits, k)
            assert np.array_equal(codes[k, 0], orc.codes(w, float(a[j]), bits))


def check_clip_hadamard_is_eq9(orc):
    """With X X^T = N I the output error is ||w - a q||^2, so the clipped
    first point is Eq. (9)'s search on the same 20-point grid."""
    rng = np.random.default_rng(42)
    W = rng.standard_normal((30, 48)).astype(np.float32)
    X = bf.hadamard(64)[:48].astype(np.float32)
    c1, s1, n1, _, _ = orc.fit_clip(W, 4, 1, 64, X)
    c0, s0, n0, _ = orc.fit(W, 4, 1, 20, 0.0)
    assert np.array_equal(s1, s0) and np.array_equal(c1, c0)


def check_clip_then_algorithm1(orc):
    """After the clipped point the fit is Algorithm 1 on the residual: the
    second scale is Eq. (9)'s argmin over the grid of the fp64 residual."""
    W, X = _clip_case(43)
    codes, scales, counts, err, _ = orc.fit_clip(W, 4, 3, 64, X)
    grid = orc.default_grid(64)
    for k in range(W.shape[0]):
        assert counts[k] == 3
        r = W[k].astype(np.float64) - float(scales[k, 0]) * codes[k, 0].astype(np.float64)
        a = orc.candidate_scales(r, 4, grid)
        E = [orc.scale_error(r, float(aj), 4) for aj in a]
        assert scales[k, 1] == a[int(np.argmin(E))], k
        assert abs(err[k, 0] - (r * r).sum()) <= 1e-12 * (r * r).sum()


def check_clip_zero_batch(orc):
    """X = 0: every candidate's output error is 0, the tie goes to the
    smallest clipping factor, 0.05 max|w|."""
    W, X = _clip_case(44)
    codes, scales, counts, err, _ = orc.fit_clip(W, 4, 1, 64, np.zeros_like(X))
    c20 = orc.default_grid(20)
    for k in range(W.shape[0]):
        assert scales[k, 0] == orc.candidate_scales(W[k].astype(np.float64), 4, c20)[0]


def check_clip_verifier(orc):
    """The clip verifier accepts the oracle's clipped fit, with either
    stopping rule, and flags fits whose first point is Eq. (9)'s."""
    W, X = _clip_case(45)
    out = orc.fit_clip(W, 4, 4, 64, X, tol=1e-3)
    v = orc.verify_clip(W, 4, 4, 64, X, *out[:3], out[3].astype(np.float32), tol=1e-3)
    assert (v["status"] == 0).all()
    out = orc.fit_clip(W, 4, 4, 64, X, calib=True, eps=1e-2)
    v = orc.verify_clip(W, 4, 4, 64, X, *out[:3], out[3].astype(np.float32), out[4].astype(np.float32),
                        calib=True, eps=1e-2)
    assert (v["status"] == 0).all()
    c0, s0, n0, e0 = orc.fit(W, 4, 4, 64, 1e-3)
    v = orc.verify_clip(W, 4, 4, 64, X, c0, s0, n0, tol=1e-3)
    assert (v["status"] != 0).mean() > 0.5
    # a genuine clipping candidate, but the one with the largest output error
    codes, scales, counts, _, _ = orc.fit_clip(W, 4, 1, 64, X)
    c20 = orc.default_grid(20)
    for k in range(W.shape[0]):
        w = W[k].astype(np.float64)
        a = orc.candidate_scales(w, 4, c20)
        e = [np.mean(((w - float(aj) * orc.codes(w, float(aj), 4)) @ X.astype(np.float64)) ** 2)
             for aj in a]
        j = int(np.argmax(e))
        scales[k, 0] = a[j]
        codes[k, 0] = orc.codes(w, float(a[j]), 4)
    v = orc.verify_clip(W, 4, 1, 64, X, codes, scales, counts)
    assert (v["status"] == 3).all()


# ------------------------------------------- Eq. (11): the paper's own grid
def check_min_gap(orc):
    """Def. 1 (reading D1), worked by hand and by pairwise brute force."""
    assert orc.min_gap([3.0, -1.0, 2.0, -3.0]) == 0.5
    assert orc.min_gap([-2.0, 2.0]) == 0.0                      # only t and -t: no gap
    assert orc.min_gap([0.5, 0.25, 0.125, -0.5]) == 0.0625
    assert orc.min_gap([3.0, 1.0, -1.0]) == 1.0                 # equal magnitudes after a gap
    rng = np.random.default_rng(51)
    for _ in range(20):
        t = rng.standard_normal(rng.integers(2, 40))
        m = np.abs(t)
        diffs = np.abs(m[:, None] - m[None, :])
        ref = diffs[diffs > 0].min() / 2 if (diffs > 0).any() else 0.0
        assert orc.min_gap(t) == ref


def check_paper_grid_size(orc):
    """Eq. (11): gamma = min(Delta / M, eta), count = floor(2 M ||r|| / gamma)."""
    r = np.array([0.75, -0.25, 0.5, 0.125])
    g, n = orc.paper_grid(r, 3, eta=2.0 ** -10)                 # M = 3, Delta = 0.0625
    assert g == 2.0 ** -10 and n == int(np.floor(2 * 3 * np.linalg.norm(r) / g))
    g, n = orc.paper_grid(r, 3, eta=0.1)
    assert g == 0.0625 / 3 and n == int(np.floor(2 * 3 * np.linalg.norm(r) / g))
    g, n = orc.paper_grid(np.array([1.0, -1.0]), 4, eta=0.01)  # no gap: eta
    assert g == 0.01


def check_paper_search_bruteforce(orc):
    """The candidate-set argmin equals the enumeration of the whole grid,
    every g from 1 to the count, errors in numpy fp64 (ties: smallest g)."""
    rng = np.random.default_rng(52)
    for bits in (2, 3, 4):
        M = 2 ** (bits - 1) - 1
        for case in range(10):
            d = int(rng.integers(2, 9))
            r = rng.integers(-96, 97, d) / 64.0                 # magnitudes 1/64 apart or equal
            if not r.any():
                continue
            eta = 2.0 ** -10 if case % 2 else 2.0 ** -6
            gamma, count = orc.paper_grid(r, bits, eta)
            a = np.arange(1, count + 1) * gamma
            q = np.clip(np.rint(r[None, :] / a[:, None]), -M, M)
            E = ((r[None, :] - a[:, None] * q) ** 2).sum(1)
            gref = int(np.argmin(E)) + 1
            g, Eg = orc.paper_grid_search(r, bits, gamma, count)
            assert E[g - 1] <= E[gref - 1] * (1 + 1e-12) and abs(Eg - E[gref - 1]) <= 1e-12 * E[gref - 1] + 1e-300
            # dyadic r and a power-of-two gamma: every error is exact, so exact
            # ties are ties on both sides and the smallest g must win
            exact = gamma == 2.0 ** np.round(np.log2(gamma))
            assert g == gref or (not exact and E[g - 1] == E[gref - 1]), (bits, case, g, gref)


def _exact_search(r, M, gamma, count):
    """Argmin of Eq. (9) over the grid a_g = fl64(g gamma), g = 1..count, with
    every error evaluated exactly: r and a are dyadic rationals, so with a
    common power of two 2^S, r_j 2^S and a 2^S are integers, the code
    [r_j / a] (ties to even, clipped) comes from an integer division, and
    E 2^(2S) is an integer.  Returns (g, exact E of every g as Fractions)."""
    from fractions import Fraction
    ratios = [float(v).as_integer_ratio() for v in r]
    a_ratios = [float(g * gamma).as_integer_ratio() for g in range(1, count + 1)]
    S = max(den.bit_length() for _, den in ratios + a_ratios)
    R = [num * ((1 << S) // den) for num, den in ratios]
    best, bestE = 0, None
    Es = []
    for g, (an, ad) in enumerate(a_ratios, start=1):
        A = an * ((1 << S) // ad)
        E = 0
        for x in R:
            q, rem = divmod(abs(x), A)
            if 2 * rem > A or (2 * rem == A and q % 2 == 1):
                q += 1
            q = min(q, M)
            e = abs(x) - A * q
            E += e * e
        Es.append(Fraction(E, 1 << (2 * S)))
        if bestE is None or E < bestE:
            best, bestE = g, E
    return best, Es


def check_paper_search_exact_rational(orc):
    """Eq. (11) on inputs off any lattice: the oracle's candidate-set argmin
    against the exact enumeration of the whole grid (rational errors), for
    both branches of the step, gamma = Delta / M (a step set by the data) and
    gamma = eta, with d up to 16.  The oracle evaluates in fp64, so its
    choice may differ from the exact argmin only between errors within
    rounding (1e-12 relative) of each other."""
    rng = np.random.default_rng(54)
    cases = [0, 0]   # grids with gamma = Delta / M, with gamma = eta
    for bits in (2, 3, 4):
        M = 2 ** (bits - 1) - 1
        for case in range(6):
            d = int(rng.integers(2, 17))
            fine = case % 2 == 0
            # random magnitudes, off any lattice: close ones give the step
            # Delta / M (a fine grid), far apart ones leave eta the smaller
            gaps = rng.uniform(0.04, 0.3, d) if fine else rng.uniform(0.3, 0.6, d)
            r = np.cumsum(gaps) * np.where(rng.random(d) < 0.5, -1.0, 1.0)
            rng.shuffle(r)
            eta = 1.0 if fine else 2.0 ** -6
            gamma, count = orc.paper_grid(r, bits, eta)
            m = np.abs(r)
            diffs = np.abs(m[:, None] - m[None, :])
            delta = diffs[diffs > 0].min() / 2
            assert gamma == min(delta / M, eta), (gamma, delta, M, eta)
            assert fine == (gamma < eta)
            if count > 40000:
                continue
            cases[0 if fine else 1] += 1
            gref, Es = _exact_search(r, M, gamma, count)
            g, Eg = orc.paper_grid_search(r, bits, gamma, count)
            assert 1 <= g <= count
            Eo, Er = float(Es[g - 1]), float(Es[gref - 1])
            assert g == gref or Eo <= Er * (1 + 1e-12), (bits, case, d, g, gref, Eo, Er)
            assert abs(Eg - Eo) <= 1e-12 * Eo + 1e-300
    assert min(cases) >= 6, cases


def _fl32_exact(F):
    """The fp32 value nearest the rational F (ties to the even significand)."""
    from fractions import Fraction
    x = np.float32(float(F))
    cands = {x}
    for _ in range(2):
        cands |= {np.nextafter(c, np.float32(np.inf)) for c in list(cands)}
        cands |= {np.nextafter(c, np.float32(-np.inf)) for c in list(cands)}
    best = None
    for c in cands:
        dist = abs(Fraction(float(c)) - F)
        key = (dist, int(np.array(c, np.float32).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def check_candidate_scales_exact(orc):
    """Reading G2 at every candidate, not only c = 1: a_g is the fp32 value
    nearest the exact rational fl32(max|r|) c_g / M, and the default
    multipliers c_g are the fp32 values nearest g / G; for residuals of
    many magnitudes, bits 2-8, the default grid and a random one."""
    from fractions import Fraction
    rng = np.random.default_rng(56)
    for G in (7, 128, 512, 1000):
        c = orc.default_grid(G)
        for g in range(G):
            assert c[g] == _fl32_exact(Fraction(g + 1, G)), (G, g)
    for bits in (2, 3, 4, 5, 8):
        M = 2 ** (bits - 1) - 1
        for scale in (1e-30, 3e-7, 0.37, 1.0, 4099.5, 1e30):
            r = rng.standard_normal(20) * scale
            m = Fraction(float(np.float32(np.abs(r).max())))
            for grid in (orc.default_grid(256),
                         np.sort(rng.uniform(0.01, 1.0, 64)).astype(np.float32)):
                a = orc.candidate_scales(r, bits, grid)
                want = [_fl32_exact(m * Fraction(float(cg)) / M) for cg in grid]
                assert np.array_equal(a, np.array(want, np.float32)), (bits, scale)


def check_paper_fit(orc):
    """A fit on the paper's grid: the error never increases, each point's
    scale is fl32 of a grid point, and the verifier accepts it and flags a
    fit on the G-point grid."""
    rng = np.random.default_rng(53)
    W = (rng.standard_normal((12, 24)) * 0.3).astype(np.float32)
    codes, scales, counts, err = orc.fit_paper(W, 3, 4, 0.0)
    for k in range(12):
        assert (np.diff(err[k, :counts[k]]) <= 0).all()
    v = orc.verify_paper(W, 3, 4, 0.0, codes, scales, counts, err.astype(np.float32))
    assert (v["status"] == 0).all()
    c0, s0, n0, _ = orc.fit(W, 3, 4, 64, 0.0)
    assert (orc.verify_paper(W, 3, 4, 0.0, c0, s0, n0)["status"] != 0).mean() > 0.5


# ------------------------------------------- reading B2: asymmetric codes
def _dyadic(seed, C=20, d=30):
    rng = np.random.default_rng(seed)
    return (rng.integers(-96, 97, (C, d)) / 64.0 + rng.integers(-8, 9, (C, 1)) / 4.0).astype(np.float32)


def check_asym_translation(orc):
    """Shifting a channel by a constant (exactly representable) leaves the
    points unchanged and moves the offset by that constant."""
    W = _dyadic(71)
    a = orc.fit_asym(W, 4, 4, 64, 0.0)
    b = orc.fit_asym(W + np.float32(3.25), 4, 4, 64, 0.0)
    assert all(np.array_equal(x, y) for x, y in zip(a[:3], b[:3]))
    assert np.array_equal(b[5], a[5] + np.float32(3.25))


def check_asym_is_the_centred_fit(orc):
    """The points of the asymmetric fit are the symmetric fit of w - beta
    (exact in fp32 on this lattice); beta is the midpoint of the range."""
    W = _dyadic(72)
    codes, scales, counts, err, _, off = orc.fit_asym(W, 3, 5, 32, 0.0)
    assert np.array_equal(off, ((W.max(1).astype(np.float64) + W.min(1)) / 2).astype(np.float32))
    c0, s0, n0, e0 = orc.fit(W - off[:, None], 3, 5, 32, 0.0)
    assert np.array_equal(codes, c0) and np.array_equal(scales, s0) and np.array_equal(counts, n0)


def check_asym_edges(orc):
    """Two distinct values per channel are reproduced exactly by one point;
    a constant channel needs no point (beta alone); 10 + small noise stops
    after one point, as the stopping rule compares with ||w||^2."""
    rng = np.random.default_rng(73)
    lo, hi = rng.integers(-128, 0, 10) / 64.0, rng.integers(32, 192, 10) / 64.0   # exact midpoints
    W = np.where(rng.random((10, 16)) < 0.5, lo[:, None], hi[:, None]).astype(np.float32)
    W[:, 0], W[:, 1] = lo, hi
    # 2 bits (M = 1): the top candidate is the half range itself, codes +-1
    codes, scales, counts, err, _, off = orc.fit_asym(W, 2, 3, 64, 0.0)
    assert (counts == 1).all() and np.array_equal(orc.reconstruct(codes, scales, counts, off), W)
    C = np.full((3, 8), 5.0, np.float32)
    codes, scales, counts, err, _, off = orc.fit_asym(C, 4, 3, 64, 1e-3)
    assert (counts == 0).all() and (off == 5.0).all()
    N = (10.0 + 0.01 * rng.standard_normal((8, 40))).astype(np.float32)
    codes, scales, counts, err, _, off = orc.fit_asym(N, 4, 4, 64, 1e-3)
    assert (counts == 1).all()


def check_asym_error_and_reconstruct(orc):
    """Output error and reconstruction with offsets against numpy fp64
    (w~ = beta + sum a q, the offset first)."""
    rng = np.random.default_rng(74)
    W = (rng.standard_normal((15, 50)) + 1.5).astype(np.float32)
    X = rng.standard_normal((50, 20)).astype(np.float32)
    codes, scales, counts, err, _, off = orc.fit_asym(W, 4, 3, 64, 1e-3)
    what = np.zeros((15, 50))
    for k in range(15):
        s = np.full(50, float(off[k]))
        for i in range(counts[k]):
            s = s + float(scales[k, i]) * codes[k, i].astype(np.float64)
        what[k] = s
    assert np.array_equal(orc.reconstruct(codes, scales, counts, off), what.astype(np.float32))
    e, _ = orc.output_error(W, codes, scales, counts, X, offsets=off)
    ref = np.mean(((W.astype(np.float64) - what) @ X.astype(np.float64)) ** 2, axis=1)
    assert np.allclose(e, ref, rtol=1e-12, atol=0)


def check_asym_verifier(orc):
    W = (np.random.default_rng(75).standard_normal((12, 40)) + 0.7).astype(np.float32)
    codes, scales, counts, err, _, off = orc.fit_asym(W, 4, 4, 64, 1e-3)
    v = orc.verify_asym(W, 4, 4, 64, codes, scales, counts, off, err.astype(np.float32), tol=1e-3)
    assert (v["status"] == 0).all()
    off2 = np.nextafter(off, np.float32(np.inf))
    assert (orc.verify_asym(W, 4, 4, 64, codes, scales, counts, off2, tol=1e-3)["status"] == 9).all()


# ------------------------------------------- Sec. 3.4: deployment arithmetic
def check_integer_scales(orc):
    """Eq. (14), reading I1: exact values, half-way ties to even (worked by
    hand), |A - 2^p a| <= 1/2, zero after the count, clamping counted."""
    p = 6
    u = 2.0 ** -p
    a = np.array([[2.5 * u, 3.5 * u, -2.5 * u, 0.5 * u, 1.5 * u, 5 * u, -7 * u]], np.float32)
    A, n = orc.integer_scales(a, np.array([7], np.int32), p)
    assert A[0].tolist() == [2, 4, -2, 0, 2, 5, -7] and n == 0
    rng = np.random.default_rng(2)
    s = rng.standard_normal((40, 5)).astype(np.float32) * 0.1
    counts = rng.integers(0, 6, 40).astype(np.int32)
    for p in (0, 7, 13, 20):
        A, n = orc.integer_scales(s, counts, p)
        assert n == 0
        for k in range(40):
            c = counts[k]
            assert (A[k, c:] == 0).all()
            assert (np.abs(A[k, :c].astype(np.float64) - np.ldexp(s[k, :c].astype(np.float64), p))
                    <= 0.5).all()
    A, n = orc.integer_scales(np.array([[1.0, -1.0, 0.25]], np.float32), np.array([3], np.int32), 31)
    assert A[0].tolist() == [2 ** 31 - 1, -(2 ** 31 - 1), 2 ** 29] and n == 2


def _int_case(seed, C=6, P=3, d=13, N=7):
    rng = np.random.default_rng(seed)
    codes = rng.integers(-7, 8, (C, P, d)).astype(np.int8)     # nonzero past the counts too
    A = rng.integers(-(2 ** 20), 2 ** 20, (C, P)).astype(np.int32)
    counts = rng.integers(0, P + 1, C).astype(np.int32)
    counts[0], counts[1] = 0, P
    X = rng.integers(-128, 128, (N, d)).astype(np.int8)
    return codes, A, counts, X


def check_integer_forward_exact(orc):
    """Eq. (15), Steps 1-3 against exact Python integers: floor of
    sum_{i<n} A_i (q_i . x) over 2^p; rows and A past the count ignored;
    negative sums floor (reading B1)."""
    for seed, p in ((1, 0), (2, 5), (3, 17), (4, 40)):
        codes, A, counts, X = _int_case(seed)
        Y = orc.integer_forward(codes, A, counts, X, p)
        C, P, d = codes.shape
        neg = 0
        for k in range(C):
            for t in range(X.shape[0]):
                s = 0
                for i in range(int(counts[k])):
                    z = sum(int(codes[k, i, j]) * int(X[t, j]) for j in range(d))
                    s += int(A[k, i]) * z
                neg += s < 0 and s % (1 << p) != 0
                assert int(Y[k, t]) == s // (1 << p), (seed, k, t)
        assert p == 0 or neg > 0


def check_integer_forward_one_point(orc):
    """One point with A = 2^p (a = 1): Step 3 undoes the scale, Y = Q X^T."""
    codes, _, _, X = _int_case(5, C=9, P=2, d=40, N=11)
    counts = np.ones(9, np.int32)
    p = 12
    A = np.full((9, 2), 1 << p, np.int32)
    Y = orc.integer_forward(codes, A, counts, X, p)
    assert np.array_equal(Y, codes[:, 0, :].astype(np.int64) @ X.T.astype(np.int64))


def check_integer_forward_approximates(orc):
    """Eq. (14)-(15) approximate the real multipoint product: with A from the
    fitted scales, |y - sum_i a_i z_i| <= 2^(-p-1) sum_i |z_i| + 1."""
    rng = np.random.default_rng(7)
    W = rng.standard_normal((20, 64)).astype(np.float32)
    codes, scales, counts, _ = orc.fit(W, 4, 4, 64, 0.0)
    X = rng.integers(-128, 128, (15, 64)).astype(np.int8)
    for p in (8, 16, 24):
        A, n = orc.integer_scales(scales * 64, counts, p)
        assert n == 0
        Y = orc.integer_forward(codes, A, counts, X, p)
        Z = np.einsum("kij,tj->kit", codes.astype(np.float64), X.astype(np.float64))
        mask = (np.arange(4)[None, :] < counts[:, None]).astype(np.float64)
        exact = np.einsum("ki,kit->kt", (scales * 64).astype(np.float64) * mask, Z)
        bound = np.einsum("ki,kit->kt", mask, np.abs(Z)) * 2.0 ** (-p - 1) + 1.0
        assert (np.abs(Y - exact) <= bound).all(), p


ALL_CHECKS = [
    check_levels, check_rounding_ties, check_codes_bruteforce, check_grid_search_bruteforce,
    check_grid_search_bounds, check_two_point_joint, check_naive_quantizer,
    check_equal_magnitudes, check_worked_examples, check_monotone_decrease,
    check_reconstruct, check_invariances, check_output_error, check_stop_rule,
    check_exponential_decay, check_verifier, check_calib_hadamard_is_isotropic,
    check_calib_stop_definition, check_calib_runs_to_cap, check_calib_zero_batch, check_calib_scaling,
    check_calib_verifier, check_calib_verifier_fp32_evaluation, check_gate_worked_example,
    check_gate_definition, check_gate_hadamard_is_isotropic, check_gate_verifier,
    check_refit_one_point,
    check_refit_residual_chain, check_refit_verifier, check_clip_bruteforce, check_clip_hadamard_is_eq9,
    check_clip_then_algorithm1, check_clip_zero_batch, check_clip_verifier, check_min_gap,
    check_paper_grid_size, check_paper_search_bruteforce, check_paper_search_exact_rational,
    check_candidate_scales_exact, check_paper_fit, check_asym_translation,
    check_asym_is_the_centred_fit, check_asym_edges, check_asym_error_and_reconstruct,
    check_asym_verifier, check_integer_scales,
    check_integer_forward_exact, check_integer_forward_one_point, check_integer_forward_approximates,
]
