"""Parity of the fit's variants with the oracle, through the C ABI:
the least-squares refit of each point's scale (reading A2), alone and with
Algorithm 2's stopping rule.  Judged by the oracle's lockstep verifier in its
refit mode (codes of the best or a tied candidate, the least-squares scale of
those codes within one fp32 ulp, the other rules as for the plain fit)."""
import numpy as np
import pytest

from gpu_util import say, to_dev
from paper_2002_09049_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2002_09049_amd import mpq
    mpq.load()
    yield


def _fit_ex(W, bits, P, G, tol=0.0, refit=True, X=None, eps=0.0, relative=True):
    import torch
    from paper_2002_09049_amd import mpq
    ls = mpq.LayerSet([to_dev(W)], P, calib=None if X is None else [to_dev(X)])
    ls.fit_ex(bits, G, tol, refit=refit, calib=X is not None, eps=eps, relative=relative)
    torch.cuda.synchronize()
    out = (ls.codes[0].cpu().numpy(), ls.scales[0].cpu().numpy(), ls.counts[0].cpu().numpy(),
           ls.fit_err[0].cpu().numpy())
    return out if X is None else out + (ls.xerr[0].cpu().numpy(),)


def _ok(v):
    bad = np.nonzero(v["status"])[0]
    assert bad.size == 0, (f"{bad.size} channels fail: channels {v['channels'][bad][:8]} "
                           f"status {v['status'][bad][:8]}")


REFIT = [
    # (C, d, bits, P, G, tol): the variants and modes of the search kernel
    (3, 1, 4, 4, 128, 1e-3),
    (40, 9, 4, 8, 512, 1e-3),
    (33, 17, 3, 8, 7, 1e-4),
    (50, 16, 3, 6, 7, 0.0),
    (30, 4, 8, 4, 1000, 1e-4),
    (64, 147, 4, 4, 256, 1e-3),
    (64, 576, 4, 4, 128, 1e-3),
    (20, 1000, 2, 6, 1000, 0.0),
    (10, 2304, 4, 8, 256, 1e-5),
    (7, 4608, 3, 8, 512, 5e-4),
    (6, 9000, 4, 4, 64, 0.0),
    (4, 20000, 3, 4, 256, 1e-4),
]


@pytest.mark.parametrize("C,d,bits,P,G,tol", REFIT, ids=[f"C{c}_d{d}_b{b}_P{p}_G{g}" for c, d, b, p, g, _ in REFIT])
def test_refit_parity(orc, C, d, bits, P, G, tol):
    say(f"case refit C={C} d={d} bits={bits} P={P} G={G} tol={tol}")
    W = wl.random_weights(C, d, seed=C * 7 + d)
    codes, scales, counts, err = _fit_ex(W, bits, P, G, tol)
    _ok(orc.verify(W, bits, P, G, float(np.float32(tol)), codes, scales, counts, err, refit=True))


def test_refit_improves_every_first_point():
    """The refit keeps the first point's codes and never raises its error."""
    W = wl.random_weights(200, 300, seed=4)
    c0, s0, n0, e0 = _fit_ex(W, 4, 1, 128, refit=False)
    c1, s1, n1, e1 = _fit_ex(W, 4, 1, 128, refit=True)
    assert np.array_equal(c0, c1)
    assert (e1[:, 0] <= e0[:, 0] * (1 + 1e-6)).all() and (e1[:, 0] < e0[:, 0]).mean() > 0.9


def test_refit_with_calibration_rule(orc):
    C, d, N = 50, 576, 256
    W = wl.random_weights(C, d, seed=9)
    X = wl.random_calib(d, N, seed=10)
    say("case refit + Algorithm 2 rule")
    codes, scales, counts, err, xerr = _fit_ex(W, 4, 6, 128, X=X, eps=2e-3)
    _ok(orc.verify_calib(W, 4, 6, 128, X, float(np.float32(2e-3)), True, codes, scales, counts, err,
                         xerr, refit=True))


def test_refit_rejects_dense_only_lengths():
    from paper_2002_09049_amd import mpq
    W = wl.random_weights(2, 40000, seed=1)
    with pytest.raises(mpq.MPQError) as e:
        _fit_ex(W, 4, 2, 16)
    assert e.value.status == mpq.MPQ_ERR_SHAPE


def test_refit_workload_resnet18_sampled(orc):
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get("resnet18")
    Ws = [to_dev(wl.layer_weights(w, i)) for i in range(len(w.layers))]
    say("case refit resnet18 full size")
    ls = mpq.LayerSet(Ws, w.max_points)
    ls.fit_ex(w.bits, w.n_grid, w.tol, refit=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(2)
    for li, (C, d) in enumerate(w.layers):
        ch = np.unique(np.concatenate([[0, C - 1], rng.choice(C, size=min(8, C), replace=False)]))
        out = (ls.codes[li].cpu().numpy(), ls.scales[li].cpu().numpy(), ls.counts[li].cpu().numpy(),
               ls.fit_err[li].cpu().numpy())
        _ok(orc.verify(Ws[li].cpu().numpy(), w.bits, w.max_points, w.n_grid,
                       float(np.float32(w.tol)), *out, channels=ch, refit=True))


def _fit_clip(W, X, bits, P, G, tol=0.0, calib=False, eps=0.0, clip_grid=20):
    import torch
    from paper_2002_09049_amd import mpq
    ls = mpq.LayerSet([to_dev(W)], P, calib=[to_dev(X)])
    ls.fit_ex(bits, G, tol, calib=calib, eps=eps, relative=True, clip_grid=clip_grid)
    torch.cuda.synchronize()
    return (ls.codes[0].cpu().numpy(), ls.scales[0].cpu().numpy(), ls.counts[0].cpu().numpy(),
            ls.fit_err[0].cpu().numpy(), ls.xerr[0].cpu().numpy())


CLIP = [
    # (C, d, bits, P, G, N, tol)
    (3, 1, 4, 4, 128, 5, 1e-3),
    (40, 9, 4, 8, 512, 64, 1e-3),
    (41, 16, 3, 6, 64, 20, 1e-4),
    (70, 147, 4, 4, 256, 300, 1e-3),
    (64, 576, 3, 6, 128, 256, 1e-4),
    (20, 2304, 4, 4, 256, 1024, 1e-3),
    (6, 9000, 4, 3, 64, 130, 0.0),
]


@pytest.mark.parametrize("C,d,bits,P,G,N,tol", CLIP, ids=[f"C{c}_d{d}_b{b}_P{p}_G{g}_N{n}" for c, d, b, p, g, n, _ in CLIP])
def test_clip_parity(orc, C, d, bits, P, G, N, tol):
    say(f"case clip C={C} d={d} bits={bits} P={P} G={G} N={N} tol={tol}")
    W = wl.random_weights(C, d, seed=C + 3 * d)
    X = wl.random_calib(d, N, seed=N)
    codes, scales, counts, err, _ = _fit_clip(W, X, bits, P, G, tol)
    _ok(orc.verify_clip(W, bits, P, G, X, codes, scales, counts, err, tol=float(np.float32(tol))))
    assert (counts >= 1).all()


def test_clip_with_calibration_rule(orc):
    C, d, N = 48, 576, 256
    W = wl.random_weights(C, d, seed=17)
    X = wl.random_calib(d, N, seed=18)
    say("case clip + Algorithm 2 rule")
    codes, scales, counts, err, xerr = _fit_clip(W, X, 4, 6, 128, calib=True, eps=2e-3)
    _ok(orc.verify_clip(W, 4, 6, 128, X, codes, scales, counts, err, xerr, calib=True,
                        eps=float(np.float32(2e-3))))


def test_clip_grid_size_and_edges(orc):
    """Another number of clipping factors; an all-zero channel (no point);
    a cap of one point; one calibration column."""
    d, N = 200, 64
    W = wl.random_weights(9, d, seed=5)
    W[4] = 0.0
    X = wl.random_calib(d, N, seed=6)
    for Gc, P, n in ((8, 4, N), (20, 1, N), (20, 3, 1)):
        say(f"case clip edges Gc={Gc} P={P} n={n}")
        Xn = np.ascontiguousarray(X[:, :n])
        codes, scales, counts, err, _ = _fit_clip(W, Xn, 4, P, 64, 1e-3, clip_grid=Gc)
        _ok(orc.verify_clip(W, 4, P, 64, Xn, codes, scales, counts, err,
                            tol=float(np.float32(1e-3)), clip_grid=Gc))
        assert counts[4] == 0 and (np.delete(counts, 4) >= 1).all()


def test_clip_rejects_refit():
    import torch
    from paper_2002_09049_amd import mpq
    W = wl.random_weights(4, 64, seed=1)
    X = wl.random_calib(64, 16, seed=2)
    ls = mpq.LayerSet([to_dev(W)], 4, calib=[to_dev(X)])
    with pytest.raises(mpq.MPQError) as e:
        ls.fit_ex(4, 64, 1e-3, refit=True, clip_grid=20)
    assert e.value.status == mpq.MPQ_ERR_INVALID_ARG
    torch.cuda.synchronize()


def test_clip_workload_resnet18_sampled(orc):
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get("resnet18")
    Ws = [to_dev(wl.layer_weights(w, i)) for i in range(len(w.layers))]
    Xs = [to_dev(wl.layer_calib(w, i)) for i in range(len(w.layers))]
    say("case clip resnet18 full size")
    ls = mpq.LayerSet(Ws, w.max_points, calib=Xs)
    ls.fit_ex(w.bits, w.n_grid, w.tol, clip_grid=20)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    for li, (C, d) in enumerate(w.layers):
        ch = np.unique(np.concatenate([[0, C - 1], rng.choice(C, size=min(6, C), replace=False)]))
        out = (ls.codes[li].cpu().numpy(), ls.scales[li].cpu().numpy(), ls.counts[li].cpu().numpy(),
               ls.fit_err[li].cpu().numpy())
        say(f"  layer {li} ({C}x{d})")
        _ok(orc.verify_clip(Ws[li].cpu().numpy(), w.bits, w.max_points, w.n_grid, Xs[li].cpu().numpy(),
                            *out, tol=float(np.float32(w.tol)), channels=ch))


def _fit_paper(W, bits, P, tol, eta):
    import torch
    from paper_2002_09049_amd import mpq
    ls = mpq.LayerSet([to_dev(W)], P)
    ls.fit_ex(bits, 1, tol, paper_eta=eta)
    torch.cuda.synchronize()
    return (ls.codes[0].cpu().numpy(), ls.scales[0].cpu().numpy(), ls.counts[0].cpu().numpy(),
            ls.fit_err[0].cpu().numpy())


PAPER = [
    # (C, d, bits, P, tol, eta): every kernel variant; Gaussian weights make
    # Delta_r tiny, so the grids hold 10^8 points and more
    (3, 1, 4, 4, 1e-3, 2.0 ** -10),
    (20, 9, 4, 6, 0.0, 2.0 ** -10),
    (30, 147, 4, 4, 1e-3, 2.0 ** -10),
    (10, 576, 3, 4, 1e-4, 2.0 ** -10),
    (6, 1000, 2, 5, 0.0, 2.0 ** -6),
    (3, 2304, 4, 3, 0.0, 2.0 ** -10),
    (2, 4608, 4, 2, 1e-3, 2.0 ** -10),
    (2, 8192, 2, 2, 0.0, 2.0 ** -10),
    # past 8192: the variant with its sorted magnitudes in global scratch
    # (the oracle's exact search costs O(d^2 M) per step: few channels)
    (2, 9000, 4, 2, 0.0, 2.0 ** -10),
]


@pytest.mark.parametrize("C,d,bits,P,tol,eta", PAPER, ids=[f"C{c}_d{d}_b{b}_P{p}" for c, d, b, p, _, _ in PAPER])
def test_paper_grid_parity(orc, C, d, bits, P, tol, eta):
    say(f"case paper grid C={C} d={d} bits={bits} P={P} tol={tol} eta={eta}")
    W = wl.random_weights(C, d, seed=11 * C + d)
    codes, scales, counts, err = _fit_paper(W, bits, P, tol, eta)
    _ok(orc.verify_paper(W, bits, P, float(np.float32(tol)), codes, scales, counts, err, eta=eta))


def test_paper_grid_exact_on_dyadic_weights(orc):
    """Weights on a 1/64 lattice and eta = 2^-10: the first step's gamma is
    2^-10 and every error of it is exact (ties included), so the GPU's first
    point equals the oracle's bit for bit; later steps (gamma = Delta / M,
    no longer dyadic) are checked in lockstep."""
    rng = np.random.default_rng(61)
    W = (rng.integers(-96, 97, (40, 24)) / 64.0).astype(np.float32)
    W[5] = 0.0
    for bits in (2, 3, 4):
        say(f"case paper grid dyadic bits={bits}")
        codes, scales, counts, err = _fit_paper(W, bits, 1, 0.0, 2.0 ** -10)
        oc, os_, on, _ = orc.fit_paper(W, bits, 1, 0.0)
        assert np.array_equal(counts, on) and np.array_equal(scales, os_) and np.array_equal(codes, oc)
        out = _fit_paper(W, bits, 4, 0.0, 2.0 ** -10)
        _ok(orc.verify_paper(W, bits, 4, 0.0, *out))


@pytest.mark.timeout(600)
def test_paper_grid_vgg16fc_length(orc):
    """VGG-16 fc's 25088-long channels (3 bits) on the paper's grid, with a
    layer of short channels in the same call (both kernels side by side):
    lockstep parity of the first point (the oracle's exact search takes about
    a minute per such channel and step)."""
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get("vgg16fc")
    W = np.ascontiguousarray(wl.layer_weights(w, 0)[:2])
    W2 = wl.random_weights(4, 300, seed=8)
    say("case paper grid d=25088 (2 channels) + d=300")
    ls = mpq.LayerSet([to_dev(W), to_dev(W2)], 1)
    ls.fit_ex(w.bits, 1, w.tol, paper_eta=2.0 ** -10)
    torch.cuda.synchronize()
    for i, Wi in enumerate((W, W2)):
        out = (ls.codes[i].cpu().numpy(), ls.scales[i].cpu().numpy(), ls.counts[i].cpu().numpy(),
               ls.fit_err[i].cpu().numpy())
        _ok(orc.verify_paper(Wi, w.bits, 1, float(np.float32(w.tol)), *out))
        assert (out[2] == 1).all()


def test_paper_grid_limits():
    from paper_2002_09049_amd import mpq
    W = wl.random_weights(1, 32769, seed=1)
    with pytest.raises(mpq.MPQError) as e:
        _fit_paper(W, 4, 2, 0.0, 2.0 ** -10)
    assert e.value.status == mpq.MPQ_ERR_SHAPE
    ls = mpq.LayerSet([to_dev(wl.random_weights(2, 64, seed=2))], 2)
    with pytest.raises(mpq.MPQError) as e:
        ls.fit_ex(4, 1, 0.0, refit=True, paper_eta=2.0 ** -10)
    assert e.value.status == mpq.MPQ_ERR_INVALID_ARG


def _fit_asym(W, bits, P, G, tol=0.0, X=None, calib=False, eps=0.0, refit=False):
    import torch
    from paper_2002_09049_amd import mpq
    ls = mpq.LayerSet([to_dev(W)], P, calib=None if X is None else [to_dev(X)])
    ls.fit_ex(bits, G, tol, refit=refit, calib=calib, eps=eps, relative=True, asym=True)
    if X is not None:
        ls.output_error()
    ls.reconstruct()
    torch.cuda.synchronize()
    out = (ls.codes[0].cpu().numpy(), ls.scales[0].cpu().numpy(), ls.counts[0].cpu().numpy(),
           ls.fit_err[0].cpu().numpy(), None if X is None else ls.xerr[0].cpu().numpy(),
           ls.offsets[0].cpu().numpy())
    extra = (None if X is None else ls.err[0].cpu().numpy(), ls.W_hat[0].cpu().numpy())
    return out, extra


ASYM = [
    # (C, d, bits, P, G, tol, shift): channels with a common offset exercise B2
    (5, 1, 4, 4, 128, 1e-3, 0.0),
    (40, 9, 4, 8, 512, 1e-3, 0.3),
    (43, 16, 3, 6, 128, 1e-4, -0.7),
    (64, 147, 4, 4, 256, 1e-3, 1.0),
    (64, 576, 3, 6, 128, 1e-4, -0.5),
    (10, 2304, 4, 4, 256, 1e-3, 2.0),
    (4, 20000, 3, 4, 256, 1e-4, 0.1),
]


@pytest.mark.parametrize("C,d,bits,P,G,tol,shift", ASYM, ids=[f"C{c}_d{d}_b{b}_P{p}_G{g}" for c, d, b, p, g, _, _ in ASYM])
def test_asym_parity(orc, C, d, bits, P, G, tol, shift):
    say(f"case asym C={C} d={d} bits={bits} P={P} G={G} tol={tol}")
    W = wl.random_weights(C, d, seed=5 * C + d) + np.float32(shift)
    W[0] = np.float32(shift)          # a constant channel: no point
    (codes, scales, counts, err, _, off), (_, what) = _fit_asym(W, bits, P, G, tol)
    _ok(orc.verify_asym(W, bits, P, G, codes, scales, counts, off, err, tol=float(np.float32(tol))))
    assert counts[0] == 0
    assert np.array_equal(what, orc.reconstruct(codes, scales, counts, off))


def test_asym_with_calibration_rule_and_output_error(orc):
    C, d, N = 48, 576, 256
    W = wl.random_weights(C, d, seed=19) + np.float32(0.8)
    X = wl.random_calib(d, N, seed=20)
    say("case asym + Algorithm 2 rule")
    (codes, scales, counts, err, xerr, off), (oe, what) = _fit_asym(W, 4, 6, 128, X=X, calib=True, eps=2e-3)
    _ok(orc.verify_asym(W, 4, 6, 128, codes, scales, counts, off, err, xerr, X=X, calib=True,
                        eps=float(np.float32(2e-3))))
    ref, _ = orc.output_error(W, codes, scales, counts, X, with_ref=False, offsets=off)
    assert np.all(np.abs(oe - ref) <= 1e-5 * ref + 1e-30)


def test_asym_with_refit(orc):
    W = wl.random_weights(30, 300, seed=21) + np.float32(-0.4)
    (codes, scales, counts, err, _, off), _ = _fit_asym(W, 4, 4, 64, 1e-3, refit=True)
    _ok(orc.verify_asym(W, 4, 4, 64, codes, scales, counts, off, err, tol=float(np.float32(1e-3)),
                        refit=True))


def test_symmetric_fit_after_asym_takes_no_offsets(orc):
    """A LayerSet's symmetric fit after an asymmetric one reconstructs
    without offsets."""
    import torch
    from paper_2002_09049_amd import mpq
    W = wl.random_weights(16, 64, seed=3) + np.float32(1.0)
    ls = mpq.LayerSet([to_dev(W)], 4)
    ls.fit_ex(4, 64, 1e-3, asym=True)
    ls.fit(4, 64, 1e-3)
    ls.reconstruct()
    torch.cuda.synchronize()
    out = (ls.codes[0].cpu().numpy(), ls.scales[0].cpu().numpy(), ls.counts[0].cpu().numpy())
    assert np.array_equal(ls.W_hat[0].cpu().numpy(), orc.reconstruct(*out))
