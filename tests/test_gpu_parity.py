"""Parity of the HIP path (through the C ABI) with the oracle.

Fit outputs are judged by the oracle's lockstep verifier: integer codes and
point counts bit-exact except at ties (top-2 candidate errors within 1e-6
relative, element half-ties within 1e-6, stop decisions within 1e-6 of the
threshold), scales bit-equal to the chosen candidate, per-point ||r||^2
within 1e-5 relative.  Output errors within 1e-5 relative of the fp64
oracle; reconstruction bit-exact.
"""
import json
import os

import numpy as np
import pytest

import bruteforce as bf
from gpu_util import assert_parity, free_running_diff, gpu_fit, say, to_dev
from paper_2002_09049_amd import workloads as wl

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2002_09049_amd import mpq
    mpq.load()   # fails loudly if libmpq.so is missing
    yield


def test_worked_examples_exact():
    cases = {c["name"]: c for c in json.load(open(GOLDEN))["cases"]}
    g = cases["two_elements_exact_tie"]
    say("case golden two_elements_exact_tie")
    codes, scales, counts, err = gpu_fit(np.array([g["w"]], np.float32), g["bits"],
                                         g["max_points"], g["n_grid"], g["tol"])
    e = g["expect"]
    assert counts[0] == e["count"] and scales[0].tolist() == e["scales"]
    assert codes[0].tolist() == e["codes"] and err[0].tolist() == e["err"]
    g = cases["stop_exactly_at_tolerance"]
    for v in g["variants"]:
        say("case golden stop_exactly_at_tolerance tol", v["tol"])
        codes, scales, counts, err = gpu_fit(np.array([g["w"]], np.float32), g["bits"],
                                             g["max_points"], g["n_grid"], v["tol"])
        assert counts[0] == v["count"] and scales[0].tolist() == v["scales"]
        assert err[0].tolist() == v["err"]
        assert codes[0, 0].tolist() == v["codes_point0"]


SWEEP = [
    # (C, d, bits, P, G, tol)
    (3, 1, 4, 4, 128, 1e-3),
    (40, 9, 4, 8, 512, 1e-3),
    (33, 17, 3, 8, 7, 1e-4),
    (64, 147, 4, 4, 256, 1e-3),
    (64, 576, 4, 4, 128, 1e-3),
    (20, 1000, 2, 6, 1000, 0.0),
    (16, 333, 8, 3, 64, 0.0),
    (24, 64, 3, 8, 512, 5e-4),
    (10, 2304, 4, 8, 2, 1e-5),
    (7, 4608, 3, 8, 512, 5e-4),
    (5, 250, 4, 64, 16, 0.0),
    (9, 100, 4, 4, 1, 0.0),
]


@pytest.mark.parametrize("dense", [False, True], ids=["hist", "dense"])
@pytest.mark.parametrize("C,d,bits,P,G,tol", SWEEP, ids=[f"C{c}_d{d}_b{b}_P{p}_G{g}" for c, d, b, p, g, _ in SWEEP])
def test_parity_sweep(orc, C, d, bits, P, G, tol, dense):
    say(f"case sweep C={C} d={d} bits={bits} P={P} G={G} tol={tol} dense={dense}")
    W = wl.random_weights(C, d, seed=C * 1000 + d)
    out = gpu_fit(W, bits, P, G, tol, dense=dense)
    v = assert_parity(orc, W, bits, P, G, tol, out)
    ties = int(v["cand_ties"].sum() + v["code_ties"].sum() + v["stop_ties"].sum())
    nd = free_running_diff(orc, W, bits, P, G, tol, out)
    say(f"  ties={ties} free-running channel diffs={nd}")
    tie_channels = int(((v["cand_ties"] + v["code_ties"] + v["stop_ties"]) > 0).sum())
    assert nd <= tie_channels


def test_edge_channels(orc):
    say("case edge channels")
    d = 50
    rng = np.random.default_rng(5)
    W = np.zeros((8, d), np.float32)
    W[1] = 0.3 * np.sign(rng.standard_normal(d))            # all |w| equal
    W[2, 7] = -2.5                                            # one nonzero
    W[3] = rng.standard_normal(d) * 1e30                      # huge
    W[4] = rng.standard_normal(d) * 1e-30                     # tiny (normal range)
    W[5, :3] = [1e-45, 0.0, -1e-45]                           # subnormal: no candidate
    W[6] = rng.standard_normal(d)
    W[6, ::2] = W[6, 1::2]                                    # repeated values
    W[7] = np.arange(d, dtype=np.float32) / 7.0
    for (bits, G, P, tol), dense in [(c, dn) for c in ((4, 128, 4, 1e-3), (2, 64, 6, 0.0), (8, 32, 2, 0.0))
                                     for dn in (False, True)]:
        say(f"  bits={bits} G={G} P={P} tol={tol} dense={dense}")
        out = gpu_fit(W, bits, P, G, tol, dense=dense)
        assert_parity(orc, W, bits, P, G, tol, out)
        codes, scales, counts, err = out
        assert counts[0] == 0 and (codes[0] == 0).all() and (scales[0] == 0).all()
        if tol > 0:
            assert counts[1] == 1          # equal magnitudes: one point (closed form)
        assert counts[5] == (1 if bits == 2 else 0)   # subnormal channel


@pytest.mark.parametrize("dense", [False, True], ids=["hist", "dense"])
def test_explicit_grid_and_no_err(orc, dense):
    say(f"case explicit grid, err=NULL, dense={dense}")
    W = wl.random_weights(32, 300, seed=77)
    grid = np.sort(np.random.default_rng(3).uniform(0.05, 1.0, 37)).astype(np.float32)
    grid[-1] = 1.0
    out = gpu_fit(W, 4, 5, 37, 1e-4, grid=grid, dense=dense)
    assert_parity(orc, W, 4, 5, 37, 1e-4, out, grid=grid)
    out2 = gpu_fit(W, 4, 5, 37, 1e-4, grid=grid, with_err=False, dense=dense)
    for a, b in zip(out[:3], out2[:3]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("dense", [False, True], ids=["hist", "dense"])
def test_deterministic(dense):
    say(f"case determinism dense={dense}")
    W = wl.random_weights(48, 777, seed=9)
    a = gpu_fit(W, 4, 6, 256, 1e-4, dense=dense)
    b = gpu_fit(W, 4, 6, 256, 1e-4, dense=dense)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("d", [2048, 2049, 2304, 2305, 8192, 8193, 16384, 16385, 32768, 32769])
def test_search_kernel_boundaries(orc, d):
    """Largest channels of each register-resident variant of the histogram
    search, and the first length that falls back to the dense search."""
    say(f"case boundary d={d}")
    W = wl.random_weights(3, d, seed=d)
    out = gpu_fit(W, 3, 4, 512, 5e-4)
    assert_parity(orc, W, 3, 4, 512, 5e-4, out)


def _lattice_rows(d, rng):
    """Channels for the lattice mode of the histogram search (default grid):
    random; elements exactly on level boundaries of 4-bit, G = 256 (max 1,
    a_g = j / 256 for g + 1 = 7 j, boundaries (2k+1) j / 512, all exact in
    fp32); a scale below 2^-100 (per-level fallback); a few outliers over many
    tiny values; equal magnitudes."""
    W = np.zeros((5, d), np.float32)
    W[0] = rng.standard_normal(d)
    k = rng.integers(0, 7, d)
    j = rng.integers(1, 37, d)
    W[1] = (2 * k + 1) * j / 512.0 * np.sign(rng.standard_normal(d))
    W[1, 0] = 1.0
    W[2] = rng.standard_normal(d) * 1e-33
    W[3] = rng.standard_normal(d) * 1e-3
    W[3, rng.integers(0, d, 4)] = [50.0, -80.0, 20.0, 1.0]
    W[4] = 0.7 * np.sign(rng.standard_normal(d))
    return W


@pytest.mark.parametrize("d", [1025, 2049, 4097, 4608, 4609, 16385, 25088, 32768])
def test_lattice_mode_channels(orc, d):
    """Lattice-bucket mode of the histogram search (default grid, channels
    longer than 1024; past 16384 the variant that rebuilds the residual from
    the weights and codes each phase): lockstep parity, including elements that sit exactly on
    a boundary (exact per-boundary corrections) and a channel below the
    mode's range; and agreement with the per-level histogram, reached by
    passing the default grid explicitly."""
    rng = np.random.default_rng(d)
    W = _lattice_rows(d, rng)
    for bits, G, P, tol in ((4, 256, 4, 1e-3), (4, 256, 8, 0.0), (3, 512, 5, 1e-4),
                            (2, 1000, 6, 0.0), (5, 128, 3, 1e-3)):
        say(f"case lattice d={d} bits={bits} G={G} P={P} tol={tol}")
        out = gpu_fit(W, bits, P, G, tol)
        v = assert_parity(orc, W, bits, P, G, tol, out)
        grid = (np.arange(1, G + 1, dtype=np.float64) / G).astype(np.float32)
        ref = gpu_fit(W, bits, P, G, tol, grid=grid)
        assert_parity(orc, W, bits, P, G, tol, ref, grid=grid)
        diff = ((out[2] != ref[2]) | (out[1] != ref[1]).any(axis=1)
                | (out[0] != ref[0]).any(axis=(1, 2)))
        tie = (v["cand_ties"] + v["code_ties"] + v["stop_ties"]) > 0
        assert not (diff & ~tie).any(), f"channels {np.nonzero(diff & ~tie)[0]} differ without a tie"


@pytest.mark.parametrize("d", [40, 64, 130, 256, 400, 512])
def test_per_level_mode_boundaries(orc, d):
    """The per-level histogram of the default grid (channels of up to 512,
    below the lattice mode), whose level counts come from an fp32 estimate
    and take one exact comparison only when the estimate lies near an
    integer: the rows of the lattice test put many elements exactly on a
    boundary (estimate an integer), plus random, tiny-scale, outlier and
    equal-magnitude rows; lockstep parity, and agreement with the binary
    search of the explicit grid."""
    rng = np.random.default_rng(1000 + d)
    W = _lattice_rows(d, rng)
    for bits, G, P, tol in ((4, 256, 4, 1e-3), (4, 256, 8, 0.0), (3, 512, 5, 1e-4), (5, 128, 3, 1e-3)):
        say(f"case per-level boundaries d={d} bits={bits} G={G} P={P} tol={tol}")
        out = gpu_fit(W, bits, P, G, tol)
        v = assert_parity(orc, W, bits, P, G, tol, out)
        grid = (np.arange(1, G + 1, dtype=np.float64) / G).astype(np.float32)
        ref = gpu_fit(W, bits, P, G, tol, grid=grid)
        diff = ((out[2] != ref[2]) | (out[1] != ref[1]).any(axis=1)
                | (out[0] != ref[0]).any(axis=(1, 2)))
        tie = (v["cand_ties"] + v["code_ties"] + v["stop_ties"]) > 0
        assert not (diff & ~tie).any(), f"channels {np.nonzero(diff & ~tie)[0]} differ without a tie"


def test_exact_ties_between_candidates(orc):
    """Channels built so that several candidate scales give exactly the same
    error (dyadic values): the smallest scale must win, in both searches."""
    say("case exact candidate ties")
    rows = [[1.0, 0.5], [1.0, 0.5, 0.5, 0.5], [0.75, 0.25, -0.5, 1.0], [2.0, 1.0, 1.0, 0.0]]
    d = 4
    W = np.zeros((len(rows), d), np.float32)
    for i, r in enumerate(rows):
        W[i, :len(r)] = r
    for bits, G in ((2, 2), (2, 4), (3, 8), (4, 16)):
        ref = orc.fit(W, bits, 4, G, 0.0)
        for dense in (False, True):
            out = gpu_fit(W, bits, 4, G, 0.0, dense=dense)
            assert_parity(orc, W, bits, 4, G, 0.0, out)
            assert np.array_equal(out[1], ref[1]) and np.array_equal(out[0], ref[0])


def test_shape_limit():
    from paper_2002_09049_amd import mpq
    import torch
    for G in (128, 512):
        dmax = mpq.fit_max_dim(G)
        say(f"case shape limit G={G} dmax={dmax}")
        assert dmax >= 25088
        W = torch.zeros((1, dmax + 1), dtype=torch.float32, device="cuda")
        with pytest.raises(mpq.MPQError) as ei:
            mpq.fit_layer(W, 4, 2, G, 1e-3)
        assert ei.value.status == mpq.MPQ_ERR_SHAPE


def test_largest_dim_fits(orc):
    from paper_2002_09049_amd import mpq
    G = 512
    d = mpq.fit_max_dim(G)
    say(f"case d = max dim {d}")
    W = wl.random_weights(2, d, seed=4)
    out = gpu_fit(W, 3, 3, G, 5e-4)
    assert_parity(orc, W, 3, 3, G, 5e-4, out)


def _oracle_err(orc, W, out, X, channels=None):
    codes, scales, counts, _ = out
    return orc.output_error(W, codes, scales, counts, X, channels=channels)


def _gpu_err(W, out, X, with_ref=True):
    import torch
    from paper_2002_09049_amd import mpq
    codes, scales, counts, _ = out
    e, r = mpq.output_error(to_dev(W), to_dev(codes), to_dev(scales), to_dev(counts), to_dev(X),
                            with_ref=with_ref)
    torch.cuda.synchronize()
    return e.cpu().numpy(), None if r is None else r.cpu().numpy()


@pytest.mark.parametrize("C,d,n", [(1, 1, 1), (130, 147, 300), (64, 576, 256), (257, 64, 129),
                                   (40, 2305, 1024), (33, 1600, 77), (5, 4608, 3), (1000, 512, 130)])
def test_output_error_and_reconstruct(orc, C, d, n):
    say(f"case output error C={C} d={d} n={n}")
    W = wl.random_weights(C, d, seed=C + d)
    X = wl.random_calib(d, n, seed=n)
    out = gpu_fit(W, 4, 4, 128, 1e-3)
    eo, ro = _oracle_err(orc, W, out, X)
    eg, rg = _gpu_err(W, out, X)
    assert np.all(np.abs(eg - eo) <= 1e-5 * eo + 1e-30), np.max(np.abs(eg - eo) / eo)
    assert np.all(np.abs(rg - ro) <= 1e-5 * ro + 1e-30)
    eg2, r2 = _gpu_err(W, out, X, with_ref=False)
    assert r2 is None and np.array_equal(eg, eg2)
    import torch
    from paper_2002_09049_amd import mpq
    codes, scales, counts, _ = out
    Wh = mpq.reconstruct(to_dev(codes), to_dev(scales), to_dev(counts))
    torch.cuda.synchronize()
    assert np.array_equal(Wh.cpu().numpy(), orc.reconstruct(codes, scales, counts))


def test_output_error_wide_range(orc):
    """The GEMM's bf16 pieces keep fp32's exponent range: rows of W scaled by
    2^-30 .. 2^30 and columns of X by 2^-20 .. 2^20 (exact scalings) keep the
    1e-5 relative agreement with the fp64 output error on every row."""
    C, d, n = 96, 300, 200
    say(f"case output error, wide range C={C} d={d} n={n}")
    rs = np.ldexp(1.0, np.round(np.linspace(-30, 30, C)).astype(int)).astype(np.float32)
    cs = np.ldexp(1.0, np.round(np.linspace(-20, 20, n)).astype(int)).astype(np.float32)
    W = (wl.random_weights(C, d, seed=31) * rs[:, None]).astype(np.float32)
    X = (wl.random_calib(d, n, seed=32) * cs[None, :]).astype(np.float32)
    out = gpu_fit(W, 4, 4, 128, 1e-3)
    eo, ro = _oracle_err(orc, W, out, X)
    eg, rg = _gpu_err(W, out, X)
    assert np.all(np.isfinite(eg)) and np.all(eo > 0)
    assert np.all(np.abs(eg - eo) <= 1e-5 * eo), np.max(np.abs(eg - eo) / eo)
    assert np.all(np.abs(rg - ro) <= 1e-5 * ro)


def test_output_error_hadamard(orc):
    say("case output error, X X^T = N I")
    d, N = 100, 128
    W = wl.random_weights(70, d, seed=12)
    out = gpu_fit(W, 3, 3, 64, 1e-2)
    X = bf.hadamard(N)[:d].astype(np.float32)
    eg, rg = _gpu_err(W, out, X)
    codes, scales, counts, err = out
    last = err[np.arange(70), counts - 1].astype(np.float64)
    assert np.allclose(eg, last, rtol=2e-5, atol=0)
    assert np.allclose(rg, (W.astype(np.float64) ** 2).sum(axis=1), rtol=1e-5, atol=0)


def test_workload_conv64x576_full(orc):
    """Single conv layer 64 x 576 (4 bits, 4 points, 128 candidates): every
    channel checked, output error and reconstruction on the full batch."""
    w = wl.get("conv64x576")
    W = wl.layer_weights(w, 0)
    X = wl.layer_calib(w, 0)
    say("case workload conv64x576 full")
    out = gpu_fit(W, w.bits, w.max_points, w.n_grid, w.tol)
    v = assert_parity(orc, W, w.bits, w.max_points, w.n_grid, w.tol, out)
    nd = free_running_diff(orc, W, w.bits, w.max_points, w.n_grid, w.tol, out)
    say(f"  counts={np.bincount(out[2]).tolist()} ties={int(v['cand_ties'].sum())} diffs={nd}")
    eo, ro = _oracle_err(orc, W, out, X)
    eg, rg = _gpu_err(W, out, X)
    assert np.all(np.abs(eg - eo) <= 1e-5 * eo)
    assert np.all(np.abs(rg - ro) <= 1e-5 * ro)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["conv64x576", "resnet18", "resnet50", "mobilenetv2", "vgg16fc"])
def test_workload_quantize_every_channel(orc, name):
    """The call the benchmark times (mpq_quantize_layers: every layer's fit,
    output error on its full calibration batch, reconstruction; batched fit
    launches, fit-written rows of D, grouped error GEMMs), at full size, with
    every channel of every layer checked: the fit in lockstep (V1-V4), the
    output error within 1e-5 relative of the fp64 oracle, the reconstruction
    bit-exact."""
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get(name)
    say(f"case quantize every channel {name}: {len(w.layers)} layers, {w.channels} channels")
    Ws = [to_dev(wl.layer_weights(w, i)) for i in range(len(w.layers))]
    Xs = [to_dev(wl.layer_calib(w, i)) for i in range(len(w.layers))]
    ls = mpq.LayerSet(Ws, w.max_points, calib=Xs, with_fit_err=True)
    ls.quantize(w.bits, w.n_grid, w.tol)
    torch.cuda.synchronize()
    tol32 = float(np.float32(w.tol))
    ties = {"cand_ties": 0, "code_ties": 0, "stop_ties": 0}
    hist = np.zeros(w.max_points + 1, np.int64)
    err_rel = 0.0
    for li, (C, d) in enumerate(w.layers):
        W = Ws[li].cpu().numpy()
        out = (ls.codes[li].cpu().numpy(), ls.scales[li].cpu().numpy(), ls.counts[li].cpu().numpy(),
               ls.fit_err[li].cpu().numpy())
        v = assert_parity(orc, W, w.bits, w.max_points, w.n_grid, w.tol, out)
        for k in ties:
            ties[k] += int(v[k].sum())
        hist += np.bincount(out[2], minlength=w.max_points + 1)
        X = Xs[li].cpu().numpy()
        eo, _ = orc.output_error(W, out[0], out[1], out[2], X, with_ref=False)
        eg = ls.err[li].cpu().numpy()
        rel = np.abs(eg - eo) / np.maximum(eo, 1e-300)
        assert np.all(np.abs(eg - eo) <= 1e-5 * eo), (li, float(rel.max()))
        err_rel = max(err_rel, float(rel.max()))
        assert np.array_equal(ls.W_hat[li].cpu().numpy(), orc.reconstruct(out[0], out[1], out[2])), li
        say(f"  layer {li} ({C}x{d}) ok: points {int(out[2].sum())}")
        del out, W, X
    say(f"  {name}: {w.channels} channels, point counts {hist.tolist()}, ties {ties}, "
        f"largest output-error deviation {err_rel:.2e}")


@pytest.mark.parametrize("name", ["resnet18", "mobilenetv2"])
def test_batched_calls_equal_single_layer_calls(orc, name):
    """mpq_fit_layers / mpq_output_error_layers / mpq_reconstruct_layers on a
    whole workload give bitwise the outputs of the per-layer calls."""
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get(name)
    idx = list(range(len(w.layers)))[:12]
    Ws = [to_dev(wl.layer_weights(w, i)) for i in idx]
    Xs = [to_dev(wl.layer_calib(w, i, n=256)) for i in idx]
    say(f"case batched {name} ({len(idx)} layers)")
    ls = mpq.LayerSet(Ws, w.max_points, calib=Xs)
    ls.fit(w.bits, w.n_grid, w.tol)
    ls.output_error()
    ls.reconstruct()
    torch.cuda.synchronize()
    for j, i in enumerate(idx):
        c, s, n, e = mpq.fit_layer(Ws[j], w.bits, w.max_points, w.n_grid, w.tol)
        err, _ = mpq.output_error(Ws[j], c, s, n, Xs[j])
        Wh = mpq.reconstruct(c, s, n)
        torch.cuda.synchronize()
        assert torch.equal(c, ls.codes[j]) and torch.equal(s, ls.scales[j])
        assert torch.equal(n, ls.counts[j]) and torch.equal(e, ls.fit_err[j])
        assert torch.equal(err, ls.err[j]) and torch.equal(Wh, ls.W_hat[j])
    # one layer in lockstep
    j = len(idx) - 1
    out = (ls.codes[j].cpu().numpy(), ls.scales[j].cpu().numpy(), ls.counts[j].cpu().numpy(),
           ls.fit_err[j].cpu().numpy())
    assert_parity(orc, Ws[j].cpu().numpy(), w.bits, w.max_points, w.n_grid, w.tol, out)


def test_batched_fit_many_layers_one_variant(orc):
    """More layers of one kernel variant than one launch holds (48), mixed
    with empty layers and layers that take other variants."""
    import torch
    from paper_2002_09049_amd import mpq
    shapes = [(3, 40)] * 50 + [(0, 40), (5, 9), (4, 1000), (2, 40)]
    Ws = [to_dev(wl.random_weights(c, d, seed=i)) if c else torch.zeros((0, d), device="cuda")
          for i, (c, d) in enumerate(shapes)]
    say(f"case batched many layers ({len(shapes)})")
    ls = mpq.LayerSet(Ws, 4)
    ls.fit(4, 64, 1e-3)
    torch.cuda.synchronize()
    for i, (c, d) in enumerate(shapes):
        if c == 0:
            continue
        W = Ws[i].cpu().numpy()
        out = (ls.codes[i].cpu().numpy(), ls.scales[i].cpu().numpy(), ls.counts[i].cpu().numpy(),
               ls.fit_err[i].cpu().numpy())
        assert_parity(orc, W, 4, 4, 64, 1e-3, out)


@pytest.mark.parametrize("name", ["resnet18", "resnet50", "mobilenetv2", "vgg16fc"])
def test_quantize_layers_equals_the_three_calls(name):
    """mpq_quantize_layers (fit, output error and reconstruction as chains on
    several streams) gives bitwise the outputs of mpq_fit_layers,
    mpq_output_error_layers and mpq_reconstruct_layers; a layer without
    out_err or W_hat is left untouched there.  ResNet-50's 54 layers take
    several fit launches and error groups; VGG-16 fc's 25088-long channels
    take the fit that rebuilds its residual (its rows of D are formed)."""
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get(name)
    idx = list(range(len(w.layers)))
    Ws = [to_dev(wl.layer_weights(w, i)) for i in idx]
    Xs = [to_dev(wl.layer_calib(w, i, n=256)) for i in idx]
    say(f"case quantize_layers {name} ({len(idx)} layers)")
    ref = mpq.LayerSet(Ws, w.max_points, calib=Xs, with_ref=True)
    ref.fit(w.bits, w.n_grid, w.tol)
    ref.output_error()
    ref.reconstruct()
    q = mpq.LayerSet(Ws, w.max_points, calib=Xs, with_ref=True)
    for t in q.err + q.W_hat:
        t.fill_(-7.0)
    q.arr[1].out_err = None
    q.arr[1].out_ref = None
    q.arr[2].W_hat = None
    q.quantize(w.bits, w.n_grid, w.tol)
    torch.cuda.synchronize()
    for j in range(len(idx)):
        for a, b in ((ref.codes, q.codes), (ref.scales, q.scales), (ref.counts, q.counts),
                     (ref.fit_err, q.fit_err)):
            assert torch.equal(a[j], b[j]), j
        if j == 1:
            assert (q.err[j] == -7.0).all()
        else:
            assert torch.equal(ref.err[j], q.err[j]) and torch.equal(ref.ref[j], q.ref[j]), j
        if j == 2:
            assert (q.W_hat[j] == -7.0).all()
        else:
            assert torch.equal(ref.W_hat[j], q.W_hat[j]), j


def test_timing_only_records_the_named_kernel():
    """mpq_timing_only: with the recording on, only the named kernel's
    launches carry events (and positive durations); None records every
    launch again."""
    import torch
    from paper_2002_09049_amd import mpq
    w = wl.get("conv64x576")
    W = to_dev(wl.layer_weights(w, 0))
    X = to_dev(wl.layer_calib(w, 0))
    ls = mpq.LayerSet([W], w.max_points, calib=[X])
    say("case timing_only")
    mpq.timing_only("gemm_err_kernel")
    mpq.timing_enable(True)
    ls.quantize(w.bits, w.n_grid, w.tol)
    torch.cuda.synchronize()
    rec = mpq.timing_read()
    mpq.timing_enable(False)
    assert rec and all(n == "gemm_err_kernel" and ms > 0 for n, ms in rec)
    mpq.timing_only(None)
    mpq.timing_enable(True)
    ls.quantize(w.bits, w.n_grid, w.tol)
    torch.cuda.synchronize()
    names = {n for n, _ in mpq.timing_read()}
    mpq.timing_enable(False)
    assert {"gemm_err_kernel", "finish_err_kernel", "reconstruct_kernel"} <= names
    # the fit wrote the rows of D, so the whole-path call forms none; the
    # output error alone forms them from the stored points
    assert "form_d_kernel" not in names
    mpq.timing_enable(True)
    ls.output_error()
    ls.reconstruct()
    torch.cuda.synchronize()
    names = {n for n, _ in mpq.timing_read()}
    mpq.timing_enable(False)
    assert {"form_d_kernel", "gemm_err_kernel", "finish_err_kernel", "reconstruct_kernel"} <= names
