"""The short-channel fit (d <= 16: one wavefront per channel, lanes over the
candidates, fit_small.hip) against the oracle's lockstep verifier.

The 3 x 3 depthwise filters (d = 9) are most of MobileNetV2's channels.
The cases span the lengths on both sides of the variant boundary (16 / 17),
channel counts that leave a workgroup's wavefronts partly idle, grids from 1
to 4096 candidates, 2 to 8 bits, and the channels that take the fp64 code
path of the search (scales outside [2^-100, 2^100], quotients on
half-integers).  The other modes (refit, clipping, asymmetric codes, the
naive-first gate, the calibration rule) have d <= 16 rows in their own
tests.
"""
import numpy as np
import pytest

from gpu_util import assert_parity, free_running_diff, gpu_fit, say
from paper_2002_09049_amd import workloads as wl

pytestmark = pytest.mark.gpu

CONFIGS = [
    # (bits, P, G, tol)
    (4, 8, 512, 1e-3),
    (2, 6, 64, 0.0),
    (8, 3, 4096, 0.0),
    (3, 8, 7, 1e-4),
    (4, 4, 1, 0.0),
]
LENGTHS = [1, 2, 3, 7, 8, 9, 12, 15, 16, 17]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2002_09049_amd import mpq
    mpq.load()
    yield


def test_short_channels_take_the_wavefront_kernel():
    from paper_2002_09049_amd import mpq
    for d in range(1, 17):
        assert mpq.fit_kernel_of(d, 4, 512, True) == f"fit_small_kernel<{d}>"
        assert mpq.fit_kernel_of(d, 4, 512, False) == f"fit_small_kernel<{d}>"
    assert mpq.fit_kernel_of(17, 4, 512, True).startswith("fit_hist_kernel<64,1,")


@pytest.mark.parametrize("d", LENGTHS)
@pytest.mark.parametrize("bits,P,G,tol", CONFIGS, ids=[f"b{b}_P{p}_G{g}" for b, p, g, _ in CONFIGS])
def test_short_parity(orc, d, bits, P, G, tol):
    C = 70   # 17 workgroups of four channels, the last one half idle
    say(f"case short d={d} bits={bits} P={P} G={G} tol={tol}")
    W = wl.random_weights(C, d, seed=31 * d + G)
    out = gpu_fit(W, bits, P, G, tol)
    v = assert_parity(orc, W, bits, P, G, tol, out)
    tie_channels = int(((v["cand_ties"] + v["code_ties"] + v["stop_ties"]) > 0).sum())
    nd = free_running_diff(orc, W, bits, P, G, tol, out)
    say(f"  tie channels={tie_channels} free-running diffs={nd}")
    assert nd <= tie_channels


@pytest.mark.parametrize("d", [9, 16])
def test_short_edge_channels(orc, d):
    rng = np.random.default_rng(d)
    W = np.zeros((13, d), np.float32)
    W[1] = 0.3 * np.sign(rng.standard_normal(d))            # all |w| equal
    W[2, d // 2] = -2.5                                       # one nonzero
    W[3] = rng.uniform(-3e38, 3e38, d)                        # scales above 2^100
    W[4] = rng.standard_normal(d) * 1e-35                     # scales below 2^-100
    W[5, :3] = [1e-45, 0.0, -1e-45]                           # subnormal: no candidate
    W[6] = rng.standard_normal(d)
    W[6, 1::2] = W[6, 0:d - 1:2]                              # repeated values
    W[7] = np.arange(d, dtype=np.float32) / 7.0
    W[8:] = rng.integers(-8, 9, (5, d)) / np.float32(4)       # quotients on half-integers
    for bits, G, P, tol in ((4, 128, 4, 1e-3), (2, 8, 6, 0.0), (3, 6, 5, 0.0), (8, 32, 2, 0.0),
                            (4, 512, 8, 0.0)):
        say(f"case short edges d={d} bits={bits} G={G} P={P} tol={tol}")
        out = gpu_fit(W, bits, P, G, tol)
        assert_parity(orc, W, bits, P, G, tol, out)
        codes, scales, counts, err = out
        assert counts[0] == 0 and (codes[0] == 0).all() and (scales[0] == 0).all()
        if tol > 0:
            assert counts[1] == 1
        assert counts[5] == (1 if bits == 2 else 0)


def test_short_explicit_grid(orc):
    W = wl.random_weights(45, 9, seed=4)
    grid = np.sort(np.random.default_rng(8).uniform(0.05, 1.0, 100)).astype(np.float32)
    grid[-1] = 1.0
    say("case short explicit grid")
    out = gpu_fit(W, 4, 6, 100, 1e-4, grid=grid)
    assert_parity(orc, W, 4, 6, 100, 1e-4, out, grid=grid)
    out2 = gpu_fit(W, 4, 6, 100, 1e-4, grid=grid, with_err=False)
    for a, b in zip(out[:3], out2[:3]):
        assert np.array_equal(a, b)


def test_short_deterministic():
    W = wl.random_weights(257, 9, seed=12)
    a = gpu_fit(W, 4, 8, 512, 1e-3)
    b = gpu_fit(W, 4, 8, 512, 1e-3)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
