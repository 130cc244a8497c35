"""Parity of the deployment arithmetic (Sec. 3.4, Eq. (14)-(15)) with the
oracle, through the C ABI: integer work, so every output is compared bit
for bit."""
import numpy as np
import pytest

from gpu_util import gpu_fit, say, to_dev
from paper_2002_09049_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2002_09049_amd import mpq
    mpq.load()
    yield


def _gpu_scales(scales, counts, p):
    import torch
    from paper_2002_09049_amd import mpq
    A, cl = mpq.integer_scales(to_dev(scales), to_dev(counts), p)
    torch.cuda.synchronize()
    return A.cpu().numpy(), int(cl.cpu().numpy()[0])


def _gpu_forward(codes, A, counts, X, p):
    import torch
    from paper_2002_09049_amd import mpq
    Y = mpq.integer_forward(to_dev(codes), to_dev(A), to_dev(counts), to_dev(X), p)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def test_integer_scales_exact(orc):
    rng = np.random.default_rng(3)
    for p in (0, 6, 15, 24, 31):
        u = 2.0 ** -p
        s = (rng.standard_normal((300, 6)) * 0.05).astype(np.float32)
        s[0, :6] = np.array([2.5, 3.5, -2.5, 0.5, 1.5, -0.5], np.float64) * u   # half-way ties
        s[1, :3] = [1.0, -1.0, 0.75]
        counts = rng.integers(0, 7, 300).astype(np.int32)
        counts[:2] = 6
        say(f"case integer scales p={p}")
        Ag, ng = _gpu_scales(s, counts, p)
        Ao, no = orc.integer_scales(s, counts, p)
        assert np.array_equal(Ag, Ao) and ng == no


CASES = [
    # (C, P, d, N, p)
    (5, 3, 13, 7, 0),       # byte loads, one tile
    (70, 2, 36, 129, 7),    # 4-byte loads, ragged columns
    (130, 4, 64, 300, 11),  # 16-byte loads, ragged rows and columns
    (257, 8, 147, 33, 20),  # byte loads, three row tiles
    (40, 4, 1, 1, 3),       # d = 1, one column
    (64, 4, 576, 260, 30),  # 16-byte loads, several K slabs
    (33, 5, 1000, 64, 16),  # 4-byte loads (1000 % 16 != 0)
]


@pytest.mark.parametrize("C,P,d,N,p", CASES, ids=[f"C{c}_P{q}_d{d}_N{n}_p{p}" for c, q, d, n, p in CASES])
def test_integer_forward_exact(orc, C, P, d, N, p):
    rng = np.random.default_rng(C * 31 + d)
    codes = rng.integers(-7, 8, (C, P, d)).astype(np.int8)     # nonzero past the counts too
    A = rng.integers(-(2 ** 24), 2 ** 24, (C, P)).astype(np.int32)
    counts = rng.integers(0, P + 1, C).astype(np.int32)
    counts[0] = 0
    counts[-1] = P
    X = rng.integers(-128, 128, (N, d)).astype(np.int8)
    say(f"case integer forward C={C} P={P} d={d} N={N} p={p}")
    Yg = _gpu_forward(codes, A, counts, X, p)
    Yo = orc.integer_forward(codes, A, counts, X, p)
    assert np.array_equal(Yg, Yo), np.argwhere(Yg != Yo)[:5]


def test_fit_then_integer_forward_at_layer_size(orc):
    """The whole deployment chain at a real layer shape: GPU fit of a
    ResNet-18 512 x 4608 layer's weights, integer scales, integer forward of
    a batch of 392 columns (8 images x 7 x 7); sampled channels against the
    oracle, bit for bit."""
    w = wl.get("resnet18")
    li = next(i for i, (c, d) in enumerate(w.layers) if (c, d) == (512, 4608))
    W = wl.layer_weights(w, li)
    say("case fit + integer forward, 512 x 4608, N = 392")
    codes, scales, counts, _ = gpu_fit(W, w.bits, w.max_points, w.n_grid, w.tol)
    p = 20
    A, ncl = _gpu_scales(scales, counts, p)
    Ao, _ = orc.integer_scales(scales, counts, p)
    assert ncl == 0 and np.array_equal(A, Ao)
    rng = np.random.default_rng(5)
    X = rng.integers(-128, 128, (392, 4608)).astype(np.int8)
    Y = _gpu_forward(codes, A, counts, X, p)
    ch = np.unique(np.concatenate([[0, 511], rng.choice(512, 12, replace=False)]))
    Yo = orc.integer_forward(codes[ch], A[ch], counts[ch], X, p)
    assert np.array_equal(Y[ch], Yo)


def test_integer_forward_layers_equals_single_calls():
    import torch
    from paper_2002_09049_amd import mpq
    rng = np.random.default_rng(8)
    shapes = [(3, 40, 17), (0, 9, 5), (130, 64, 140), (20, 147, 1), (64, 576, 300)] + [(4, 16, 8)] * 33
    layers, singles = [], []
    P, p = 4, 9
    say(f"case integer forward layers ({len(shapes)})")
    for C, d, N in shapes:
        codes = to_dev(rng.integers(-7, 8, (C, P, d)).astype(np.int8))
        A = to_dev(rng.integers(-(2 ** 20), 2 ** 20, (C, P)).astype(np.int32))
        counts = to_dev(rng.integers(0, P + 1, C).astype(np.int32))
        X = to_dev(rng.integers(-128, 128, (N, d)).astype(np.int8))
        Y = torch.full((C, N), -7, dtype=torch.int64, device="cuda")
        layers.append((codes, A, counts, X, Y))
    mpq.integer_forward_layers(layers, P, p)
    torch.cuda.synchronize()
    for codes, A, counts, X, Y in layers:
        Y1 = mpq.integer_forward(codes, A, counts, X, p)
        torch.cuda.synchronize()
        assert torch.equal(Y, Y1)
