"""The error GEMM's operand split, modelled on the host: each fp32 value is
hi + mid + lo, three bf16 values each rounded to nearest from the remainder
so far, and a product is summed from six of the nine piece products.  These
checks pin the two facts the kernel's accuracy rests on: the split is exact
for finite values below bf16's largest, and the three products left out
(mid lo, lo mid, lo lo) stay below 2^-23 of the product."""
import numpy as np


def bf16_rne(x):
    """fp32 -> nearest bf16 (ties to even), returned as fp32."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return r.astype(np.uint32).view(np.float32)


def pieces(x):
    x = np.asarray(x, dtype=np.float32)
    h = bf16_rne(x)
    r1 = (x - h).astype(np.float32)
    m = bf16_rne(r1)
    r2 = (r1 - m).astype(np.float32)
    lo = bf16_rne(r2)
    return h, m, lo, r2


def _samples(n, seed):
    rng = np.random.default_rng(seed)
    mant = rng.uniform(1.0, 2.0, n)
    ex = rng.integers(-100, 100, n)
    sign = rng.choice([-1.0, 1.0], n)
    return (sign * np.ldexp(mant, ex)).astype(np.float32)


def test_split_is_exact():
    x = _samples(1 << 18, 1)
    h, m, lo, r2 = pieces(x)
    assert np.array_equal(lo, r2)                                  # the last remainder fits bf16
    exact = h.astype(np.float64) + m.astype(np.float64) + lo.astype(np.float64)
    assert np.array_equal(exact, x.astype(np.float64))
    # every piece is a bf16 value (low 16 bits zero)
    for p in (h, m, lo):
        assert not np.any(p.view(np.uint32) & 0xFFFF)


def test_six_products_within_bound():
    a, b = _samples(1 << 18, 2), _samples(1 << 18, 3)
    ah, am, al, _ = pieces(a)
    bh, bm, bl, _ = pieces(b)
    f = lambda v: v.astype(np.float64)
    six = f(ah) * f(bh) + f(ah) * f(bm) + f(am) * f(bh) + f(ah) * f(bl) + f(al) * f(bh) + f(am) * f(bm)
    exact = f(a) * f(b)
    assert np.all(np.abs(six - exact) <= 2.0 ** -23 * np.abs(exact))


def test_worked_example():
    # 1 + 2^-9 + 2^-18 + 2^-23: bf16 keeps 8 significant bits, so hi = 1
    # (the rest is below half of 2^-7), mid = 2^-9 (the rest below half of
    # 2^-16), lo = 2^-18 + 2^-23 (six bits apart: exact)
    x = np.float32(1.0 + 2.0 ** -9 + 2.0 ** -18 + 2.0 ** -23)
    h, m, lo, _ = pieces(np.array([x]))
    assert h[0] == 1.0 and m[0] == np.float32(2.0 ** -9) and lo[0] == np.float32(2.0 ** -18 + 2.0 ** -23)
