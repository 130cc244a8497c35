"""Host-side check of the index arithmetic by which the fit writes its rows of
the output error's residual D (the tiled layout of the error GEMM).

D holds tiles of 128 rows by 32 k, row-major inside, chunks of a row tile
contiguous: element j of row k sits at float
((k / 128) * nkb + j / 32) * 4096 + (k % 128) * 32 + j % 32, nkb = ceil(d / 32).
A fit workgroup of T threads holds EPT elements per thread, element
j = t + T * u.  Lane t stores element u when its chunk t / 32 + u T / 32 is
below nkb, at the row's base plus the byte offset (t / 32 * 4096 + t % 32) * 4
+ u (T / 32) * 4096 * 4.  This test restates that arithmetic for every
register-resident variant of the fit kernel and every channel length the
variant takes, and checks that:
  * every element j < d lands on its own slot of the tiled layout,
  * the stores past d fill exactly the row's zero padding (d <= j < 32 nkb),
  * no store leaves the row's nkb chunks (the buffer resource's range).
"""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2002_09049_amd", "csrc", "fit_hist.hip")


def _variants():
    text = open(SRC).read()
    body = re.search(r"kVariants\[\]\s*=\s*\{(.*?)\};", text, re.S).group(1)
    out = []
    for t, e, rb in re.findall(r"\{\s*(\d+)\s*,\s*(\d+)\s*,\s*(true|false)\s*\}", body):
        out.append((int(t), int(e), rb == "true"))
    assert out, "variant table not found"
    return out


def _cases():
    vs = _variants()
    cases = []
    lo = 1
    for T, EPT, rebuilt in vs:
        hi = T * EPT
        if not rebuilt:
            ds = sorted({lo, lo + 1, (lo + hi) // 2, hi - 31, hi - 1, hi} & set(range(lo, hi + 1)))
            for d in ds:
                cases.append((T, EPT, d))
        lo = hi + 1
    return cases


def tiled_slot(k, j, nkb):
    return ((k // 128) * nkb + j // 32) * 4096 + (k % 128) * 32 + j % 32


@pytest.mark.parametrize("T,EPT,d", _cases())
def test_fit_d_rows_land_in_their_row(T, EPT, d):
    assert T % 32 == 0
    nkb = (d + 31) // 32
    t = np.arange(T)[:, None]
    u = np.arange(EPT)[None, :]
    j = t + T * u
    chunk = t // 32 + u * (T // 32)
    store = chunk < nkb
    # every element of the channel is held by some (t, u)
    assert T * EPT >= d
    for k in (0, 5, 127, 128, 300):
        base = (k // 128) * nkb * 4096 + (k % 128) * 32            # floats
        byte = ((t // 32) * 4096 + t % 32) * 4 + u * (T // 32) * 4096 * 4
        assert (byte % 4 == 0).all()
        addr = base + byte // 4
        rec = (nkb * 4096 - (k % 128) * 32) * 4                     # the resource's bytes
        assert (byte[store] < rec).all() and (byte[store] >= 0).all()
        # each stored (t, u) hits element j's own slot
        want = tiled_slot(k, j, nkb)
        assert np.array_equal(addr[store], want[store])
        # elements j < d are all stored, once
        js = j[store]
        assert set(range(d)) <= set(js.tolist())
        assert len(js) == len(set(js.tolist()))
        # the stores past d are the row's padding and nothing else
        pad = sorted(js[js >= d].tolist())
        assert pad == list(range(d, 32 * nkb))
        # the slots written all belong to row k
        slots = addr[store]
        assert ((slots % 4096) // 32 == k % 128).all()
        assert ((slots // 4096) // nkb == k // 128).all()
