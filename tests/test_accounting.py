"""Size and OPs accounting of Sec. 3.4 / Table 1 (host arithmetic) pinned to
the sizes and OPs the paper prints for naively quantized networks, and to
Table 1's closed forms."""
import json
import os

import numpy as np

from paper_2002_09049_amd import accounting as ac, workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table_sizes_ops.json")


def _layers(net, counted):
    if net == "resnet18":
        L = [(c, d, h * h) for (c, d), h in zip(wl.resnet18_shapes(), wl.resnet18_out_hw())]
    elif net == "resnet50":
        L = [(c, d, h * h) for (c, d), h in zip(wl.resnet50_shapes(), wl.resnet50_out_hw())]
    else:
        L = [(c, d, h * h) for (c, d), h, _ in wl.mobilenetv2_full_layers()]
    return L[1:-1] if counted == "first_last_excluded" else L[:-1]


def test_printed_naive_sizes_and_ops():
    """Every printed figure is reproduced to its printed precision.  ResNet-18
    W4/A8 computes 847.77 M against a printed 847.78 M: twice the rounded
    W4/A4 figure (2 x 423.89); the test allows that last-digit difference."""
    for c in json.load(open(GOLDEN))["cases"]:
        r = ac.network_cost(_layers(c["net"], c["counted"]), *c["bits"])
        got_ops = r["ops"] / 1e6
        slack = 0.011 if c["bits"] == [4, 8] else 0.005
        assert abs(got_ops - c["ops_M"]) <= slack, (c, got_ops)
        if "MB" in c:
            assert abs(r["bytes"] / 2 ** 20 - c["MB"]) <= 0.005, (c, r["bytes"] / 2 ** 20)
        if "fp32_MB" in c:
            assert abs(r["fp32_bytes"] / 2 ** 20 - c["fp32_MB"]) <= 0.005, c


def test_layer_shapes_are_the_architectures():
    assert len(wl.resnet18_out_hw()) == len(wl.resnet18_shapes())
    assert len(wl.resnet50_out_hw()) == len(wl.resnet50_shapes())
    full = [s for s, _, k in wl.mobilenetv2_full_layers() if k in ("pw", "dw")]
    assert full == [s for s, _ in wl.mobilenetv2_shapes()]


def test_table1_closed_forms():
    """Table 1 for one channel of d = 9, N = 4 bits, n = 3 points, worked by
    hand: memory 3*9*4 + 32*3 = 204 bits; multiplications
    3*(9*16 + 1024) = 3504 binary ops."""
    assert ac.channel_memory_bits(9, 4) == 36 and ac.channel_mul_binops(9, 4, 4) == 144
    assert ac.channel_memory_bits(9, 4, 3) == 204
    assert ac.channel_mul_binops(9, 4, 4, 3) == 3504


def test_multipoint_cost_is_linear_in_points():
    """With one point per channel the multipoint layer costs the naive one
    plus a 32-bit scale per channel and a 32 x 32 product per output; each
    further point adds the naive cost again plus the same overhead."""
    L = [(64, 576, 3136), (128, 1152, 784), (1000, 512, 1)]
    naive = ac.network_cost(L, 4, 8)
    one = ac.network_cost(L, 4, 8, [np.ones(c, np.int64) for c, _, _ in L])
    two = ac.network_cost(L, 4, 8, [np.full(c, 2, np.int64) for c, _, _ in L])
    ch = sum(c for c, _, _ in L)
    outs = sum(c * hw for c, _, hw in L)
    assert one["bytes"] == naive["bytes"] + 4 * ch
    assert one["ops"] == naive["ops"] + outs * 1024 / 64
    assert two["bytes"] - one["bytes"] == one["bytes"] and two["ops"] - one["ops"] == one["ops"]
