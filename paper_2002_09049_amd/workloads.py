"""Seeded synthetic inputs for the multipoint fit.

This module only draws random numbers and knows layer shapes. It holds none
of the fit's arithmetic, so both the HIP path and the oracle may use it.

The paper fits pretrained ImageNet/VOC networks (Sec. 5, "Experiment Results
on ImageNet Benchmark"); those weights and images are not available here.
Each workload below instead draws weights of the real layer shapes of the
named architecture from a stated distribution, and a synthetic calibration
batch X (the per-layer input batch D_L of Algorithm 2) of stated size.

Shapes are (C_out, d) with d = C_in * k * k, i.e. a conv kernel flattened to
one vector per output channel (Sec. 3.1, Eq. (3) and the remark after it).

Generation uses ``numpy.random.default_rng([seed, layer_index])`` and draws,
in this order: the weights, the per-channel scale factors, the outlier
positions, then X.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Tuple

import numpy as np

Shape = Tuple[int, int]


# ---------------------------------------------------------------- layer shapes
def resnet18_shapes() -> List[Shape]:
    """All 20 conv layers plus fc of ResNet-18 as (C_out, C_in*k*k)."""
    s: List[Shape] = [(64, 3 * 7 * 7)]
    s += [(64, 64 * 9)] * 4
    cin = 64
    for w in (128, 256, 512):
        s.append((w, cin * 9))          # first 3x3 of the stage (stride 2)
        s.append((w, w * 9))            # second 3x3 of the first block
        s.append((w, cin))              # 1x1 downsample
        s += [(w, w * 9)] * 2           # second block
        cin = w
    s.append((1000, 512))               # fc
    return s


def resnet50_shapes() -> List[Shape]:
    """The 53 conv layers plus fc of ResNet-50 (bottleneck blocks)."""
    s: List[Shape] = [(64, 3 * 7 * 7)]
    cin = 64
    for w, nblocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(nblocks):
            s.append((w, cin))          # 1x1 reduce
            s.append((w, w * 9))        # 3x3
            s.append((4 * w, w))        # 1x1 expand
            if b == 0:
                s.append((4 * w, cin))  # 1x1 downsample
            cin = 4 * w
    s.append((1000, 2048))
    return s


def mobilenetv2_shapes() -> List[Tuple[Shape, str]]:
    """Depthwise (C x 9) and pointwise (C_out x C_in) layers of MobileNetV2.

    The stem conv and the classifier are not included.  Returns
    ((C_out, d), kind) with kind in {"dw", "pw"}.
    """
    out: List[Tuple[Shape, str]] = []
    cin = 32
    for t, c, n in ((1, 16, 1), (6, 24, 2), (6, 32, 3), (6, 64, 4),
                    (6, 96, 3), (6, 160, 3), (6, 320, 1)):
        for _ in range(n):
            h = cin * t
            if t != 1:
                out.append(((h, cin), "pw"))   # expand
            out.append(((h, 9), "dw"))         # depthwise 3x3
            out.append(((c, h), "pw"))         # project
            cin = c
    out.append(((1280, 320), "pw"))
    return out


def vgg16_fc_shapes() -> List[Shape]:
    return [(4096, 25088), (4096, 4096), (1000, 4096)]


# ------------------------------------------- output sizes at a 224 x 224 input
def resnet18_out_hw() -> List[int]:
    """Output height (= width) of each layer of resnet18_shapes() for a 224 x
    224 image (the stem conv has stride 2, then a stride-2 max pool; each
    later stage halves the size in its first 3x3 and its downsample)."""
    return [112] + [56] * 4 + [28] * 5 + [14] * 5 + [7] * 5 + [1]


def resnet50_out_hw() -> List[int]:
    """Output size of each layer of resnet50_shapes() for a 224 x 224 image
    (the stride of a stage's first block sits in its 3x3 conv and its
    downsample)."""
    out, res = [112], 56
    for w, nblocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(nblocks):
            o = res // 2 if (b == 0 and w != 64) else res
            out += [res, o, o] + ([o] if b == 0 else [])
            res = o
    out.append(1)
    return out


def mobilenetv2_full_layers() -> List[Tuple[Shape, int, str]]:
    """Every weight layer of MobileNetV2 with its output size for a 224 x 224
    image: the stem 3x3 conv (32 x 27, stride 2), the inverted-residual
    blocks of mobilenetv2_shapes() (a block's stride sits in its depthwise
    conv), the final 1x1 conv and the classifier.  ((C_out, d), hw, kind)."""
    out: List[Tuple[Shape, int, str]] = [((32, 27), 112, "stem")]
    cin, res = 32, 112
    for t, c, n, st in ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
                        (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1)):
        for b in range(n):
            h = cin * t
            if t != 1:
                out.append(((h, cin), res, "pw"))
            o = res // (st if b == 0 else 1)
            out.append(((h, 9), o, "dw"))
            out.append(((c, h), o, "pw"))
            cin, res = c, o
    out.append(((1280, 320), 7, "pw"))
    out.append(((1000, 1280), 1, "fc"))
    return out


# ------------------------------------------------------------------- workloads
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    layers: Tuple[Shape, ...]
    bits: int
    max_points: int
    n_grid: int
    tol: float
    n_calib: int          # columns of X (calibration batch size)
    seed: int
    weight_dist: str      # "gauss_lognorm" | "laplace_outlier"
    fan: str              # variance numerator: "he" -> 2/d, "lecun" -> 1/d
    chan_sigma: float     # sigma of the per-channel log-normal factor (0: none)
    x_dist: str           # "normal" | "relu_normal"
    dw_shared_x: bool = False  # depthwise layers share one 9 x N batch

    @property
    def channels(self) -> int:
        return sum(c for c, _ in self.layers)

    @property
    def weights(self) -> int:
        return sum(c * d for c, d in self.layers)


def _single_conv() -> Workload:
    return Workload("conv64x576", ((64, 576),), bits=4, max_points=4,
                    n_grid=128, tol=1e-3, n_calib=256, seed=0,
                    weight_dist="gauss_lognorm", fan="he", chan_sigma=0.5,
                    x_dist="normal")


def _resnet18() -> Workload:
    return Workload("resnet18", tuple(resnet18_shapes()), bits=4, max_points=4,
                    n_grid=256, tol=1e-3, n_calib=1024, seed=1,
                    weight_dist="gauss_lognorm", fan="he", chan_sigma=0.5,
                    x_dist="relu_normal")


def _resnet50() -> Workload:
    return Workload("resnet50", tuple(resnet50_shapes()), bits=4, max_points=8,
                    n_grid=256, tol=1e-3, n_calib=1024, seed=2,
                    weight_dist="laplace_outlier", fan="he", chan_sigma=0.0,
                    x_dist="relu_normal")


def _mobilenetv2() -> Workload:
    return Workload("mobilenetv2", tuple(s for s, _ in mobilenetv2_shapes()),
                    bits=4, max_points=8, n_grid=512, tol=1e-3, n_calib=1024,
                    seed=3, weight_dist="gauss_lognorm", fan="he",
                    chan_sigma=1.0, x_dist="normal", dw_shared_x=True)


def _vgg16_fc() -> Workload:
    return Workload("vgg16fc", tuple(vgg16_fc_shapes()), bits=3, max_points=8,
                    n_grid=512, tol=5e-4, n_calib=2048, seed=4,
                    weight_dist="gauss_lognorm", fan="lecun", chan_sigma=0.5,
                    x_dist="normal")


WORKLOADS = {w.name: w for w in (_single_conv(), _resnet18(), _resnet50(),
                                 _mobilenetv2(), _vgg16_fc())}
# configs in the order they are numbered in the docs (1..5)
ORDER = ["conv64x576", "resnet18", "resnet50", "mobilenetv2", "vgg16fc"]


def get(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return WORKLOADS[ORDER[name_or_index - 1]]
    return WORKLOADS[name_or_index]


def _rng(seed: int, layer: int) -> np.random.Generator:
    return np.random.default_rng([seed, layer])


def layer_weights(wl: Workload, layer: int) -> np.ndarray:
    """fp32 weights [C_out, d] of layer ``layer`` (draws W, scales, outliers)."""
    c, d = wl.layers[layer]
    rng = _rng(wl.seed, layer)
    sigma = math.sqrt((2.0 if wl.fan == "he" else 1.0) / d)
    if wl.weight_dist == "gauss_lognorm":
        w = rng.standard_normal((c, d)) * sigma
    elif wl.weight_dist == "laplace_outlier":
        w = rng.laplace(0.0, sigma / math.sqrt(2.0), size=(c, d))
    else:
        raise ValueError(wl.weight_dist)
    if wl.chan_sigma > 0:
        w *= np.exp(rng.standard_normal((c, 1)) * wl.chan_sigma)
    if wl.weight_dist == "laplace_outlier":
        n_out = int(round(0.001 * c * d))
        pos = rng.choice(c * d, size=n_out, replace=False)
        flat = w.reshape(-1)
        flat[pos] = np.where(flat[pos] < 0, -1.0, 1.0) * 8.0 * sigma
    return np.ascontiguousarray(w, dtype=np.float32)


def layer_calib(wl: Workload, layer: int, n: Optional[int] = None) -> np.ndarray:
    """fp32 calibration batch X [d, N] of layer ``layer``.

    Drawn after the weights from the same per-layer generator, so a layer's
    X does not depend on any other layer.  With ``dw_shared_x`` every
    depthwise (d == 9) layer uses the batch of the first depthwise layer.
    """
    c, d = wl.layers[layer]
    if wl.dw_shared_x and d == 9:
        first = next(i for i, (_, dd) in enumerate(wl.layers) if dd == 9)
        if first != layer:
            return layer_calib(wl, first, n)
    layer_weights_rng = _rng(wl.seed, layer)
    # replay the weight draws so X comes after them in the stream
    _replay_weight_draws(wl, layer, layer_weights_rng)
    n = wl.n_calib if n is None else n
    x = layer_weights_rng.standard_normal((d, n))
    if wl.x_dist == "relu_normal":
        x = np.maximum(x, 0.0)
    return np.ascontiguousarray(x, dtype=np.float32)


def _replay_weight_draws(wl: Workload, layer: int, rng: np.random.Generator) -> None:
    c, d = wl.layers[layer]
    if wl.weight_dist == "gauss_lognorm":
        rng.standard_normal((c, d))
    else:
        rng.laplace(0.0, 1.0, size=(c, d))
    if wl.chan_sigma > 0:
        rng.standard_normal((c, 1))
    if wl.weight_dist == "laplace_outlier":
        rng.choice(c * d, size=int(round(0.001 * c * d)), replace=False)


def random_weights(c: int, d: int, seed: int, chan_sigma: float = 0.5) -> np.ndarray:
    """Small ad-hoc weights for tests: N(0, 2/d) times a per-channel log-normal."""
    rng = np.random.default_rng([seed, 999])
    w = rng.standard_normal((c, d)) * math.sqrt(2.0 / max(d, 1))
    if chan_sigma > 0:
        w *= np.exp(rng.standard_normal((c, 1)) * chan_sigma)
    return np.ascontiguousarray(w, dtype=np.float32)


def random_calib(d: int, n: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng([seed, 998])
    return np.ascontiguousarray(rng.standard_normal((d, n)), dtype=np.float32)
