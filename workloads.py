"""Seeded synthetic workloads: layer shapes and input generators.

This module is shared by the tests, the benchmark and the smoke check.  It
holds only data (layer shapes, including each layer's output extent as a
stated configuration value) and random-number recipes; none of the
convolution's arithmetic lives here, so neither the oracle nor the HIP
library depends on it.

Recipe (used for every config):
  * each tensor is drawn in consecutive chunks of 2^22 elements of its
    row-major order; chunk j of tensor t of layer ``layer`` of configuration
    ``cfg`` comes from ``numpy.random.default_rng([1903, cfg, layer, t, j])``
    with t = 0 for x, 1 for w, 2 for b, 3 for dy (chunks are drawn on
    parallel threads; the values do not depend on the thread count, and a
    smaller batch gives exactly the leading images of the full batch);
  * values are drawn in float64 and rounded once to float32 (round to
    nearest even); the float32 arrays are the canonical inputs to both sides;
  * x, dy ~ N(0, 1);
  * w ~ He-uniform U(+-sqrt(6 / fan_in)) or Xavier-uniform
    U(+-sqrt(6 / (fan_in + fan_out))), fan_in = (C/G) R S, fan_out = (K/G) R S;
  * b ~ U(-0.1, 0.1).

The configurations (five convolution stacks, and the AlexNet network step
with its pooling and inner-product layers) stand in for the paper's ImageNet
networks (AlexNet, VGG-16, ResNet-50, GoogLeNet; Sec. VI, Tables II and III):
same layer shapes, synthetic values, no dataset and no trained weights.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

CHUNK = 1 << 22


@dataclass(frozen=True)
class Layer:
    name: str
    N: int
    C: int
    H: int
    W: int
    K: int
    R: int
    S: int
    stride: int
    pad: int
    group: int
    P: int          # stated output height (configuration data)
    Q: int          # stated output width
    init: str       # "he" | "xavier"
    count: int = 1  # how many times the layer occurs in its stack
    first: bool = False  # network's first layer: its bwd-data is not needed

    @property
    def shape(self):
        return (self.N, self.C, self.H, self.W, self.K, self.R, self.S,
                self.stride, self.pad, self.group)

    def with_batch(self, n: int) -> "Layer":
        return replace(self, N=n)


def _sq(name, N, C, HW, K, RS, stride, pad, group, PQ, init, count=1, first=False):
    return Layer(name, N, C, HW, HW, K, RS, RS, stride, pad, group, PQ, PQ, init, count, first)


def _tiny():
    return [_sq("conv", 2, 16, 32, 32, 3, 1, 1, 1, 32, "he")]


def _alexnet(N=128):
    x = "xavier"
    return [
        _sq("conv1", N, 3, 227, 96, 11, 4, 0, 1, 55, x, first=True),
        _sq("conv2", N, 96, 27, 256, 5, 1, 2, 2, 27, x),
        _sq("conv3", N, 256, 13, 384, 3, 1, 1, 1, 13, x),
        _sq("conv4", N, 384, 13, 384, 3, 1, 1, 2, 13, x),
        _sq("conv5", N, 384, 13, 256, 3, 1, 1, 2, 13, x),
    ]


def _vgg16(N=32):
    h = "he"
    plan = [("conv1_1", 3, 64, 224), ("conv1_2", 64, 64, 224),
            ("conv2_1", 64, 128, 112), ("conv2_2", 128, 128, 112),
            ("conv3_1", 128, 256, 56), ("conv3_2", 256, 256, 56), ("conv3_3", 256, 256, 56),
            ("conv4_1", 256, 512, 28), ("conv4_2", 512, 512, 28), ("conv4_3", 512, 512, 28),
            ("conv5_1", 512, 512, 14), ("conv5_2", 512, 512, 14), ("conv5_3", 512, 512, 14)]
    return [_sq(n, N, c, s, k, 3, 1, 1, 1, s, h, first=(i == 0))
            for i, (n, c, k, s) in enumerate(plan)]


def _resnet50(N=64):
    # Steady-state bottleneck block of each stage (reduce input is 4x the
    # width), weighted by ResNet-50's block counts 3/4/6/3; the three
    # stride-2 1x1 projections and the 7x7 stem occur once each.
    h = "he"
    out = [_sq("stem", N, 3, 224, 64, 7, 2, 3, 1, 112, h, first=True)]
    for s, w, blocks in ((56, 64, 3), (28, 128, 4), (14, 256, 6), (7, 512, 3)):
        out += [
            _sq(f"s{s}_reduce", N, 4 * w, s, w, 1, 1, 0, 1, s, h, blocks),
            _sq(f"s{s}_3x3", N, w, s, w, 3, 1, 1, 1, s, h, blocks),
            _sq(f"s{s}_expand", N, w, s, 4 * w, 1, 1, 0, 1, s, h, blocks),
        ]
    for s, cin in ((56, 256), (28, 512), (14, 1024)):
        out.append(_sq(f"proj{s}", N, cin, s, 2 * cin, 1, 2, 0, 1, s // 2, h))
    return out


def _googlenet(N=64):
    # Three inception modules built from the stated channel ranges: the low
    # and high endpoints, and one interpolated module between them.
    x = "xavier"
    out = []
    for tag, s, cin, c1, r3, c3, r5, c5 in (("lo", 28, 192, 64, 96, 128, 16, 32),
                                           ("mid", 14, 512, 192, 128, 256, 32, 64),
                                           ("hi", 14, 832, 384, 192, 384, 48, 128)):
        out += [
            _sq(f"{tag}_1x1", N, cin, s, c1, 1, 1, 0, 1, s, x),
            _sq(f"{tag}_r3", N, cin, s, r3, 1, 1, 0, 1, s, x),
            _sq(f"{tag}_3x3", N, r3, s, c3, 3, 1, 1, 1, s, x),
            _sq(f"{tag}_r5", N, cin, s, r5, 1, 1, 0, 1, s, x),
            _sq(f"{tag}_5x5", N, r5, s, c5, 5, 1, 2, 1, s, x),
        ]
    return out


@dataclass(frozen=True)
class PoolLayer:
    """A pooling layer (max or average over R x S windows)."""
    name: str
    N: int
    C: int
    H: int
    W: int
    R: int
    S: int
    stride: int
    pad: int
    mode: str       # "max" | "avg"
    P: int          # stated output extent (configuration data)
    Q: int
    count: int = 1
    first: bool = False

    @property
    def pshape(self):
        return (self.N, self.C, self.H, self.W, self.R, self.S, self.stride, self.pad)

    def with_batch(self, n: int) -> "PoolLayer":
        return replace(self, N=n)


def _alexnet_net(N=128):
    # The AlexNet-shaped stack with its three overlapping 3x3 / 2 max-pools and
    # its three inner-product layers (each the convolution of 1 x 1 images
    # with 1 x 1 filters): the layers of a whole network step minus the
    # element-wise ones (activations, normalisation, dropout, loss).
    c = _alexnet(N)
    x = "xavier"

    def pool(name, C, HW, PQ):
        return PoolLayer(name, N, C, HW, HW, 3, 3, 2, 0, "max", PQ, PQ)

    def fc(name, cin, cout):
        return _sq(name, N, cin, 1, cout, 1, 1, 0, 1, 1, x)

    return [c[0], pool("pool1", 96, 55, 27), c[1], pool("pool2", 256, 27, 13), c[2], c[3],
            c[4], pool("pool5", 256, 13, 6), fc("fc6", 256 * 6 * 6, 4096),
            fc("fc7", 4096, 4096), fc("fc8", 4096, 1000)]


CONFIGS = {
    0: ("tiny", _tiny()),
    1: ("alexnet", _alexnet()),
    2: ("vgg16", _vgg16()),
    3: ("resnet50", _resnet50()),
    4: ("googlenet", _googlenet()),
    5: ("alexnet_net", _alexnet_net()),
}


def config(cfg: int):
    """(name, [Layer, ...]) of configuration ``cfg``."""
    return CONFIGS[cfg]


def _draw(key, shape, fill):
    """float32 array of ``shape`` whose chunk j is ``fill(rng_j, n)`` (float64
    draws, rounded to float32) with rng_j = default_rng([1903, *key, j])."""
    out = np.empty(shape, dtype=np.float32)
    flat = out.reshape(-1)
    total = flat.size

    def one(j):
        n = min(CHUNK, total - j * CHUNK)
        flat[j * CHUNK:j * CHUNK + n] = fill(np.random.default_rng([1903, *key, j]), n)

    nchunks = (total + CHUNK - 1) // CHUNK
    if nchunks <= 1:
        for j in range(nchunks):
            one(j)
    else:
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1, nchunks)) as ex:
            list(ex.map(one, range(nchunks)))
    return out


def _normal(key, shape):
    return _draw(key, shape, lambda rng, n: rng.standard_normal(n, dtype=np.float64))


def _uniform(key, lim, shape):
    return _draw(key, shape, lambda rng, n: rng.uniform(-lim, lim, n))


def weight_limit(C, K, R, S, group, init):
    fan_in = (C // group) * R * S
    fan_out = (K // group) * R * S
    if init == "he":
        return float(np.sqrt(6.0 / fan_in))
    if init == "xavier":
        return float(np.sqrt(6.0 / (fan_in + fan_out)))
    raise ValueError(init)


def make_inputs(shape, P, Q, seed=(0, 0), init="he", tensors=("x", "w", "b", "dy")):
    """Seeded float32 inputs for a layer of ``shape`` =
    (N,C,H,W,K,R,S,stride,pad,group) whose output is P x Q.
    Returns a dict with the requested keys among x, w, b, dy."""
    N, C, H, W, K, R, S, _, _, group = shape
    cfg, li = seed
    out = {}
    if "x" in tensors:
        out["x"] = _normal((cfg, li, 0), (N, C, H, W))
    if "w" in tensors:
        lim = weight_limit(C, K, R, S, group, init)
        out["w"] = _uniform((cfg, li, 1), lim, (K, C // group, R, S))
    if "b" in tensors:
        out["b"] = _uniform((cfg, li, 2), 0.1, (K,))
    if "dy" in tensors:
        out["dy"] = _normal((cfg, li, 3), (N, K, P, Q))
    return out


def pool_inputs(cfg: int, li: int, layer: PoolLayer):
    """x [N,C,H,W] and dy [N,C,P,Q] of pooling layer ``li`` of ``cfg``, drawn
    like a convolution layer's x and dy (t = 0 and 3)."""
    return {"x": _normal((cfg, li, 0), (layer.N, layer.C, layer.H, layer.W)),
            "dy": _normal((cfg, li, 3), (layer.N, layer.C, layer.P, layer.Q))}


def layer_inputs(cfg: int, li: int, layer: Layer | None = None, tensors=("x", "w", "b", "dy")):
    """Inputs of layer ``li`` of configuration ``cfg`` (optionally with a
    replaced Layer, e.g. a smaller batch: its arrays are then drawn at that
    batch from the same seeds)."""
    if layer is None:
        layer = CONFIGS[cfg][1][li]
    return make_inputs(layer.shape, layer.P, layer.Q, (cfg, li), layer.init, tensors)
