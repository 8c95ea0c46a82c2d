"""Pins of the oracle's pooling layer (Sec. IV-D) against values the
definition fixes independently of the oracle's own loops: hand-worked
examples, closed forms for constant inputs, global pooling as numpy's
max / mean, the adjoint identity of average pooling, mass conservation and
finite differences of max pooling, and the configurations' stated extents.

Each pin takes an oracle build, so that tests/test_oracle_mutants.py can run
them against copies with planted mistakes (POOL_CHECKS)."""
import numpy as np
import pytest

import oracle

SIZES = [
    (55, 3, 2, 0, 27), (27, 3, 2, 0, 13), (13, 3, 2, 0, 6),   # AlexNet pool1 / pool2 / pool5
    (224, 2, 2, 0, 112), (14, 2, 2, 0, 7),                    # VGG-16 pools
    (112, 3, 2, 0, 56),                                       # ResNet-50 stem pool (Caffe: no pad)
    (6, 3, 2, 0, 3),    # ceil: the last window hangs over the edge
    (3, 2, 2, 1, 2),    # ceil gives 3, but that window would start in the padding
    (4, 4, 4, 0, 1),    # one non-overlapping tile
]

POOL_SHAPES = [
    (2, 3, 13, 13, 3, 3, 2, 0),   # AlexNet-style overlapping
    (2, 2, 12, 11, 2, 2, 2, 0),   # non-overlapping tiles, odd width
    (1, 2, 9, 10, 3, 3, 2, 1),    # padded, ceil-mode edge
    (2, 1, 7, 6, 3, 2, 1, 1),     # stride 1, R != S
    (1, 2, 5, 5, 3, 3, 3, 2),     # stride 3, pad 2
]


def _x(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def pin_pool_out_size(o):
    for n_in, f, st, pad, want in SIZES:
        assert o.pool_out_size(n_in, f, st, pad) == want, (n_in, f, st, pad)


def pin_every_window_holds_an_element(o):
    """Every window of an accepted extent holds at least one image element
    (brute force over small extents); without padding and with a stride
    above the window the ceil rule can put its last window past the image,
    and such an extent is refused (0): 10 elements, window 1, stride 2 would
    be 6 windows, the sixth starting at 10."""
    for n in range(1, 13):
        for f in range(1, min(n, 5) + 1):
            for st in range(1, 6):
                for pad in range(f):
                    for p in range(o.pool_out_size(n, f, st, pad)):
                        start = p * st - pad
                        assert min(start + f, n) > max(start, 0), (n, f, st, pad, p)
    assert o.pool_out_size(10, 1, 2, 0) == 0
    assert o.pool_out_size(18, 1, 4, 0) == 0
    assert o.pool_out_size(9, 1, 2, 0) == 5     # windows at 0, 2, 4, 6, 8
    assert o.pool_out_size(10, 3, 4, 0) == 3    # windows at 0, 4, 8 (the last one overhangs)


def pin_max_hand_example(o):
    """Non-overlapping 2 x 2 tiles (the paper's case) of a 4 x 4 plane."""
    x = np.array([[1, 5, 2, 0],
                  [3, 4, 8, 8],
                  [0, -1, -3, -2],
                  [-1, 7, -4, -5]], np.float32).reshape(1, 1, 4, 4)
    y, _, mask = o.pool_fwd("max", (1, 1, 4, 4, 2, 2, 2, 0), x)
    assert y.reshape(2, 2).tolist() == [[5, 8], [7, -2]]
    # argmax: first maximum in row-major order (the tie 8/8 keeps (1, 2))
    assert mask.reshape(2, 2).tolist() == [[1, 6], [13, 11]]
    dy = np.array([10, 20, 30, 40], np.float32).reshape(1, 1, 2, 2)
    dx, _ = o.pool_bwd("max", (1, 1, 4, 4, 2, 2, 2, 0), dy, mask)
    want = np.zeros(16)
    want[[1, 6, 13, 11]] = [10, 20, 30, 40]
    assert dx.ravel().tolist() == want.tolist()


def pin_avg_constant_with_padding(o):
    """3 x 3 windows, stride 1, pad 1 on a 3 x 3 plane of ones: padding counts
    in the divisor, so a corner sees 4/9, an edge 6/9, the centre 9/9."""
    x = np.ones((1, 1, 3, 3), np.float32)
    y, _, _ = o.pool_fwd("avg", (1, 1, 3, 3, 3, 3, 1, 1), x)
    want = np.array([[4, 6, 4], [6, 9, 6], [4, 6, 4]]) / 9.0
    assert np.allclose(y.reshape(3, 3), want, rtol=0, atol=1e-15)


def pin_avg_overhang_does_not_count(o):
    """6 wide, window 3, stride 2, no padding: the third window covers columns
    4, 5 and one past the edge, and averages over its two columns only."""
    x = np.arange(6, dtype=np.float32).reshape(1, 1, 1, 6)
    y, _, _ = o.pool_fwd("avg", (1, 1, 1, 6, 1, 3, 2, 0), x)
    assert y.ravel().tolist() == [1.0, 3.0, 4.5]


def pin_global_pooling_is_numpy_reduction(o):
    x = _x((2, 3, 7, 5), 1)
    for mode in ("max", "avg"):
        y, _, _ = o.pool_fwd(mode, (2, 3, 7, 5, 7, 5, 1, 0), x)
        ref = x.astype(np.float64).max(axis=(2, 3)) if mode == "max" else \
            x.astype(np.float64).mean(axis=(2, 3))
        assert np.allclose(y.reshape(2, 3), ref, rtol=1e-14, atol=0)


def pin_avg_adjoint(o):
    """Average pooling is linear: <pool(x), dy> = <x, pool_bwd(dy)>."""
    for pshape in POOL_SHAPES:
        x = _x(pshape[:4], 2).astype(np.float64)
        y, _, _ = o.pool_fwd("avg", pshape, x)
        dy = _x(y.shape, 3).astype(np.float64)
        dx, _ = o.pool_bwd("avg", pshape, dy)
        lhs, rhs = float((y * dy).sum()), float((x * dx).sum())
        assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + abs(rhs) + 1), pshape


def pin_max_mask_mass_and_finite_differences(o):
    for pshape in POOL_SHAPES:
        x = _x(pshape[:4], 4)
        y, _, mask = o.pool_fwd("max", pshape, x)
        N, C, H, W = pshape[:4]
        planes = x.reshape(N * C, H * W).astype(np.float64)
        assert np.array_equal(
            np.take_along_axis(planes, mask.reshape(N * C, -1), 1).ravel(), y.ravel())
        dy = _x(y.shape, 5).astype(np.float64)
        dx, _ = o.pool_bwd("max", pshape, dy, mask)
        assert abs(dx.sum() - dy.sum()) <= 1e-12 * np.abs(dy).sum()
        # d/dx_i of sum(y * dy) by central differences (no ties in random data)
        rng = np.random.default_rng(6)
        xd = x.astype(np.float64)
        for i in rng.choice(x.size, size=min(40, x.size), replace=False):
            e = np.zeros(x.size)
            e[i] = 1e-6
            yp, _, _ = o.pool_fwd("max", pshape, (xd.ravel() + e).reshape(x.shape))
            ym, _, _ = o.pool_fwd("max", pshape, (xd.ravel() - e).reshape(x.shape))
            fd = ((yp - ym) * dy).sum() / 2e-6
            assert abs(fd - dx.ravel()[i]) <= 1e-6 * (1 + abs(dx.ravel()[i]))


def pin_avg_finite_differences(o):
    pshape = (1, 2, 9, 10, 3, 3, 2, 1)
    x = _x(pshape[:4], 7).astype(np.float64)
    y, _, _ = o.pool_fwd("avg", pshape, x)
    dy = _x(y.shape, 8).astype(np.float64)
    dx, _ = o.pool_bwd("avg", pshape, dy)
    for i in (0, 7, 33, 99, 179):
        e = np.zeros(x.size)
        e[i] = 1e-3
        yp, _, _ = o.pool_fwd("avg", pshape, (x.ravel() + e).reshape(x.shape))
        fd = ((yp - y) * dy).sum() / 1e-3
        assert abs(fd - dx.ravel()[i]) <= 1e-9 * (1 + abs(fd))


POOL_CHECKS = [pin_pool_out_size, pin_every_window_holds_an_element, pin_max_hand_example, pin_avg_constant_with_padding,
               pin_avg_overhang_does_not_count, pin_global_pooling_is_numpy_reduction,
               pin_avg_adjoint, pin_max_mask_mass_and_finite_differences,
               pin_avg_finite_differences]


@pytest.mark.parametrize("check", POOL_CHECKS, ids=lambda c: c.__name__)
def test_pool_pin(check):
    check(oracle.default())
