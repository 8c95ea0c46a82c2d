"""The adjacent layers on the GPU against the oracle: pooling (Sec. IV-D)
forward and backward through pool_fwd / pool_bwd, and the inner-product
layer (Sec. IV-A) as the convolution with H = W = R = S = 1.

Max pooling is compared exactly (values and argmax masks; the oracle's
maximum of fp32 inputs is an fp32 value); average pooling and every
backward pass to the usual bar |gpu - ref| <= 1e-4 * sum|terms|."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_within, dev, gpu_bwd_data, gpu_bwd_weight, gpu_fwd, host

pytestmark = pytest.mark.gpu

POOL_CASES = [
    ("max", (4, 96, 55, 55, 3, 3, 2, 0)),    # AlexNet pool1 (batch 4)
    ("max", (4, 256, 27, 27, 3, 3, 2, 0)),   # AlexNet pool2
    ("max", (128, 256, 13, 13, 3, 3, 2, 0)), # AlexNet pool5, bench batch
    ("max", (2, 64, 224, 224, 2, 2, 2, 0)),  # VGG-16 pool1: the paper's non-overlapping tiles
    ("avg", (2, 8, 15, 15, 3, 3, 1, 1)),     # padded, stride 1
    ("max", (2, 8, 15, 15, 3, 3, 1, 1)),
    ("avg", (3, 5, 9, 10, 3, 3, 2, 1)),      # ceil-mode edge with padding
    ("max", (3, 5, 9, 10, 3, 3, 2, 1)),
    ("avg", (2, 3, 6, 5, 3, 3, 2, 0)),       # overhang past the edge
    ("max", (2, 3, 7, 7, 7, 7, 1, 0)),       # global
    ("avg", (2, 3, 7, 7, 7, 7, 1, 0)),
    ("max", (1, 2, 3, 3, 2, 2, 2, 1)),       # last window dropped (would start in padding)
    ("avg", (2, 4, 11, 13, 2, 3, 3, 1)),     # R != S, stride 3
]


def _pool_gpu(mode, pshape, x, dy):
    import paper_1903_06934_amd as m
    N, C, H, W, R, S, st, pad = pshape
    y, mask = m.pool_fwd(dev(x), (R, S), st, pad, mode)
    dx = m.pool_bwd(dev(dy), (H, W), (R, S), st, pad, mode, mask)
    return host(y), None if mask is None else host(mask), host(dx)


@pytest.mark.parametrize("mode,pshape", POOL_CASES, ids=lambda v: str(v))
def test_pool_matches_oracle(mode, pshape):
    N, C, H, W, R, S, st, pad = pshape
    rng = np.random.default_rng(list(pshape))
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    y_ref, ay, mask_ref = oracle.pool_fwd(mode, pshape, x)
    dy = rng.standard_normal(y_ref.shape).astype(np.float32)
    y, mask, dx = _pool_gpu(mode, pshape, x, dy)
    if mode == "max":
        assert np.array_equal(y.astype(np.float64), y_ref)
        assert np.array_equal(mask.astype(np.int64), mask_ref)
    else:
        assert_within(y, y_ref, ay, f"avg pool fwd {pshape}")
    dx_ref, adx = oracle.pool_bwd(mode, pshape, dy, mask_ref)
    assert_within(dx, dx_ref, adx, f"{mode} pool bwd {pshape}")
    # bitwise repeatable
    y2, mask2, dx2 = _pool_gpu(mode, pshape, x, dy)
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))
    assert np.array_equal(dx.view(np.uint32), dx2.view(np.uint32))


def _random_pool_cases(count=60, seed=1903, lo=0, hi=21):
    """Seeded random pooling shapes with planes of lo..hi-1 rows and columns
    (small planes go through the per-element kernels, planes of 512 to 12288
    elements through the whole-plane ones)."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        R = int(rng.integers(1, 6))
        S = int(rng.choice([R, int(rng.integers(1, 6))]))
        st = int(rng.integers(1, 5))
        pad = int(rng.integers(0, min(R, S)))
        H = int(rng.integers(max(R, S, lo), hi))
        W = int(rng.integers(max(R, S, lo), hi))
        if oracle.pool_out_size(H, R, st, pad) < 1 or oracle.pool_out_size(W, S, st, pad) < 1:
            continue  # a window past the image: refused (tested on the CPU)
        out.append(("max" if len(out) % 2 == 0 else "avg",
                    (int(rng.integers(1, 4)), int(rng.integers(1, 9)), H, W, R, S, st, pad)))
    return out


@pytest.mark.parametrize("mode,pshape", _random_pool_cases() +
                         _random_pool_cases(30, 2024, lo=23, hi=100), ids=lambda v: str(v))
def test_pool_random_shapes(mode, pshape):
    """Seeded random windows, strides, padding and plane sizes (ceil-mode
    edges, overhangs and dropped last windows among them)."""
    N, C, H, W, R, S, st, pad = pshape
    rng = np.random.default_rng(list(pshape) + [7])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    y_ref, ay, mask_ref = oracle.pool_fwd(mode, pshape, x)
    dy = rng.standard_normal(y_ref.shape).astype(np.float32)
    y, mask, dx = _pool_gpu(mode, pshape, x, dy)
    if mode == "max":
        assert np.array_equal(y.astype(np.float64), y_ref)
        assert np.array_equal(mask.astype(np.int64), mask_ref)
    else:
        assert_within(y, y_ref, ay, f"avg pool fwd {pshape}")
    dx_ref, adx = oracle.pool_bwd(mode, pshape, dy, mask_ref)
    assert_within(dx, dx_ref, adx, f"{mode} pool bwd {pshape}")


def test_max_pool_ties_take_the_first_element():
    """A constant plane: every window's argmax is its first element inside
    the image, in row-major order."""
    pshape = (1, 2, 7, 7, 3, 3, 2, 1)
    x = np.full((1, 2, 7, 7), 0.5, np.float32)
    _, _, mask_ref = oracle.pool_fwd("max", pshape, x)
    dy = np.ones(mask_ref.shape, np.float32)
    _, mask, _ = _pool_gpu("max", pshape, x, dy)
    assert np.array_equal(mask.astype(np.int64), mask_ref)
    assert mask_ref[0, 0, 0, 0] == 0 and mask_ref[0, 0, 1, 1] == 1 * 7 + 1


# The inner-product layer: y[n][o] = b[o] + sum_i W[o][i] x[n][i], i.e. the
# convolution of 1 x 1 images with 1 x 1 filters (AlexNet fc6 / fc7 / fc8).
FC_SHAPES = [
    (16, 9216, 1, 1, 4096, 1, 1, 1, 0, 1),
    (16, 4096, 1, 1, 4096, 1, 1, 1, 0, 1),
    (16, 4096, 1, 1, 1000, 1, 1, 1, 0, 1),
    (5, 300, 1, 1, 70, 1, 1, 1, 0, 1),   # ragged everywhere
]


@pytest.mark.parametrize("shape", FC_SHAPES, ids=lambda s: f"{s[1]}x{s[4]}")
def test_inner_product_matches_matmul_oracle(shape):
    N, C, _, _, K = shape[:5]
    d = workloads.make_inputs(shape, 1, 1, seed=(77, C), init="xavier")
    x, w, b, dy = d["x"], d["w"], d["b"], d["dy"]
    X, Wm, DY = (a.astype(np.float64).reshape(a.shape[0], -1) for a in (x, w, dy))
    y = gpu_fwd(shape, x, w, b).reshape(N, K)
    assert_within(y, X @ Wm.T + b.astype(np.float64), np.abs(X) @ np.abs(Wm).T + np.abs(b), "fc fwd")
    dx = gpu_bwd_data(shape, dy, w).reshape(N, C)
    assert_within(dx, DY @ Wm, np.abs(DY) @ np.abs(Wm), "fc bwd_data")
    dw, db = gpu_bwd_weight(shape, x, dy)
    assert_within(dw.reshape(K, C), DY.T @ X, np.abs(DY).T @ np.abs(X), "fc bwd_weight")
    assert_within(db, DY.sum(0), np.abs(DY).sum(0), "fc bias grad")
