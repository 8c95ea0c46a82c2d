"""Parity of the HIP passes (through the C ABI) with the CPU oracle.

Bar: every element within 1e-4 * sum|products| of the oracle's fp64 value;
elements with no product (uncovered input pixels in dx) exactly 0.
Full tensors at sizes the oracle finishes in seconds (several tiles and
ragged tails; every layer of every configuration at batch 2); sampled
elements at the configurations' full batch, in the launch configuration the
benchmark times."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import (assert_within, dev, dw_indices, gpu_bwd_data, gpu_bwd_weight, gpu_fwd,
                      sample_indices)
from oracle_pins import SMALL_SHAPES

pytestmark = pytest.mark.gpu


def _inputs(shape, seed, init="he"):
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = oracle.out_size(H, R, st, pad), oracle.out_size(W, S, st, pad)
    return workloads.make_inputs(shape, P, Q, seed=seed, init=init)


def full_parity(shape, seed=(99, 0), init="he", bias=True):
    d = _inputs(shape, seed, init)
    x, w, b, dy = d["x"], d["w"], d["b"] if bias else None, d["dy"]
    y_ref, ay = oracle.conv_fwd(shape, x, w, b)
    assert_within(gpu_fwd(shape, x, w, b), y_ref, ay, f"fwd {shape}")
    dx_ref, adx = oracle.conv_bwd_data(shape, dy, w)
    assert_within(gpu_bwd_data(shape, dy, w), dx_ref, adx, f"bwd_data {shape}")
    dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, x, dy)
    dw, db = gpu_bwd_weight(shape, x, dy)
    assert_within(dw, dw_ref, adw, f"bwd_weight {shape}")
    assert_within(db, db_ref, adb, f"bias_grad {shape}")


def test_tiny_config_all_passes():
    """The single-layer configuration (N=2, C=16, 32x32, K=32, 3x3 s1 p1)."""
    L = workloads.config(0)[1][0]
    d = workloads.layer_inputs(0, 0)
    shape = L.shape
    y_ref, ay = oracle.conv_fwd(shape, d["x"], d["w"], d["b"])
    assert_within(gpu_fwd(shape, d["x"], d["w"], d["b"]), y_ref, ay, "fwd")
    dx_ref, adx = oracle.conv_bwd_data(shape, d["dy"], d["w"])
    assert_within(gpu_bwd_data(shape, d["dy"], d["w"]), dx_ref, adx, "bwd_data")
    dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    dw, db = gpu_bwd_weight(shape, d["x"], d["dy"])
    assert_within(dw, dw_ref, adw, "bwd_weight")
    assert_within(db, db_ref, adb, "bias_grad")


EDGE_SHAPES = SMALL_SHAPES + [
    (3, 5, 7, 9, 7, 3, 3, 1, 1, 1),        # odd C, K
    (2, 6, 8, 8, 6, 3, 3, 1, 1, 6),        # depthwise (C/G = 1)
    (1, 4, 6, 6, 1, 3, 3, 1, 1, 1),        # K = 1
    (2, 8, 5, 5, 4, 5, 5, 1, 0, 1),        # P = Q = 1 (fully connected)
    (1, 3, 5, 5, 2, 2, 2, 1, 3, 1),        # pad >= R
    (2, 4, 9, 9, 4, 1, 1, 3, 0, 1),        # stride > R: uncovered dx pixels
    (2, 3, 31, 31, 8, 11, 11, 4, 0, 1),    # 11x11 stride 4
    (2, 3, 32, 32, 16, 7, 7, 2, 3, 1),     # 7x7 stride 2 pad 3
    (2, 16, 14, 14, 32, 1, 1, 2, 0, 1),    # 1x1 stride 2
    (2, 32, 10, 10, 48, 3, 3, 2, 1, 2),    # stride 2, groups, K/G = 24
    (2, 64, 9, 9, 64, 3, 3, 3, 2, 1),      # stride 3, channel-aligned slices
    (2, 48, 12, 12, 32, 5, 5, 4, 2, 1),    # stride 4 pad 2
    (1, 17, 13, 11, 19, 4, 2, 2, 1, 1),    # R != S, all odd
    (2, 32, 20, 20, 32, 3, 3, 1, 1, 1),    # channel-aligned, several tiles
    (1, 1, 1, 1, 1, 1, 1, 1, 0, 1),        # smallest layer
    (2, 16, 3, 3, 16, 3, 3, 1, 2, 1),      # map smaller than the filter span
    (2, 4, 1, 1, 3, 1, 1, 3, 1, 1),        # 1x1 image, padded: reads only padding
    (16, 8, 1, 1, 32, 1, 1, 5, 2, 1),      # the same with a batch of 16s
]


@pytest.mark.parametrize("shape", EDGE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_edge_shapes(shape):
    full_parity(shape)


# Shapes for each image-GEMM tile: 128x64 and 96x128 need at least 1024
# tiles (128x64 also 128-row multiples); the others cover ragged rows and
# columns.
TILE_SHAPES = [
    (16, 32, 65, 63, 128, 3, 3, 1, 1, 1),  # fwd 128x64, ragged columns
    (16, 128, 63, 65, 16, 3, 3, 1, 1, 1),  # bwd-data 128x64, ragged columns
    (8, 32, 64, 64, 200, 3, 3, 1, 1, 1),   # fwd 64x64, channel-aligned, ragged M
    (8, 3, 128, 128, 96, 3, 3, 1, 1, 1),   # fwd 96x128, per-element tap decode
    (33, 48, 64, 63, 16, 3, 3, 1, 1, 1),   # bwd-data 48x64 (three waves), ragged columns
    # Narrow-row tiles (16, 32, 48 and 96 rows), with ragged rows and columns.
    (4, 64, 20, 20, 80, 3, 3, 1, 1, 1),    # fwd M = 80 (96x64)
    (4, 80, 21, 21, 40, 3, 3, 1, 1, 1),    # fwd M = 40 (48), bwd-data M = 80, tap decode
    (4, 32, 24, 24, 12, 3, 3, 1, 1, 1),    # fwd M = 12 (16), bwd-data M = 32, tap decode
    (4, 96, 15, 15, 64, 5, 5, 1, 2, 2),    # bwd-data M = 48 over groups
    (3, 48, 11, 11, 96, 5, 5, 2, 2, 1),    # bwd-data M = 48, stride phases
]


@pytest.mark.parametrize("shape", TILE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_large_tile_paths(shape):
    full_parity(shape)


# 1x1 stride-1 layers (and the first stride phase of a 1x1 stride-2 layer's
# backward-data) whose pixels per image are a multiple of 4 and whose
# channels per group are a multiple of 16 run the image GEMM's direct 1x1
# variant (16-byte staging loads) on its 64-column tiles: each such row tile
# class, groups, ragged column tails, a split reduction; and 7 x 7 maps
# (49 pixels) that keep the one-dword gather.
ONE_BY_ONE_SHAPES = [
    (2, 32, 14, 14, 48, 1, 1, 1, 0, 1),    # 196 pixels, M = 48 (three waves), ragged columns
    (3, 64, 6, 10, 80, 1, 1, 1, 0, 1),     # M = 80 (96-row tile), bwd-data M = 64
    (2, 128, 8, 8, 256, 1, 1, 1, 0, 1),    # M = 256 (128x64), bwd-data M = 128
    (3, 64, 12, 12, 32, 1, 1, 1, 0, 2),    # groups, M = 16 / 32 per group
    (2, 64, 28, 28, 32, 1, 1, 2, 0, 1),    # stride 2: bwd-data phase (0, 0) is direct
    (1, 3072, 4, 4, 64, 1, 1, 1, 0, 1),    # one tile, deep reduction: split
    (2, 32, 7, 7, 32, 1, 1, 1, 0, 1),      # 49 pixels: the gather path
]


@pytest.mark.parametrize("shape", ONE_BY_ONE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_one_by_one_direct(shape):
    full_parity(shape)


# Backward-data with few input channels: the blocked plan (b x b input pixels
# of a block as GEMM rows, b = stride * f).  Many edge shapes above take it
# too; these add each row-tile class and several column tiles.
BLOCK_SHAPES = [
    (3, 4, 37, 35, 32, 8, 8, 4, 2, 1),     # b = 4, 64 rows, channel-aligned reduction
    (2, 6, 33, 30, 24, 5, 5, 2, 2, 2),     # groups, 12 rows, K/G = 12 (tap decode)
    (4, 3, 67, 61, 32, 5, 5, 2, 1, 1),     # 12 rows (shared-A tile), many column tiles
    (2, 3, 45, 43, 48, 3, 3, 1, 1, 1),     # stride 1 in 2 x 2 blocks
    (2, 5, 30, 29, 20, 6, 4, 3, 7, 1),     # 45 rows, pad > b, R != S, tap decode
]


@pytest.mark.parametrize("shape", BLOCK_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_bwd_data_blocked(shape):
    d = _inputs(shape, (7, 1))
    dx_ref, adx = oracle.conv_bwd_data(shape, d["dy"], d["w"])
    assert_within(gpu_bwd_data(shape, d["dy"], d["w"]), dx_ref, adx, f"bwd_data {shape}")


def _all_layers():
    out = []
    for cfg in (1, 2, 3, 4):
        name, layers = workloads.config(cfg)
        for li, L in enumerate(layers):
            out.append(pytest.param(cfg, li, id=f"{name}-{L.name}"))
    return out


@pytest.mark.parametrize("cfg,li", _all_layers())
def test_config_layer_batch2(cfg, li):
    """Every layer of every configuration, full tensors, at batch 2."""
    L = workloads.config(cfg)[1][li].with_batch(2)
    d = workloads.layer_inputs(cfg, li, L)
    shape = L.shape
    y_ref, ay = oracle.conv_fwd(shape, d["x"], d["w"], d["b"])
    assert_within(gpu_fwd(shape, d["x"], d["w"], d["b"]), y_ref, ay, "fwd")
    dx_ref, adx = oracle.conv_bwd_data(shape, d["dy"], d["w"])
    assert_within(gpu_bwd_data(shape, d["dy"], d["w"]), dx_ref, adx, "bwd_data")
    dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    dw, db = gpu_bwd_weight(shape, d["x"], d["dy"])
    assert_within(dw, dw_ref, adw, "bwd_weight")
    assert_within(db, db_ref, adb, "bias_grad")


@pytest.mark.parametrize("cfg,li", _all_layers())
def test_config_layer_full_batch_sampled(cfg, li):
    """Every layer at its configured batch, in the benchmark's launch
    configuration; sampled elements against the oracle's gather forms."""
    L = workloads.config(cfg)[1][li]
    d = workloads.layer_inputs(cfg, li)
    shape = L.shape
    N, C, H, W, K, R, S, st, pad, G = shape
    rng = np.random.default_rng([cfg, li])
    y = gpu_fwd(shape, d["x"], d["w"], d["b"])
    idx = sample_indices(y.shape, rng, groups=G)
    v, a = oracle.conv_fwd_at(shape, d["x"], d["w"], d["b"], idx)
    assert_within(y.ravel()[idx], v, a, "fwd")
    del y
    dx = gpu_bwd_data(shape, d["dy"], d["w"])
    idx = sample_indices(dx.shape, rng, groups=G)
    v, a = oracle.conv_bwd_data_at(shape, d["dy"], d["w"], idx)
    assert_within(dx.ravel()[idx], v, a, "bwd_data")
    del dx
    dw, db = gpu_bwd_weight(shape, d["x"], d["dy"])
    idx = dw_indices(dw.shape, N * L.P * L.Q, rng)  # every element when |dw| <= 64k
    v, a = oracle.conv_bwd_weight_at(shape, d["x"], d["dy"], idx)
    assert_within(dw.ravel()[idx], v, a, "bwd_weight")
    v, a = oracle.bias_grad(d["dy"])
    assert_within(db, v, a, "bias_grad")


def test_delta_filter_is_exact():
    """One unit tap per filter: y is a shifted copy of x and dx a shifted
    copy of dy, bit for bit (a single product reaches each element)."""
    for shape, tap in (((2, 32, 12, 13, 32, 3, 3, 1, 1, 1), (2, 0)),
                       ((2, 5, 12, 13, 7, 5, 3, 2, 2, 1), (1, 2))):
        N, C, H, W, K, R, S, st, pad, G = shape
        d = _inputs(shape, (98, 1))
        w = np.zeros((K, C, R, S), np.float32)
        for k in range(K):
            w[k, (3 * k + 1) % C, tap[0], tap[1]] = 1.0
        y_ref, _ = oracle.conv_fwd(shape, d["x"], w, None)
        assert np.array_equal(gpu_fwd(shape, d["x"], w, None), y_ref.astype(np.float32))
        if K <= C:  # every dx pixel gets at most one product
            dx_ref, _ = oracle.conv_bwd_data(shape, d["dy"], w)
            assert np.array_equal(gpu_bwd_data(shape, d["dy"], w), dx_ref.astype(np.float32))


def test_bitwise_repeatable():
    """Each pass run twice on the same inputs gives identical bits."""
    for shape in ((4, 64, 28, 28, 128, 3, 3, 1, 1, 1), (2, 3, 31, 31, 8, 11, 11, 4, 0, 1),
                  (8, 32, 64, 64, 200, 3, 3, 1, 1, 1)):
        d = _inputs(shape, (97, 2))
        assert np.array_equal(gpu_fwd(shape, d["x"], d["w"], d["b"]),
                              gpu_fwd(shape, d["x"], d["w"], d["b"]))
        assert np.array_equal(gpu_bwd_data(shape, d["dy"], d["w"]),
                              gpu_bwd_data(shape, d["dy"], d["w"]))
        a = gpu_bwd_weight(shape, d["x"], d["dy"])
        b = gpu_bwd_weight(shape, d["x"], d["dy"])
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_same_sign_stress():
    """All-positive x and dy (no cancellation): the fp32 accumulation error
    grows fastest here; it must still meet the bound on a long reduction."""
    shape = (8, 64, 56, 56, 64, 3, 3, 1, 1, 1)
    d = _inputs(shape, (96, 3))
    x, dy, w = np.abs(d["x"]), np.abs(d["dy"]), np.abs(d["w"])
    rng = np.random.default_rng(3)
    y = gpu_fwd(shape, x, w, None)
    idx = sample_indices(y.shape, rng)
    v, a = oracle.conv_fwd_at(shape, x, w, None, idx)
    assert_within(y.ravel()[idx], v, a, "fwd")
    dw, db = gpu_bwd_weight(shape, x, dy)
    v, a = oracle.conv_bwd_weight_at(shape, x, dy, np.arange(dw.size))
    assert_within(dw.ravel(), v, a, "bwd_weight")
    v, a = oracle.bias_grad(dy)
    assert_within(db, v, a, "bias_grad")


def test_no_bias_and_no_db():
    shape = (2, 16, 9, 9, 24, 3, 3, 1, 1, 1)
    d = _inputs(shape, (95, 4))
    y_ref, ay = oracle.conv_fwd(shape, d["x"], d["w"], None)
    assert_within(gpu_fwd(shape, d["x"], d["w"], None), y_ref, ay, "fwd no bias")
    dw_ref, adw, _, _ = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    dw, db = gpu_bwd_weight(shape, d["x"], d["dy"], with_bias=False)
    assert db is None
    assert_within(dw, dw_ref, adw, "bwd_weight no db")


def test_failed_call_writes_nothing():
    """On the device too, a call that reports an error has launched nothing:
    outputs filled with a sentinel keep it (workspace too small, an output
    overlapping an input, a misaligned pointer)."""
    import torch
    import paper_1903_06934_amd as m
    L = m.lib()
    shape = (2, 32, 12, 12, 48, 3, 3, 1, 1, 1)
    N, C, H, W, K, R, S, st, pad, G = shape
    d = _inputs(shape, (96, 0))
    x, w, b, dy = (dev(d[k]) for k in ("x", "w", "b", "dy"))
    y = torch.full((N, K, 12, 12), 7.0, device="cuda")
    dx = torch.full((N, C, H, W), 7.0, device="cuda")
    dw = torch.full((K, C, R, S), 7.0, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    need = [m.plan_workspace_size(p, shape, m.plan_get(p, shape)) for p in (0, 1, 2)]
    ws = torch.empty(max(need) + 64, dtype=torch.uint8, device="cuda")
    p = lambda t: t.data_ptr()  # noqa: E731
    small = [max(n - 1, 0) for n in need]
    if need[0]:
        assert L.conv_fwd(*shape, p(x), p(w), p(b), p(y), p(ws), small[0], stream) == -3
    assert L.conv_fwd(*shape, p(x), p(w), p(b), p(x), p(ws), need[0], stream) == -4
    assert L.conv_bwd_data(*shape, p(dy), p(w), p(dx) + 4, p(ws), need[1], stream) == -5
    if need[2]:
        assert L.conv_bwd_weight(*shape, p(x), p(dy), p(dw), None, p(ws), small[2],
                                 stream) == -3
    torch.cuda.synchronize()
    for t in (y, dx, dw):
        assert bool((t == 7.0).all())
