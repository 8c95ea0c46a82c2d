"""Parity over a fixed set of seeded random small shapes: every pass with the
built-in rule and with up to two more candidate plans drawn from the pass's
list, against the oracle (full tensors).  The shapes mix strides 1-4, padding
up to the larger filter side minus one (so at times past the smaller one),
1-4 groups, square and oblong filters and images, and channel counts on and
off multiples of 16, so that every tile, the blocked and phase backward-data
plans and the tap-uniform and packed backward-weight tiles meet ragged edges
they are not tuned for; inner-product shapes, some with batches that are
multiples of 16, cover the batch-transposed plans."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_within, dev, host

pytestmark = pytest.mark.gpu

PASSES = (0, 1, 2)


def _shapes(count=120, seed=1903):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        G = int(rng.choice([1, 1, 1, 2, 3, 4]))
        Cg = int(rng.choice([1, 3, 5, 8, 16, 17, 24, 32, 48]))
        Kg = int(rng.choice([3, 8, 16, 20, 32, 48, 64, 96]))
        R = int(rng.integers(1, 8))
        S = int(rng.choice([R, R, int(rng.integers(1, 8))]))
        st = int(rng.choice([1, 1, 2, 2, 3, 4]))
        pad = int(rng.integers(0, max(R, S)))
        H = int(rng.integers(max(R, S), 24))
        W = int(rng.integers(max(R, S), 24))
        N = int(rng.integers(1, 4))
        P = oracle.out_size(H, R, st, pad)
        Q = oracle.out_size(W, S, st, pad)
        if P < 1 or Q < 1 or pad >= 32767:
            continue
        out.append((N, Cg * G, H, W, Kg * G, R, S, st, pad, G))
    return out


def _wide_shapes(count=60, seed=3141):
    """Padding past the filter (windows wholly in the padding: outputs equal to
    the bias, no contribution to dx or dw) and images smaller than the filter
    that only the padding lets fit."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        G = int(rng.choice([1, 1, 2, 4]))
        Cg = int(rng.choice([1, 3, 16, 20, 32]))
        Kg = int(rng.choice([8, 16, 24, 64]))
        R = int(rng.integers(1, 8))
        S = int(rng.integers(1, 8))
        st = int(rng.integers(1, 5))
        pad = int(rng.integers(0, max(R, S) + 4))
        H = int(rng.integers(1, 20))
        W = int(rng.integers(1, 20))
        N = int(rng.integers(1, 4))
        if oracle.out_size(H, R, st, pad) < 1 or oracle.out_size(W, S, st, pad) < 1:
            continue
        out.append((N, Cg * G, H, W, Kg * G, R, S, st, pad, G))
    return out


def _fc_shapes(count=24, seed=2718):
    """Inner-product layers (1 x 1 images and filters) of ragged sizes: the
    batch-transposed plans with padded copies of w and dy."""
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, 300)), int(rng.integers(1, 600)), 1, 1, int(rng.integers(1, 300)),
             1, 1, 1, 0, 1) for _ in range(count)]


def _fc16_shapes(count=16, seed=1618):
    """Inner-product layers whose batch is a multiple of 16, where the
    backward-weight rule is one image GEMM over the batch (dw = dy^T x), with
    ragged input and output widths."""
    rng = np.random.default_rng(seed)
    return [(16 * int(rng.integers(1, 12)), int(rng.integers(1, 700)), 1, 1,
             int(rng.integers(1, 400)), 1, 1, 1, 0, 1) for _ in range(count)]


SHAPES = _shapes() + _wide_shapes() + _fc_shapes() + _fc16_shapes()


@pytest.fixture(autouse=True)
def _clean():
    import paper_1903_06934_amd as m
    m.plan_clear()
    yield
    m.plan_clear()


def _run(p, shape, t, ws):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    if p == 0:
        return [m.conv_fwd(t["x"], t["w"], t["b"], st, pad, G, ws=ws)]
    if p == 1:
        return [m.conv_bwd_data(t["dy"], t["w"], (H, W), st, pad, G, ws=ws)]
    return list(m.conv_bwd_weight(t["x"], t["dy"], (R, S), st, pad, G, ws=ws))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_random_shape_rule_and_two_candidates(shape):
    import torch
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = oracle.out_size(H, R, st, pad), oracle.out_size(W, S, st, pad)
    d = workloads.make_inputs(shape, P, Q, seed=(1903, sum(shape)), init="he")
    t = {k: dev(v) for k, v in d.items()}
    y_ref, ay = oracle.conv_fwd(shape, d["x"], d["w"], d["b"])
    dx_ref, adx = oracle.conv_bwd_data(shape, d["dy"], d["w"])
    dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    refs = {0: [(y_ref, ay)], 1: [(dx_ref, adx)], 2: [(dw_ref, adw), (db_ref, adb)]}
    rng = np.random.default_rng(list(shape))
    for p in PASSES:
        n = m.plan_count(p, shape)
        picks = sorted({0, int(rng.integers(n)), int(rng.integers(n))})
        for i in picks:
            m.plan_set(p, shape, i)
            nbytes = m.plan_workspace_size(p, shape, i)
            ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
            outs = [host(o) for o in _run(p, shape, t, ws)]
            name = m.plan_name(p, shape, i)
            for (ref, absum), got in zip(refs[p], outs):
                assert_within(got, ref, absum, f"pass {p} plan {i} ({name}) {shape}")
        m.plan_set(p, shape, 0)


@pytest.mark.parametrize("shape", _fc16_shapes(6, seed=1414), ids=lambda s: "x".join(map(str, s)))
def test_fc_batch16_every_weight_plan(shape):
    """Every backward-weight plan of an inner-product layer with a batch that
    is a multiple of 16: the image-GEMM plans over the batch and the
    batch-transposed split plans give the same dw and db as the oracle."""
    import torch
    import paper_1903_06934_amd as m
    d = workloads.make_inputs(shape, 1, 1, seed=(1414, sum(shape)), init="he")
    t = {k: dev(v) for k, v in d.items()}
    dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    names = []
    for i in range(m.plan_count(2, shape)):
        m.plan_set(2, shape, i)
        ws = torch.empty(max(m.plan_workspace_size(2, shape, i), 16), dtype=torch.uint8, device="cuda")
        dw, db = _run(2, shape, t, ws)
        name = m.plan_name(2, shape, i)
        names.append(name)
        assert_within(host(dw), dw_ref, adw, f"dw plan {i} ({name}) {shape}")
        assert_within(host(db), db_ref, adb, f"db plan {i} ({name}) {shape}")
    assert any("image GEMM" in n for n in names), names
