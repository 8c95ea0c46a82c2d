"""Launch-splitting paths at sizes where they occur, on sampled elements
against the oracle's gather forms:

* batch chunking: a batch whose input tensor exceeds 2^29 elements runs as
  several launches of whole images (here 2 + 1 images of 176 x 1024 x 1024);
* the explicit plan's column chunks: 256 MB of column tensor a chunk (here
  2 + 1 images of a 64-channel 224 x 224 layer), for each pass."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_within, dev, host, sample_indices

pytestmark = pytest.mark.gpu


def _gpu_all(shape, d, ws=None):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    y = host(m.conv_fwd(dev(d["x"]), dev(d["w"]), dev(d["b"]), st, pad, G))
    dx = host(m.conv_bwd_data(dev(d["dy"]), dev(d["w"]), (H, W), st, pad, G))
    dw, db = m.conv_bwd_weight(dev(d["x"]), dev(d["dy"]), (R, S), st, pad, G)
    return y, dx, host(dw), host(db)


def _check_sampled(shape, d, y, dx, dw, db, what, dw_count=256):
    N, C, H, W, K, R, S, st, pad, G = shape
    rng = np.random.default_rng(list(shape))
    idx = sample_indices(y.shape, rng, groups=G)
    v, a = oracle.conv_fwd_at(shape, d["x"], d["w"], d["b"], idx)
    assert_within(y.ravel()[idx], v, a, f"{what} fwd")
    idx = sample_indices(dx.shape, rng, groups=G)
    v, a = oracle.conv_bwd_data_at(shape, d["dy"], d["w"], idx)
    assert_within(dx.ravel()[idx], v, a, f"{what} bwd_data")
    idx = sample_indices(dw.shape, rng, count=dw_count, groups=1, channel_axis=0)
    v, a = oracle.conv_bwd_weight_at(shape, d["x"], d["dy"], idx)
    assert_within(dw.ravel()[idx], v, a, f"{what} bwd_weight")
    v, a = oracle.bias_grad(d["dy"])
    assert_within(db, v, a, f"{what} bias_grad")


def test_batch_chunking():
    shape = (3, 176, 1024, 1024, 16, 3, 3, 1, 1, 1)
    d = workloads.make_inputs(shape, 1024, 1024, seed=(90, 1), init="he")
    y, dx, dw, db = _gpu_all(shape, d)
    _check_sampled(shape, d, y, dx, dw, db, "chunked")


def test_explicit_plan_column_chunks():
    import paper_1903_06934_amd as m
    shape = (3, 64, 224, 224, 32, 3, 3, 1, 1, 1)
    d = workloads.make_inputs(shape, 224, 224, seed=(91, 1), init="he")
    try:
        for p in (m.PASS_FWD, m.PASS_BWD_DATA, m.PASS_BWD_WEIGHT):
            n = m.plan_count(p, shape)
            ex = [i for i in range(n) if m.plan_name(p, shape, i).startswith("explicit")]
            assert ex and "(2 images a chunk)" in m.plan_name(p, shape, ex[0])
            m.plan_set(p, shape, ex[0])
        y, dx, dw, db = _gpu_all(shape, d)
    finally:
        m.plan_clear()
    _check_sampled(shape, d, y, dx, dw, db, "explicit")
