"""conv_bwd_weight_noalloc: the backward-weight pass with its workspace in
the library's fixed device scratch array, for callers that cannot allocate.
Through the C ABI, two calls in a row (the second on a smaller layer) must
give the bits conv_bwd_weight gives with a caller workspace, and both must
meet the oracle bar; a plan that needs more than the array is refused before
anything is written."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_within, dev, host

pytestmark = pytest.mark.gpu

SCRATCH_ERR = -11


def _inputs(shape, seed):
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = oracle.out_size(H, R, st, pad), oracle.out_size(W, S, st, pad)
    return workloads.make_inputs(shape, P, Q, seed=seed, init="he"), P, Q


def _both(shape, d):
    """(dw, db) from conv_bwd_weight_noalloc, then from conv_bwd_weight."""
    import torch
    import paper_1903_06934_amd as m
    L = m.lib()
    N, C, H, W, K, R, S, st, pad, G = shape
    x, dy = dev(d["x"]), dev(d["dy"])
    stream = torch.cuda.current_stream().cuda_stream
    dw0 = torch.full((K, C // G, R, S), 7.0, device="cuda")
    db0 = torch.full((K,), 7.0, device="cuda")
    st0 = L.conv_bwd_weight_noalloc(*shape, x.data_ptr(), dy.data_ptr(), dw0.data_ptr(),
                                    db0.data_ptr(), stream)
    assert st0 == 0, m.MiconvError(st0, "conv_bwd_weight_noalloc")
    ref = host(dw0), host(db0)  # synchronises: the scratch is free again
    dw1, db1 = m.conv_bwd_weight(x, dy, (R, S), st, pad, G)
    return ref, (host(dw1), host(db1))


@pytest.fixture(autouse=True)
def _clean():
    import paper_1903_06934_amd as m
    m.plan_clear()
    yield
    m.plan_clear()


def test_two_calls_match_the_workspace_entry_point():
    import paper_1903_06934_amd as m
    # A layer with split partials and tap-ordered reduction (AlexNet conv2,
    # two groups, batch 16), then a smaller one (the single-layer config).
    big = workloads.config(1)[1][1].with_batch(16)
    small = workloads.config(0)[1][0]
    for L, seed in ((big, (61, 1)), (small, (61, 2))):
        shape = L.shape
        d, P, Q = _inputs(shape, seed)
        need = m.plan_workspace_size(m.PASS_BWD_WEIGHT, shape, 0)
        assert 0 < need <= (96 << 20)
        (dw, db), (dw_ws, db_ws) = _both(shape, d)
        assert np.array_equal(dw.view(np.uint32), dw_ws.view(np.uint32)), L.name
        assert np.array_equal(db.view(np.uint32), db_ws.view(np.uint32)), L.name
        dw_ref, adw, db_ref, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
        assert_within(dw, dw_ref, adw, f"noalloc dw {shape}")
        assert_within(db, db_ref, adb, f"noalloc db {shape}")


def test_stored_plan_and_no_bias():
    """With a stored (non-rule) plan and db = NULL the variant runs that plan."""
    import torch
    import paper_1903_06934_amd as m
    L = m.lib()
    shape = (4, 64, 14, 14, 96, 3, 3, 1, 1, 1)
    N, C, H, W, K, R, S, st, pad, G = shape
    d, P, Q = _inputs(shape, (62, 0))
    n = m.plan_count(m.PASS_BWD_WEIGHT, shape)
    fits = [i for i in range(1, n)
            if 0 < m.plan_workspace_size(m.PASS_BWD_WEIGHT, shape, i) <= (96 << 20)]
    assert fits
    m.plan_set(m.PASS_BWD_WEIGHT, shape, fits[-1])
    x, dy = dev(d["x"]), dev(d["dy"])
    dw0 = torch.empty((K, C, R, S), device="cuda")
    assert L.conv_bwd_weight_noalloc(*shape, x.data_ptr(), dy.data_ptr(), dw0.data_ptr(), None,
                                     torch.cuda.current_stream().cuda_stream) == 0
    got = host(dw0)
    dw1, _ = m.conv_bwd_weight(x, dy, (R, S), st, pad, G, with_bias=False)
    assert np.array_equal(got.view(np.uint32), host(dw1).view(np.uint32))
    dw_ref, adw, _, _ = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    assert_within(got, dw_ref, adw, "noalloc dw, stored plan")


def test_plan_beyond_the_scratch_is_refused():
    """A plan whose workspace exceeds the array: MICONV_ERR_SCRATCH, and the
    outputs keep their contents."""
    import torch
    import paper_1903_06934_amd as m
    L = m.lib()
    shape = (32, 512, 28, 28, 512, 3, 3, 1, 1, 1)  # VGG conv4_2: 72 MB rule plan
    n = m.plan_count(m.PASS_BWD_WEIGHT, shape)
    big = [i for i in range(n) if m.plan_workspace_size(m.PASS_BWD_WEIGHT, shape, i) > (96 << 20)]
    assert big
    m.plan_set(m.PASS_BWD_WEIGHT, shape, big[0])
    x = torch.zeros(64, device="cuda")  # never read: the call is refused first
    dw = torch.full((16,), 7.0, device="cuda")
    assert L.conv_bwd_weight_noalloc(*shape, x.data_ptr(), x.data_ptr(), dw.data_ptr(), None,
                                     torch.cuda.current_stream().cuda_stream) == SCRATCH_ERR
    torch.cuda.synchronize()
    assert bool((dw == 7.0).all())
