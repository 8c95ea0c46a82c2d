"""Every candidate plan of every pass against the oracle, and tuning.

Each candidate (tile, split of the reduction, stride phases or pixel blocks)
is selected with conv_plan_set and run through the C ABI on the same seeded
inputs; all must meet the parity bar.  conv_tune must store a candidate,
leave that candidate's result in the outputs, and later calls must repeat it
bitwise."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_within, dev, host

pytestmark = pytest.mark.gpu

PLAN_SHAPES = [
    (2, 64, 12, 12, 32, 5, 5, 1, 2, 1),    # forward split candidates
    (2, 32, 12, 12, 96, 5, 5, 1, 2, 1),    # backward-data split candidates
    (2, 3, 35, 33, 24, 11, 11, 4, 2, 1),   # blocked backward-data, f = 1 and 2
    (2, 6, 17, 16, 16, 3, 3, 1, 1, 2),     # groups, stride 1 blocks, tap decode
    (3, 48, 11, 11, 40, 3, 3, 2, 1, 2),    # stride phases with groups
    (4, 64, 1, 1, 48, 1, 1, 1, 0, 1),      # inner product, channel-aligned (w read in place)
    (5, 300, 1, 1, 70, 1, 1, 1, 0, 1),     # inner product, ragged (w and dy padded copies)
    (32, 200, 1, 1, 72, 1, 1, 1, 0, 1),    # inner product, batch of 16s: dW as an image GEMM
    (8, 1024, 1, 1, 100, 1, 1, 1, 0, 1),   # inner product, forward fine splits
    (8, 100, 1, 1, 1024, 1, 1, 1, 0, 1),   # inner product, backward-data fine splits
    (2, 64, 12, 12, 48, 1, 1, 1, 0, 1),    # 1x1 direct GEMM on every 64-column tile
    # Halo GEMM (stride-1 3x3, channel-aligned): each pixel block width, padding
    # 0-2, groups, ragged rows and columns, split channel blocks.
    (2, 32, 10, 20, 48, 3, 3, 1, 1, 1),    # 28 x 4 blocks, 16-byte halo loads
    (2, 16, 6, 9, 32, 3, 3, 1, 1, 1),      # 14 x 8 blocks, one-word loads (width 9)
    (1, 32, 2, 100, 128, 3, 3, 1, 1, 1),   # 112 x 1 blocks, 100 of 112 columns used
    (2, 16, 5, 116, 32, 3, 3, 1, 1, 1),    # 56 x 2 blocks, three segments a row
    (1, 64, 7, 7, 64, 3, 3, 1, 1, 2),      # groups, 7 x 7 maps
    (2, 16, 9, 12, 16, 3, 3, 1, 2, 1),     # pad 2
    (2, 16, 8, 12, 16, 3, 3, 1, 0, 1),     # pad 0
    (1, 256, 6, 6, 128, 3, 3, 1, 1, 1),    # few tiles, 16 channel blocks: split
    # Halo GEMM of 5x5 layers (one-word loads, 28- and 14-wide blocks): a
    # 27-wide map with groups and 48 channels per group (the backward-data
    # phase's 48 rows leave the 64-row tile's last wave idle), padding 0, 1
    # and 3, 14-wide maps.  The first two shapes above are 5x5 too.
    (2, 96, 27, 27, 128, 5, 5, 1, 2, 2),
    (2, 16, 10, 30, 32, 5, 5, 1, 1, 1),
    (1, 32, 9, 18, 16, 5, 5, 1, 0, 1),
    (1, 16, 7, 7, 32, 5, 5, 1, 3, 1),
    (2, 48, 14, 14, 128, 5, 5, 1, 2, 1),
    # Split reductions of 2^18 elements or more (their 16-byte form): dw of
    # 128 x 256 x 9 over split pixels, split-K y of 8 x 128 x 256.
    (8, 256, 16, 16, 128, 3, 3, 1, 1, 1),
    # Halo backward-weight (stride-1 3x3, dy and x rows multiples of 4 wide):
    # filters not a multiple of 64, pad 3.
    (2, 32, 6, 28, 80, 3, 3, 1, 1, 1),
    (1, 16, 4, 8, 16, 3, 3, 1, 3, 1),
    (2, 64, 6, 12, 48, 3, 3, 1, 1, 2),     # two 16-channel sub-tiles a workgroup, groups
    (2, 32, 14, 14, 80, 3, 3, 1, 1, 1),    # 14-wide maps: whole-row blocks, one-word x loads
    (2, 16, 12, 16, 32, 3, 3, 1, 0, 1),    # 14 wide by pad 0, 10 rows
    # Whole-map halo blocks (13 x 13 outputs, 3x3; 14 x 14 ones keep the 14 x 8
    # blocks): groups, rows past one 64-row tile, a batch of 12, pad 0 and 2.
    (2, 64, 13, 13, 96, 3, 3, 1, 1, 2),
    (12, 32, 13, 13, 80, 3, 3, 1, 1, 1),
    (1, 128, 13, 13, 128, 3, 3, 1, 1, 1),  # 8 channel blocks: split whole-map plans
    (1, 32, 14, 14, 144, 3, 3, 1, 1, 1),
    (1, 16, 15, 15, 32, 3, 3, 1, 0, 1),
    (1, 16, 12, 12, 16, 3, 3, 1, 2, 1),
    (1, 32, 8, 12, 32, 3, 3, 1, 2, 1),     # 14 wide by pad 2
]


def _random_halo_shapes(count=8, seed=20261202):
    """Seeded stride-1 3x3 and 5x5 shapes with channels per group a multiple
    of 16 (so the halo GEMM is a candidate of forward and backward-data, and
    for 3x3 the halo backward-weight where the rows allow): random maps 5-40
    pixels a side, pads 0..R, one or two groups, filters per group 16-96."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        R = int(rng.choice([3, 5]))
        G = int(rng.choice([1, 2]))
        N = int(rng.integers(1, 4))
        C = G * 16 * int(rng.integers(1, 4))
        K = G * int(rng.choice([16, 32, 48, 64, 80, 96]))
        H, W = int(rng.integers(5, 41)), int(rng.integers(5, 41))
        pad = int(rng.integers(0, R + 1))
        if H + 2 * pad < R or W + 2 * pad < R:
            continue
        out.append((N, C, H, W, K, R, R, 1, pad, G))
    return out


@pytest.mark.parametrize("shape", _random_halo_shapes(), ids=lambda s: "x".join(map(str, s)))
def test_random_halo_shapes_every_candidate(shape):
    test_every_candidate_matches_oracle(shape)


def _random_whole_map_shapes(count=4, seed=20261203):
    """Seeded stride-1 3x3 shapes whose forward output is 13 x 13 (the
    whole-map halo block): pads 0..2 (source 15 - 2 pad a side), one or two
    groups, 16-48 channels and 16-96 filters a group."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        G = int(rng.choice([1, 2]))
        pad = int(rng.integers(0, 3))
        H = 15 - 2 * pad
        out.append((int(rng.integers(1, 4)), G * 16 * int(rng.integers(1, 4)), H, H,
                    G * int(rng.choice([16, 32, 48, 64, 80, 96])), 3, 3, 1, pad, G))
    return out


@pytest.mark.parametrize("shape", _random_whole_map_shapes(), ids=lambda s: "x".join(map(str, s)))
def test_random_whole_map_shapes_every_candidate(shape):
    test_every_candidate_matches_oracle(shape)


@pytest.fixture(autouse=True)
def _clean():
    import paper_1903_06934_amd as m
    m.plan_clear()
    yield
    m.plan_clear()


def _inputs(shape, seed):
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = oracle.out_size(H, R, st, pad), oracle.out_size(W, S, st, pad)
    return workloads.make_inputs(shape, P, Q, seed=seed, init="he")


def _run(pass_id, shape, t, ws):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    if pass_id == m.PASS_FWD:
        return (m.conv_fwd(t["x"], t["w"], t["b"], st, pad, G, ws=ws),)
    if pass_id == m.PASS_BWD_DATA:
        return (m.conv_bwd_data(t["dy"], t["w"], (H, W), st, pad, G, ws=ws),)
    return m.conv_bwd_weight(t["x"], t["dy"], (R, S), st, pad, G, ws=ws)


def _refs(shape, d):
    y, ay = oracle.conv_fwd(shape, d["x"], d["w"], d["b"])
    dx, adx = oracle.conv_bwd_data(shape, d["dy"], d["w"])
    dw, adw, db, adb = oracle.conv_bwd_weight(shape, d["x"], d["dy"])
    return {0: [(y, ay)], 1: [(dx, adx)], 2: [(dw, adw), (db, adb)]}


@pytest.mark.parametrize("shape", PLAN_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_candidate_matches_oracle(shape):
    import torch
    import paper_1903_06934_amd as m
    d = _inputs(shape, (31, 2))
    refs = _refs(shape, d)
    t = {k: dev(v) for k, v in d.items()}
    for p in (m.PASS_FWD, m.PASS_BWD_DATA, m.PASS_BWD_WEIGHT):
        n = m.plan_count(p, shape)
        for i in range(n):
            name = m.plan_name(p, shape, i)
            m.plan_set(p, shape, i)
            nbytes = m.plan_workspace_size(p, shape, i)
            assert nbytes <= m.workspace_size(p, shape)
            ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
            outs = _run(p, shape, t, ws)
            for (ref, absum), got in zip(refs[p], outs):
                assert_within(host(got), ref, absum, f"pass {p} plan {i} ({name})")
        m.plan_set(p, shape, 0)


@pytest.mark.parametrize("cfg,lname", [(1, "conv2"), (1, "conv1"), (3, "s14_3x3")])
def test_tune_stores_and_repeats(cfg, lname):
    """Tune the three passes of a benchmark layer at batch 4: the stored
    index is the one returned, the outputs of the tuning call meet the bar,
    and a plain call afterwards repeats them bitwise."""
    import torch
    import paper_1903_06934_amd as m
    name, layers = workloads.config(cfg)
    L = [l for l in layers if l.name == lname][0].with_batch(4)
    shape = L.shape
    N, C, H, W, K, R, S, st, pad, G = shape
    d = _inputs(shape, (32, cfg))
    refs = _refs(shape, d)
    t = {k: dev(v) for k, v in d.items()}
    outs = {0: [torch.empty((N, K, L.P, L.Q), device="cuda")],
            1: [torch.empty((N, C, H, W), device="cuda")],
            2: [torch.empty((K, C // G, R, S), device="cuda"), torch.empty(K, device="cuda")]}
    ins = {0: (t["x"], t["w"], t["b"]), 1: (t["dy"], t["w"], None), 2: (t["x"], t["dy"], None)}
    for p in (m.PASS_FWD, m.PASS_BWD_DATA, m.PASS_BWD_WEIGHT):
        n = m.plan_count(p, shape)
        nbytes = max(m.plan_workspace_size(p, shape, i) for i in range(n))
        ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
        o = outs[p] + [None] * (2 - len(outs[p]))
        chosen = m.conv_tune(p, shape, *ins[p], o[0], o[1], ws, reps=2)
        assert 0 <= chosen < n
        assert m.plan_get(p, shape) == chosen
        tuned = [host(x) for x in outs[p]]
        for (ref, absum), got in zip(refs[p], tuned):
            assert_within(got, ref, absum, f"tuned pass {p} ({m.plan_name(p, shape, chosen)})")
        again = [host(x) for x in _run(p, shape, t, ws)]
        for a, b in zip(tuned, again):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_tune_respects_workspace():
    """With the rule's workspace, only candidates that fit may be chosen."""
    import torch
    import paper_1903_06934_amd as m
    shape = (2, 64, 12, 12, 32, 5, 5, 1, 2, 1)
    N, C, H, W, K, R, S, st, pad, G = shape
    d = _inputs(shape, (33, 0))
    t = {k: dev(v) for k, v in d.items()}
    nbytes = m.plan_workspace_size(m.PASS_FWD, shape, 0)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    y = torch.empty((N, K, 12, 12), device="cuda")
    chosen = m.conv_tune(m.PASS_FWD, shape, t["x"], t["w"], t["b"], y, None, ws, reps=1)
    assert m.plan_workspace_size(m.PASS_FWD, shape, chosen) <= nbytes
    ref, absum = oracle.conv_fwd(shape, d["x"], d["w"], d["b"])
    assert_within(host(y), ref, absum, "tuned forward")


def _tuned_cases():
    out = []
    for cfg in (1, 2, 3, 4, 5):
        name, layers = workloads.config(cfg)
        for li, L in enumerate(layers):
            if isinstance(L, workloads.PoolLayer) or (cfg == 5 and L.R > 1):
                continue  # pooling has its own tests; config 5's convolutions are config 1's
            out.append(pytest.param(cfg, li, id=f"{name}-{L.name}"))
    return out


@pytest.mark.parametrize("cfg,li", _tuned_cases())
def test_tuned_plans_full_batch_sampled(cfg, li):
    """The benchmark's launch configuration: every pass of the layer at its
    configured batch with the plan conv_tune keeps (as bench.py does before
    timing), then sampled elements (every dw element when dw has at most 64k)
    against the oracle's gather forms."""
    import torch
    import paper_1903_06934_amd as m
    from gpu_util import dw_indices, sample_indices
    L = workloads.config(cfg)[1][li]
    d = workloads.layer_inputs(cfg, li)
    shape = L.shape
    N, C, H, W, K, R, S, st, pad, G = shape
    t = {k: dev(v) for k, v in d.items()}
    outs = {0: [torch.empty((N, K, L.P, L.Q), device="cuda")],
            1: [torch.empty((N, C, H, W), device="cuda")],
            2: [torch.empty((K, C // G, R, S), device="cuda"), torch.empty(K, device="cuda")]}
    ins = {0: (t["x"], t["w"], t["b"]), 1: (t["dy"], t["w"], None), 2: (t["x"], t["dy"], None)}
    names = {}
    for p in (m.PASS_FWD, m.PASS_BWD_DATA, m.PASS_BWD_WEIGHT):
        n = m.plan_count(p, shape)
        nbytes = max(m.plan_workspace_size(p, shape, i) for i in range(n))
        ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
        o = outs[p] + [None] * (2 - len(outs[p]))
        chosen = m.conv_tune(p, shape, *ins[p], o[0], o[1], ws, reps=2)
        names[p] = f"{chosen}: {m.plan_name(p, shape, chosen)}"
        del ws
    # The ordinary calls now run the stored plans.
    rng = np.random.default_rng([cfg, li, 77])
    y = host(m.conv_fwd(t["x"], t["w"], t["b"], st, pad, G))
    idx = sample_indices(y.shape, rng, groups=G)
    v, a = oracle.conv_fwd_at(shape, d["x"], d["w"], d["b"], idx)
    assert_within(y.ravel()[idx], v, a, f"fwd with plan {names[0]}")
    del y
    dx = host(m.conv_bwd_data(t["dy"], t["w"], (H, W), st, pad, G))
    idx = sample_indices(dx.shape, rng, groups=G)
    v, a = oracle.conv_bwd_data_at(shape, d["dy"], d["w"], idx)
    assert_within(dx.ravel()[idx], v, a, f"bwd_data with plan {names[1]}")
    del dx
    dw, db = m.conv_bwd_weight(t["x"], t["dy"], (R, S), st, pad, G)
    dw, db = host(dw), host(db)
    idx = dw_indices(dw.shape, N * L.P * L.Q, rng)  # every element when |dw| <= 64k
    v, a = oracle.conv_bwd_weight_at(shape, d["x"], d["dy"], idx)
    assert_within(dw.ravel()[idx], v, a, f"bwd_weight with plan {names[2]}")
    v, a = oracle.bias_grad(d["dy"])
    assert_within(db, v, a, f"bias_grad with plan {names[2]}")
