"""Plan selection on the host (no GPU): candidate lists, names, the rule as
candidate 0, storing and clearing a choice, per-candidate workspace sizes and
argument errors."""
import pytest

import paper_1903_06934_amd as m
import workloads

PASSES = (m.PASS_FWD, m.PASS_BWD_DATA, m.PASS_BWD_WEIGHT)
SHAPE_ERR, NULL_ERR, PASS_ERR, PLAN_ERR = -1, -2, -8, -9


def _layers():
    out = []
    for cfg in (0, 1, 2, 3, 4):
        name, layers = workloads.config(cfg)
        out += [pytest.param(L.shape, id=f"{name}-{L.name}") for L in layers]
    return out


@pytest.fixture(autouse=True)
def _clean():
    m.plan_clear()
    yield
    m.plan_clear()


@pytest.mark.parametrize("shape", _layers())
def test_candidates_are_distinct_and_rule_first(shape):
    for p in PASSES:
        n = m.plan_count(p, shape)
        assert n >= 1
        names = [m.plan_name(p, shape, i) for i in range(n)]
        assert len(set(names)) == n, names
        assert m.plan_get(p, shape) == 0
        assert m.plan_workspace_size(p, shape, 0) <= m.workspace_size(p, shape)


def test_rule_names_for_alexnet():
    """The built-in rule on the AlexNet-shaped stack (batch 128)."""
    _, layers = workloads.config(1)
    by = {L.name: L.shape for L in layers}
    assert m.plan_name(m.PASS_BWD_DATA, by["conv1"], 0) == \
        "blocked 4x4 pixels (f=1), image GEMM 48x64"
    assert m.plan_name(m.PASS_BWD_DATA, by["conv2"], 0) == \
        "stride phases, halo GEMM 64x112 (28x4 pixels)"
    assert m.plan_name(m.PASS_FWD, by["conv2"], 0) == "halo GEMM 64x112 (28x4 pixels)"
    for name in ("conv3", "conv4", "conv5"):  # 13 x 13 maps: whole-map blocks
        assert m.plan_name(m.PASS_FWD, by[name], 0) == "halo GEMM 64x176 (13x13 pixels)"
        assert m.plan_name(m.PASS_BWD_DATA, by[name], 0) == \
            "stride phases, halo GEMM 64x176 (13x13 pixels)"
    assert m.plan_name(m.PASS_FWD, by["conv1"], 0) == "image GEMM 96x128"
    assert m.plan_name(m.PASS_BWD_WEIGHT, by["conv2"], 0).startswith("tap 64x48, ")
    assert m.plan_name(m.PASS_BWD_WEIGHT, by["conv1"], 0).startswith("pixel 96x64, ")


def test_rule_splits_uneven_halo_grids():
    """GoogLeNet-shaped 14 x 14 3x3 layers at batch 64: 384 backward-data
    tiles (1.5 a CU) split in two; 768 tiles run unsplit, 256 or 512 (one or
    two a CU, evenly) with two wave groups."""
    _, layers = workloads.config(4)
    by = {L.name: L.shape for L in layers}
    assert m.plan_name(m.PASS_BWD_DATA, by["hi_3x3"], 0) == \
        "stride phases, halo GEMM 64x112 (14x8 pixels), 2 splits"
    assert m.plan_name(m.PASS_FWD, by["hi_3x3"], 0) == "halo GEMM 64x112 (14x8 pixels)"
    assert m.plan_name(m.PASS_BWD_DATA, by["mid_3x3"], 0) == \
        "stride phases, halo GEMM 64x112 (14x8 pixels), 8 waves"
    assert m.plan_name(m.PASS_FWD, by["mid_3x3"], 0) == "halo GEMM 64x112 (14x8 pixels), 8 waves"


def test_rule_two_wave_groups_for_vgg_conv5():
    """VGG-16-shaped conv5_x at batch 32 (512 tiles of 64 rows, two a CU):
    two wave groups over the 32 channel blocks; conv4_x (1024 tiles) and the
    224-wide conv1_2 keep four waves."""
    _, layers = workloads.config(2)
    by = {L.name: L.shape for L in layers}
    for p in (m.PASS_FWD, m.PASS_BWD_DATA):
        assert m.plan_name(p, by["conv5_1"], 0).endswith("(14x8 pixels), 8 waves")
        assert "8 waves" not in m.plan_name(p, by["conv4_2"], 0)
        assert "8 waves" not in m.plan_name(p, by["conv1_2"], 0)


def test_two_wave_group_candidates_need_even_channel_blocks():
    """Two wave groups split a tile's channel blocks in halves: offered for
    3x3 halo plans with an even number of 16-channel blocks and few tiles,
    never with an odd number, for 112-wide blocks or with a split."""
    even = (2, 64, 14, 14, 32, 3, 3, 1, 1, 1)   # 4 channel blocks
    odd = (2, 48, 14, 14, 32, 3, 3, 1, 1, 1)    # 3 channel blocks
    wide = (1, 64, 4, 112, 32, 3, 3, 1, 1, 1)   # 112-wide blocks
    names = lambda sh: [m.plan_name(m.PASS_FWD, sh, i) for i in range(m.plan_count(m.PASS_FWD, sh))]
    assert any(n.endswith("8 waves") for n in names(even))
    assert not any("8 waves" in n for n in names(odd))
    assert not any("112x1 pixels), 8 waves" in n for n in names(wide))
    assert not any("splits, 8 waves" in n or ("8 waves" in n and "splits" in n) for n in names(even))


def test_set_get_clear_and_workspace():
    shape = (8, 3, 67, 67, 32, 11, 11, 4, 2, 1)
    n = m.plan_count(m.PASS_BWD_DATA, shape)
    assert n > 2
    m.plan_set(m.PASS_BWD_DATA, shape, n - 1)
    assert m.plan_get(m.PASS_BWD_DATA, shape) == n - 1
    assert m.plan_get(m.PASS_FWD, shape) == 0  # per pass
    assert m.workspace_size(m.PASS_BWD_DATA, shape) == \
        max(m.plan_workspace_size(m.PASS_BWD_DATA, shape, i) for i in range(n))
    m.plan_set(m.PASS_BWD_DATA, shape, 0)
    assert m.plan_get(m.PASS_BWD_DATA, shape) == 0
    m.plan_set(m.PASS_BWD_DATA, shape, 1)
    m.plan_clear()
    assert m.plan_get(m.PASS_BWD_DATA, shape) == 0


def test_split_candidates_grow_the_workspace():
    """A split plan's partial sums are in the workspace; the rule here does
    not split (the grid is large), a split candidate does."""
    shape = (2, 64, 12, 12, 32, 5, 5, 1, 2, 1)
    n = m.plan_count(m.PASS_FWD, shape)
    names = [m.plan_name(m.PASS_FWD, shape, i) for i in range(n)]
    split = [i for i, s in enumerate(names) if "splits" in s]
    assert split, names
    for i in split:
        assert m.plan_workspace_size(m.PASS_FWD, shape, i) > m.plan_workspace_size(m.PASS_FWD,
                                                                                 shape, 0)


def test_plan_errors():
    good = (2, 16, 32, 32, 32, 3, 3, 1, 1, 1)
    bad = (2, 15, 32, 32, 32, 3, 3, 1, 1, 2)
    L = m.lib()
    assert L.conv_plan_count(7, *good) == PASS_ERR
    assert L.conv_plan_count(0, *bad) == SHAPE_ERR
    assert L.conv_plan_get(3, *good) == PASS_ERR
    n = m.plan_count(0, good)
    assert L.conv_plan_set(0, *good, n) == PLAN_ERR
    assert L.conv_plan_set(0, *good, -1) == PLAN_ERR
    assert L.conv_plan_name(0, *good, 0, None, 16) == NULL_ERR
    assert L.conv_plan_name(0, *good, n, b"x" * 8, 8) == PLAN_ERR
    assert L.conv_plan_workspace_size(0, *good, n) == 0
    assert m.plan_get(0, good) == 0


def test_explicit_candidates():
    """The explicit plan (im2col / col2im around the 1x1 GEMM) is a candidate
    of every pass where its columns differ from the input, with a column
    chunk of at most 256 MB in its workspace; not for a 1x1 stride-1 layer."""
    conv1 = (128, 3, 227, 227, 96, 11, 11, 4, 0, 1)
    for p in PASSES:
        n = m.plan_count(p, conv1)
        names = [m.plan_name(p, conv1, i) for i in range(n)]
        ex = [i for i, s in enumerate(names) if s.startswith("explicit")]
        assert len(ex) == 1, names
        col_chunk = int(names[ex[0]].split("(")[1].split()[0])   # images a chunk
        assert col_chunk * 3 * 121 * 55 * 55 * 4 <= 256 << 20
        assert m.plan_workspace_size(p, conv1, ex[0]) >= col_chunk * 3 * 121 * 55 * 55 * 4
    one = (64, 256, 56, 56, 64, 1, 1, 1, 0, 1)
    for p in PASSES:
        n = m.plan_count(p, one)
        assert not any(m.plan_name(p, one, i).startswith("explicit") for i in range(n))


def test_plan_table_is_thread_safe():
    """Threads storing and reading choices for their own shapes at the same
    time (ctypes releases the GIL around each call) each read back exactly
    what they stored."""
    import threading
    shapes = [(8 + i, 16, 20, 20, 32, 3, 3, 1, 1, 1) for i in range(8)]
    errors = []

    def work(shape):
        try:
            n = m.plan_count(m.PASS_FWD, shape)
            for r in range(400):
                idx = r % n
                m.plan_set(m.PASS_FWD, shape, idx)
                got = m.plan_get(m.PASS_FWD, shape)
                if got != idx:
                    errors.append((shape, idx, got))
                    return
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(e)

    threads = [threading.Thread(target=work, args=(s,)) for s in shapes]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:3]


def test_workspace_sized_before_tuning_stays_sufficient():
    """A caller sizes its workspace, then (say, another thread) a plan with
    the largest need of all candidates is stored for the same shape: the
    caller's next call must still pass the workspace check (on this host
    without a GPU it then stops at the device check)."""
    L = m.lib()
    X, W_, B, Y, WSP = 0x10000000, 0x20000000, 0x28000000, 0x30000000, 0x40000000
    DEVICE, WS = -6, -3
    shape = (2, 64, 12, 12, 32, 5, 5, 1, 2, 1)
    for p in PASSES:
        ws = m.workspace_size(p, shape)
        n = m.plan_count(p, shape)
        needs = [m.plan_workspace_size(p, shape, i) for i in range(n)]
        big = max(range(n), key=lambda i: needs[i])
        assert needs[big] > needs[0]  # the check below is not vacuous
        m.plan_set(p, shape, big)
        assert m.workspace_size(p, shape) == ws
        if p == m.PASS_FWD:
            call = lambda nb: L.conv_fwd(*shape, X, W_, B, Y, WSP, nb, None)  # noqa: E731
        elif p == m.PASS_BWD_DATA:
            call = lambda nb: L.conv_bwd_data(*shape, Y, W_, X, WSP, nb, None)  # noqa: E731
        else:
            call = lambda nb: L.conv_bwd_weight(*shape, X, Y, W_, B, WSP, nb, None)  # noqa: E731
        assert call(ws) == DEVICE
        assert call(needs[big] - 1) == WS


@pytest.mark.parametrize("shape", [
    (2, 4, 1, 1, 3, 1, 1, 3, 1, 1),     # 1x1 image, 1x1 filter, pad 1, stride 3: P = Q = 1
    (16, 8, 1, 1, 32, 1, 1, 5, 2, 1),   # the same with a batch of 16s
])
def test_padded_one_by_one_is_not_an_inner_product(shape):
    """With padding, the lone output pixel of a 1x1 image reads only zero
    padding (y = b, dx = 0, dw = 0); the batch-transposed inner-product plans
    ignore padding, so such shapes must take the implicit plans."""
    for p in PASSES:
        for i in range(m.plan_count(p, shape)):
            assert "batch-transposed" not in m.plan_name(p, shape, i)
    unpadded = shape[:8] + (0, 1)
    assert "batch-transposed" in m.plan_name(m.PASS_FWD, unpadded[:7] + (1, 0, 1), 0)
