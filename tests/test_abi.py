"""The C-ABI library on the CPU: it loads, exports every function that
include/miconv.h declares, computes geometry and workspace sizes on the
host, and rejects bad arguments before touching any device.  No kernel runs
here: the pointers below are fake device addresses that the library never
dereferences, because every check fails first."""
import ctypes
import os
import re

import pytest

import paper_1903_06934_amd as m
from paper_1903_06934_amd import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "miconv.h")

OK, SHAPE, NULL, WS, ALIAS, ALIGN, DEVICE = 0, -1, -2, -3, -4, -5, -6


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(libbuild.LIBRARY):
        libbuild.build()
    return m.lib()


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"sizeof", "defined"})


def test_exports_every_declared_function(L):
    names = declared_functions()
    assert set(names) == {"conv_output_size", "conv_workspace_size", "conv_fwd",
                          "conv_bwd_data", "conv_bwd_weight", "conv_error_string",
                          "conv_set_timing_events", "conv_plan_count", "conv_plan_get",
                          "conv_plan_set", "conv_plan_clear", "conv_plan_name",
                          "conv_plan_workspace_size", "conv_tune", "pool_output_size",
                          "pool_fwd", "pool_bwd", "conv_bwd_weight_noalloc"}
    for n in names:
        assert hasattr(L, n), n


def test_peak_library_exports_its_header():
    """libmipeak.so (the benchmark's measured reference points) loads and
    exports what include/mipeak.h declares; its calls reject bad arguments
    before launching anything."""
    from paper_1903_06934_amd import peaks
    if not os.path.exists(peaks.LIBRARY):
        libbuild.build()
    P = peaks.lib()
    names = declared_functions(os.path.join(ROOT, "include", "mipeak.h"))
    assert set(names) == {"peak_mfma_f32", "peak_copy"}
    for n in names:
        assert hasattr(P, n), n
    assert P.peak_mfma_f32(1, 4, 10, 5, 0x1000, None, None) == -1   # chains not 4, 8, 16
    assert P.peak_mfma_f32(1, 17, 10, 8, 0x1000, None, None) == -1  # more than 16 waves
    assert P.peak_mfma_f32(1, 4, 10, 8, None, None, None) == -1     # no sink
    assert P.peak_copy(0x1000, 0x2000, 24, 8, None) == -1           # not a multiple of 16
    assert P.peak_copy(0x1004, 0x2000, 32, 8, None) == -1           # misaligned


@pytest.mark.parametrize("n_in,f,st,pad,want", [
    (227, 11, 4, 0, 55), (224, 7, 2, 3, 112), (56, 1, 2, 0, 28), (224, 3, 1, 1, 224),
    (27, 5, 1, 2, 27), (13, 3, 1, 1, 13), (4, 3, 2, 1, 2), (5, 2, 3, 0, 2), (3, 5, 1, 1, 1),
    (1, 1, 1, 0, 1)])
def test_output_size(L, n_in, f, st, pad, want):
    assert m.output_size(n_in, n_in, f, f, st, pad) == (want, want)
    assert m.output_size(n_in, 7, f, 1, st, pad)[0] == want


@pytest.mark.parametrize("args", [(3, 3, 5, 5, 1, 0), (0, 3, 1, 1, 1, 0), (3, 3, 1, 1, 0, 0),
                                  (3, 3, 1, 1, 1, -1), (3, 3, 0, 1, 1, 0)])
def test_output_size_rejects(L, args):
    import ctypes
    P, Q = ctypes.c_int(-7), ctypes.c_int(-7)
    assert L.conv_output_size(*args, ctypes.byref(P), ctypes.byref(Q)) == SHAPE
    assert (P.value, Q.value) == (-7, -7)
    assert L.conv_output_size(5, 5, 3, 3, 1, 0, None, ctypes.byref(Q)) == NULL


def test_timing_events_arguments(L):
    L.conv_set_timing_events.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    assert L.conv_set_timing_events(None, None) == OK
    assert L.conv_set_timing_events(0x1000, None) == NULL
    assert L.conv_set_timing_events(None, 0x1000) == NULL


def test_error_strings(L):
    for s in range(-10, 1):
        assert L.conv_error_string(s)
    assert L.conv_error_string(12345) == b"unknown status"


GOOD = (2, 16, 32, 32, 32, 3, 3, 1, 1, 1)
BAD_SHAPES = [
    (0, 16, 32, 32, 32, 3, 3, 1, 1, 1), (2, 16, 32, 32, 32, 3, 3, 0, 1, 1),
    (2, 16, 32, 32, 32, 3, 3, 1, -1, 1), (2, 15, 32, 32, 32, 3, 3, 1, 1, 2),
    (2, 16, 32, 32, 30, 3, 3, 1, 1, 4), (2, 16, 2, 2, 32, 5, 5, 1, 0, 1),
    (2048, 1024, 64, 64, 8, 1, 1, 1, 0, 1),  # x above 2^31 - 1 elements
]

X, W_, B, Y, WSP = 0x10000000, 0x20000000, 0x28000000, 0x30000000, 0x40000000


def test_workspace_sizes(L):
    for p in (0, 1, 2):
        assert m.workspace_size(p, GOOD) > 0
        for bad in BAD_SHAPES:
            assert m.workspace_size(p, bad) == 0
    assert m.workspace_size(3, GOOD) == 0
    # the rule (candidate 0): one packed filter per pass; stride phases
    # partition the taps
    assert m.plan_workspace_size(0, GOOD, 0) == 32 * 16 * 9 * 4
    assert m.plan_workspace_size(1, (2, 4, 9, 9, 8, 3, 3, 2, 1, 1), 0) >= 8 * 4 * 9 * 4
    # the size to allocate covers every candidate plan of the shape
    for p in (0, 1, 2):
        n = m.plan_count(p, GOOD)
        assert m.workspace_size(p, GOOD) == max(m.plan_workspace_size(p, GOOD, i)
                                                for i in range(n))


def _align(n):
    return (n + 255) // 256 * 256


@pytest.mark.parametrize("shape,b,taps", [
    # AlexNet conv1: 4 x 4 blocks (48 rows), 3 x 3 dy taps per block
    ((128, 3, 227, 227, 96, 11, 11, 4, 0, 1), 4, 9),
    # ResNet stem: 4 x 4 blocks (f = 2), 5 x 5 taps
    ((64, 3, 224, 224, 64, 7, 7, 2, 3, 1), 4, 25),
    # VGG conv1_1 (stride 1): 2 x 2 blocks, 4 x 4 taps
    ((32, 3, 224, 224, 64, 3, 3, 1, 1, 1), 2, 16),
])
def test_bwd_data_blocked_plan_for_first_layers(L, shape, b, taps):
    """Few input channels: backward-data stacks the b x b pixels of a block
    into the GEMM rows, and its workspace is that one packed filter bank of
    C b^2 rows by (K/G) x taps reduction rows (padded to 16)."""
    N, C, H, W, K, R, S, st, pad, G = shape
    rows = C * b * b
    red = (K // G * taps + 15) // 16 * 16
    assert m.plan_workspace_size(1, shape, 0) == _align(rows * red * 4)


def test_bwd_data_phase_plan_for_wide_layers(L):
    """Channel-aligned layers keep one GEMM per stride phase (AlexNet conv2)."""
    shape = (128, 96, 27, 27, 256, 5, 5, 1, 2, 2)
    assert m.plan_workspace_size(1, shape, 0) == _align(96 * 128 * 25 * 4)


@pytest.mark.parametrize("shape", BAD_SHAPES)
def test_bad_shapes(L, shape):
    assert L.conv_fwd(*shape, X, W_, None, Y, WSP, 1 << 30, None) == SHAPE
    assert L.conv_bwd_data(*shape, Y, W_, X, WSP, 1 << 30, None) == SHAPE
    assert L.conv_bwd_weight(*shape, X, Y, W_, None, WSP, 1 << 30, None) == SHAPE


def test_fwd_checks(L):
    ws = m.plan_workspace_size(0, GOOD, 0)  # the rule's need (no plan stored)
    f = lambda *a: L.conv_fwd(*GOOD, *a, None)
    assert f(None, W_, B, Y, WSP, ws) == NULL
    assert f(X, None, B, Y, WSP, ws) == NULL
    assert f(X, W_, B, None, WSP, ws) == NULL
    assert f(X + 4, W_, B, Y, WSP, ws) == ALIGN
    assert f(X, W_, B + 8, Y, WSP, ws) == ALIGN
    assert f(X, W_, B, Y, WSP, ws - 1) == WS
    assert f(X, W_, B, Y, None, ws) == WS
    assert f(X, W_, B, Y, WSP + 4, ws) == ALIGN
    assert f(X, W_, B, X + 64, WSP, ws) == ALIAS          # y overlaps x
    assert f(X, W_, B, Y, Y + 256, ws) == ALIAS           # ws overlaps y
    assert f(X, W_, B, Y, W_, ws) == ALIAS                # ws overlaps w
    # inputs may overlap each other
    assert f(X, X, None, Y, WSP, ws) in (OK, DEVICE)


def test_bwd_checks(L):
    ws = m.plan_workspace_size(1, GOOD, 0)
    g = lambda *a: L.conv_bwd_data(*GOOD, *a, None)
    assert g(None, W_, X, WSP, ws) == NULL
    assert g(Y, W_, None, WSP, ws) == NULL
    assert g(Y, W_, X, WSP, ws - 4) == WS
    assert g(Y, W_, Y + 16, WSP, ws) == ALIAS
    ws = m.plan_workspace_size(2, GOOD, 0)
    h = lambda *a: L.conv_bwd_weight(*GOOD, *a, None)
    assert h(X, Y, None, B, WSP, ws) == NULL
    assert h(X, None, W_, B, WSP, ws) == NULL
    assert h(X, Y, W_, W_ + 16, WSP, ws) == ALIAS        # db overlaps dw
    assert h(X, Y, W_, X, WSP, ws) == ALIAS              # db overlaps x
    assert h(X, Y, W_, None, WSP, 0) == WS
    assert h(X, Y, W_ + 4, None, WSP, ws) == ALIGN


def test_noalloc_checks_before_any_device_use(L):
    """conv_bwd_weight_noalloc refuses, on the host, a shape whose plan needs
    more than the fixed scratch (96 MiB) and a bad shape; a well-formed call
    reaches the device check."""
    import torch
    SCRATCH = -11
    big = (32, 512, 28, 28, 512, 3, 3, 1, 1, 1)
    n = m.plan_count(2, big)
    i = max(range(n), key=lambda j: m.plan_workspace_size(2, big, j))
    assert m.plan_workspace_size(2, big, i) > (96 << 20)
    m.plan_set(2, big, i)
    try:
        assert L.conv_bwd_weight_noalloc(*big, X, Y, W_, None, None) == SCRATCH
    finally:
        m.plan_clear()
    assert L.conv_bwd_weight_noalloc(*BAD_SHAPES[0], X, Y, W_, None, None) == SHAPE
    if not torch.cuda.is_available():
        assert L.conv_bwd_weight_noalloc(*GOOD, X, Y, W_, B, None) == DEVICE


def test_device_check_without_gpu(L):
    """On a host without a gfx950 device, a well-formed call reports
    MICONV_ERR_DEVICE (and launches nothing)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    ws = m.workspace_size(0, GOOD)
    assert L.conv_fwd(*GOOD, X, W_, B, Y, WSP, ws, None) == DEVICE


@pytest.mark.parametrize("args,want", [
    ((55, 55, 3, 3, 2, 0), (27, 27)), ((224, 224, 2, 2, 2, 0), (112, 112)),
    ((6, 5, 3, 3, 2, 0), (3, 2)), ((3, 3, 2, 2, 2, 1), (2, 2))])
def test_pool_output_size(L, args, want):
    assert m.pool_output_size(*args) == want


def test_pool_rejects(L):
    X, Y, M = 0x10000000, 0x20000000, 0x30000000
    MODE = -10
    assert L.pool_fwd(2, 1, 1, 8, 8, 2, 2, 2, 0, X, Y, M, None) == MODE
    assert L.pool_fwd(0, 1, 1, 8, 8, 2, 2, 2, 2, X, Y, M, None) == SHAPE   # pad >= window
    assert L.pool_fwd(0, 1, 1, 2, 2, 5, 5, 1, 0, X, Y, M, None) == SHAPE   # window > image
    assert L.pool_fwd(0, 1, 1, 10, 9, 1, 1, 2, 0, X, Y, M, None) == SHAPE  # last window past the image
    assert L.pool_bwd(1, 1, 1, 9, 10, 1, 1, 2, 0, Y, None, X, None) == SHAPE
    assert L.pool_fwd(0, 1, 1, 8, 8, 2, 2, 2, 0, None, Y, M, None) == NULL
    assert L.pool_bwd(0, 1, 1, 8, 8, 2, 2, 2, 0, Y, None, X, None) == NULL   # max needs mask
    assert L.pool_fwd(1, 1, 1, 8, 8, 2, 2, 2, 0, X + 4, Y, None, None) == ALIGN
    assert L.pool_fwd(1, 1, 1, 8, 8, 2, 2, 2, 0, X, X + 64, None, None) == ALIAS
