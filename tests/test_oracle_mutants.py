"""The oracle's pins are sensitive: copies of the oracle with one planted,
plausible mistake each (a dropped term, a wrong sign or index, a transposed
operand, a wrong rounding or boundary) are built on the CPU, and every one
of them must fail at least one pin.  CPU only; the planted mistakes live in
temporary copies, never in the oracle itself."""
import os

import pytest

import oracle
from oracle_pins import ALL_CHECKS
from test_oracle_pool import POOL_CHECKS

# (name, text in oracle.c, replacement, which occurrence (0-based))
MUTANTS = [
    ("fwd_drops_bias", "acc = b[k];", "acc = 0.0;", 0),
    ("fwd_flipped_filter", "w[(((i64)k * Cg + c) * R + r) * S + s]",
     "w[(((i64)k * Cg + c) * R + (R - 1 - r)) * S + (S - 1 - s)]", 0),
    ("fwd_abs_sum_signed", "aacc += fabs(xv * wv);", "aacc += xv * wv;", 0),
    ("fwd_wrong_group_offset", "x_at(x, C, H, W, n, g * Cg + c,", "x_at(x, C, H, W, n, c,", 0),
    ("boundary_off_by_one", "w < 0 || w >= W", "w < 1 || w >= W", 0),
    ("size_ceil_rounding", "span / stride + 1", "(span + stride - 1) / stride + 1", 0),
    ("bwd_data_group_dropped", "for (int k = g * Kg; k < (g + 1) * Kg; k++)",
     "for (int k = 0; k < Kg; k++)", 0),
    ("bwd_data_stride_dropped", "i64 h = (i64)p * stride - pad + r;",
     "i64 h = (i64)p - pad + r;", 0),
    ("bwd_data_transposed_filter", "d * w[(((i64)k * Cg + c) * R + r) * S + s]",
     "d * w[(((i64)k * Cg + c) * S + s) * R + r]", 0),
    ("bwd_weight_transposed_taps", "i64 o = ((i64)c * R + r) * S + s;",
     "i64 o = ((i64)c * S + s) * R + r;", 0),
    ("bias_grad_dropped_term", "bsum += d;", "bsum += (p > 0) ? d : 0.0;", 0),
    ("gather_dx_phase_check_dropped", "ph < 0 || qw < 0 || ph % stride || qw % stride",
     "ph < 0 || qw < 0 || qw % stride", 0),
    ("gather_dw_group_dropped", "x_at(x, C, H, W, n, g * Cg + c,", "x_at(x, C, H, W, n, c,", 2),
]

# Pooling (checked against the pooling pins).
POOL_MUTANTS = [
    ("pool_size_floor", "i64 out = (span + stride - 1) / stride + 1;",
     "i64 out = span / stride + 1;", 0),
    ("pool_size_no_last_window_rule", "if (pad > 0 && (out - 1) * stride >= (i64)in + pad)",
     "if (0)", 0),
    ("pool_size_allows_empty_window", "if ((out - 1) * stride - pad >= (i64)in)", "if (0)", 0),
    ("pool_window_ignores_pad", "i64 start = (i64)p * stride - pad;",
     "i64 start = (i64)p * stride;", 0),
    ("pool_avg_divisor_without_padding", "*ext = end - start;",
     "*ext = (end > in ? in : end) - (start < 0 ? 0 : start);", 0),
    ("pool_avg_overhang_counted", "end = (i64)in + pad;", "end = end + 0;", 0),
    ("pool_max_last_maximum", "if (xp[h * W + w] > best) {", "if (xp[h * W + w] >= best) {", 0),
    ("pool_bwd_avg_share_undivided", "double share = g / (double)(eh * ew);",
     "double share = g;", 0),
    ("pool_bwd_max_wrong_element", "dxp[arg] += g;", "dxp[arg > 0 ? arg - 1 : 0] += g;", 0),
]


def _mutate(text, old, new, nth):
    pos = -1
    for _ in range(nth + 1):
        pos = text.find(old, pos + 1)
        assert pos >= 0, f"mutation site not found: {old!r} #{nth}"
    return text[:pos] + new + text[pos + len(old):]


@pytest.mark.parametrize("name,old,new,nth", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, nth):
    src = open(oracle.SOURCE).read()
    path = tmp_path / f"{name}.c"
    path.write_text(_mutate(src, old, new, nth))
    lib = oracle.build(str(path), str(tmp_path / f"lib{name}.so"), werror=False)
    o = oracle.Oracle(lib)
    failed = []
    for check in ALL_CHECKS:
        try:
            check(o)
        except Exception:  # any pin that fails or cannot even run catches it
            failed.append(check.__name__)
    assert failed, f"mutant {name} passed every pin"


@pytest.mark.parametrize("name,old,new,nth", POOL_MUTANTS, ids=[m[0] for m in POOL_MUTANTS])
def test_pool_mutant_is_caught(tmp_path, name, old, new, nth):
    src = open(oracle.SOURCE).read()
    path = tmp_path / f"{name}.c"
    path.write_text(_mutate(src, old, new, nth))
    lib = oracle.build(str(path), str(tmp_path / f"lib{name}.so"), werror=False)
    o = oracle.Oracle(lib)
    failed = []
    for check in POOL_CHECKS:
        try:
            check(o)
        except Exception:
            failed.append(check.__name__)
    assert failed, f"mutant {name} passed every pooling pin"
