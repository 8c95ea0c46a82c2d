"""The CPU oracle against its pins (hand cases, GEMM identities, the
explicit im2col plan, torch's CPU fp64 conv, adjoint, finite differences,
delta filters and invariants).  CPU only."""
import json
import os

import pytest

import oracle
import workloads
from oracle_pins import ALL_CHECKS, GOLDEN


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(check):
    check(oracle.default())


def test_stated_output_sizes_of_every_config():
    """Each configured layer's stated P x Q is what the size formula gives."""
    o = oracle.default()
    for cfg, (_, layers) in workloads.CONFIGS.items():
        for L in layers:
            size = o.pool_out_size if isinstance(L, workloads.PoolLayer) else o.out_size
            assert size(L.H, L.R, L.stride, L.pad) == L.P, (cfg, L.name)
            assert size(L.W, L.S, L.stride, L.pad) == L.Q, (cfg, L.name)


def test_table2_flop_convention():
    """Table II's Gflops column equals 2 N K P Q (C/G) R S / time within the
    rounding of its printed times (VGG-16, batch 128, 3x3 s1 p1)."""
    t = json.load(open(os.path.join(GOLDEN, "table2_vgg16.json")))
    N = t["batch"]
    for row in t["rows"]:
        s = row["map"]
        flops = 2.0 * N * row["No"] * s * s * row["Ni"] * 9
        for key in ("fwd", "wdiff", "indiff"):
            if row[key] is None:
                continue
            secs, gflops = row[key]
            assert abs(flops / secs / 1e9 - gflops) <= 0.03 * gflops, (row["conv"], key)
