"""The passes on two HIP streams at once: the library keeps no per-call state
besides the caller's workspace, so two layers launched concurrently on
different streams (each with its own workspace) give bit for bit what they
give one after the other."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import dev, host

pytestmark = pytest.mark.gpu

LAYERS = [(4, 64, 27, 27, 96, 5, 5, 1, 2, 2), (4, 96, 13, 13, 128, 3, 3, 1, 1, 1)]


def _passes(shape, t, ws):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    y = m.conv_fwd(t["x"], t["w"], t["b"], st, pad, G, ws=ws[0])
    dx = m.conv_bwd_data(t["dy"], t["w"], (H, W), st, pad, G, ws=ws[1])
    dw, db = m.conv_bwd_weight(t["x"], t["dy"], (R, S), st, pad, G, ws=ws[2])
    return [y, dx, dw, db]


def test_two_streams_match_sequential():
    import torch
    import paper_1903_06934_amd as m
    data = []
    for i, shape in enumerate(LAYERS):
        N, C, H, W, K, R, S, st, pad, G = shape
        P, Q = oracle.out_size(H, R, st, pad), oracle.out_size(W, S, st, pad)
        d = workloads.make_inputs(shape, P, Q, seed=(55, i), init="he")
        t = {k: dev(v) for k, v in d.items()}
        ws = [torch.empty(max(m.workspace_size(p, shape), 16), dtype=torch.uint8, device="cuda")
              for p in (0, 1, 2)]
        data.append((shape, t, ws))
    seq = [[host(o) for o in _passes(*x)] for x in data]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    outs = [None, None]
    for rep in range(3):
        for i, (x, s) in enumerate(zip(data, streams)):
            with torch.cuda.stream(s):
                outs[i] = _passes(*x)
        torch.cuda.synchronize()
        for i in range(2):
            for a, b in zip(seq[i], outs[i]):
                got = host(b)
                assert np.array_equal(a.view(np.uint32), got.view(np.uint32)), (i, rep)


def test_bench_step_on_two_streams_matches_one():
    """The benchmark's step with backward-weight on a second stream writes
    bit for bit what the one-stream step writes, on the AlexNet-shaped
    network step at batch 4 (its pooling and inner-product layers included)."""
    import torch
    import bench
    import workloads
    cfg = 5
    _, layers = workloads.config(cfg)
    stream = torch.cuda.current_stream().cuda_stream
    runs = []
    for li, L in enumerate(layers):
        L = L.with_batch(4)
        runs.append(bench.PoolRun(cfg, li, L, stream) if isinstance(L, workloads.PoolLayer)
                    else bench.LayerRun(cfg, li, L, stream))

    def written(r):  # the first layer's dx is not computed by a step
        return [n for n in ("y", "dx", "dw", "db") if hasattr(r, n) and not (n == "dx" and r.L.first)]

    def outputs():
        return [host(getattr(r, n)).copy() for r in runs for n in written(r)]

    bench.stack_step(runs)
    torch.cuda.synchronize()
    ref = outputs()
    for r in runs:
        for n in written(r):
            getattr(r, n).fill_(float("nan"))
    side = torch.cuda.Stream()
    for r in runs:
        if isinstance(r, bench.LayerRun):
            r.bind_side(side.cuda_stream)
    for _ in range(2):
        bench.stack_step(runs, side)
    torch.cuda.synchronize()
    got = outputs()
    assert len(got) == len(ref) > 0
    for a, b in zip(ref, got):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
