"""The passes launch kernels only (no allocation, synchronisation or memset),
so a caller can capture them into a HIP graph.  Each test captures the three
passes of a layer on torch's capture stream, replays the graph several
times with eager work and synchronisation in between (outputs cleared by a
fill kernel), and checks every replay bit for bit against the eager calls."""
import numpy as np
import pytest

import workloads
from gpu_util import dev

pytestmark = pytest.mark.gpu

GRAPH_SHAPES = [
    (2, 32, 24, 24, 48, 3, 3, 1, 1, 1),    # plain image GEMM, tap-uniform backward-weight
    (2, 64, 12, 12, 32, 5, 5, 1, 2, 1),    # forward split-K candidate (set below)
    (2, 3, 35, 33, 24, 11, 11, 4, 2, 1),   # blocked backward-data, packed-column backward-weight
]


def _passes(m, shape, t, out, ws, stream):
    N, C, H, W, K, R, S, st, pad, G = shape
    L = m.lib()
    assert L.conv_fwd(*shape, t["x"].data_ptr(), t["w"].data_ptr(), t["b"].data_ptr(),
                      out["y"].data_ptr(), ws[0].data_ptr(), ws[0].numel(), stream) == 0
    assert L.conv_bwd_data(*shape, t["dy"].data_ptr(), t["w"].data_ptr(), out["dx"].data_ptr(),
                           ws[1].data_ptr(), ws[1].numel(), stream) == 0
    assert L.conv_bwd_weight(*shape, t["x"].data_ptr(), t["dy"].data_ptr(), out["dw"].data_ptr(),
                             out["db"].data_ptr(), ws[2].data_ptr(), ws[2].numel(), stream) == 0


@pytest.mark.parametrize("shape", GRAPH_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_passes_replay_in_a_graph(shape):
    import torch
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = m.output_size(H, W, R, S, st, pad)
    d = workloads.make_inputs(shape, P, Q, seed=(55, C))
    t = {k: dev(v) for k, v in d.items()}
    m.plan_clear()
    try:
        if shape[1] == 64:   # take a split-K forward plan: partial slabs plus a reduction kernel
            names = [m.plan_name(0, shape, i) for i in range(m.plan_count(0, shape))]
            m.plan_set(0, shape, next(i for i, s in enumerate(names) if "splits" in s))
        ws = [torch.empty(max(m.workspace_size(p, shape), 16), dtype=torch.uint8, device="cuda")
              for p in range(3)]
        out = {"y": torch.empty((N, K, P, Q), device="cuda"),
               "dx": torch.empty((N, C, H, W), device="cuda"),
               "dw": torch.empty((K, C // G, R, S), device="cuda"),
               "db": torch.empty((K,), device="cuda")}
        _passes(m, shape, t, out, ws, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        eager = {k: v.clone() for k, v in out.items()}

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            _passes(m, shape, t, out, ws, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for rep in range(3):
            for v in out.values():
                v.fill_(float("nan"))
            junk = torch.randn(512, 512, device="cuda") @ torch.randn(512, 512, device="cuda")
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for k in out:
                a = out[k].cpu().numpy().view(np.uint32)
                b = eager[k].cpu().numpy().view(np.uint32)
                assert np.array_equal(a, b), (rep, k)
            del junk
    finally:
        m.plan_clear()
