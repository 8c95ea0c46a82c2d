"""Helpers for the GPU tests: run the HIP passes through the C-ABI binding
on numpy inputs, and compare with the oracle to the per-element bound
|gpu - ref| <= 1e-4 * sum|products| (elements whose abs-sum is 0 must be
exactly 0)."""
from __future__ import annotations

import numpy as np

REL_TOL = 1e-4


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def gpu_fwd(shape, x, w, b):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    return host(m.conv_fwd(dev(x), dev(w), None if b is None else dev(b), st, pad, G))


def gpu_bwd_data(shape, dy, w):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    return host(m.conv_bwd_data(dev(dy), dev(w), (H, W), st, pad, G))


def gpu_bwd_weight(shape, x, dy, with_bias=True):
    import paper_1903_06934_amd as m
    N, C, H, W, K, R, S, st, pad, G = shape
    dw, db = m.conv_bwd_weight(dev(x), dev(dy), (R, S), st, pad, G, with_bias=with_bias)
    return host(dw), (host(db) if db is not None else None)


def assert_within(got, ref, absum, what, rel=REL_TOL):
    got = np.asarray(got, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    absum = np.asarray(absum, np.float64).ravel()
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    zero = absum == 0
    bad_zero = zero & (got != 0)
    assert not bad_zero.any(), f"{what}: {bad_zero.sum()} elements must be exactly 0"
    err = np.abs(got - ref)
    lim = rel * absum
    bad = err > lim
    if bad.any():
        i = int(np.argmax(err - lim))
        raise AssertionError(
            f"{what}: {bad.sum()}/{bad.size} elements out of tolerance; worst flat "
            f"index {i}: gpu {got[i]!r} ref {ref[i]!r} err {err[i]:.3e} limit {lim[i]:.3e}")
    return float(np.max(err / np.where(zero, 1, absum))) if err.size else 0.0


def sample_indices(dims, rng, count=2048, groups=1, channel_axis=1):
    """Flat indices into a row-major tensor of shape ``dims`` (4-D): random
    positions plus every border row and column of a few (n, channel) planes,
    the first and last channel and each group's first and last channel."""
    dims = tuple(int(d) for d in dims)
    total = int(np.prod(dims))
    if total <= count:
        return np.arange(total, dtype=np.int64)
    a, b, h, w = dims
    picks = [rng.integers(0, total, size=count)]
    cb = b // groups if channel_axis == 1 else None
    chans = {0, b - 1}
    if cb:
        for g in range(groups):
            chans |= {g * cb, (g + 1) * cb - 1}
    firsts = [(0, c) for c in sorted(chans)] + [(a - 1, b - 1), (int(rng.integers(a)), int(rng.integers(b)))]
    for i0, i1 in firsts:
        base = (i0 * b + i1) * h * w
        ring = set()
        for y in range(h):
            ring |= {y * w, y * w + w - 1}
        for x in range(w):
            ring |= {x, (h - 1) * w + x}
        picks.append(base + np.fromiter(sorted(ring), dtype=np.int64))
    out = np.unique(np.concatenate(picks).astype(np.int64))
    return out


# Filter gradients with at most this many elements are checked in full at
# every batch; larger ones on sampled elements.
FULL_DW_ELEMS = 65536


def dw_indices(dw_shape, npq, rng):
    """Flat dw indices to compare with the oracle's gather form: all of them
    when dw has at most FULL_DW_ELEMS elements, else a sample (every filter's
    first and last input channel included) sized to the reduction length npq
    (the products per element)."""
    size = int(np.prod(dw_shape))
    if size <= FULL_DW_ELEMS:
        return np.arange(size, dtype=np.int64)
    count = int(min(2048, max(128, 1e9 / npq)))
    return sample_indices(dw_shape, rng, count=count, groups=1, channel_axis=0)
