"""Checks that pin the CPU oracle to facts outside itself.

Each ``check_*`` function takes an ``oracle.Oracle`` and raises
AssertionError when the oracle disagrees with something the paper or the
mathematics fixes: hand-computed cases, the GEMM special cases, the explicit
im2col + GEMM plan, an independent library convolution (torch, CPU, fp64),
the adjoint identity, exact finite differences of a linear map, delta
filters, and structural invariants.  ``test_oracle.py`` runs them on the
oracle as built; ``test_oracle_mutants.py`` runs them on deliberately broken
copies of the oracle to show that each plausible mistake is caught.

Semantics being pinned: Sec. IV-B of the paper (im2col + GEMM forward,
col2im in the backward pass, zero padding), Sec. IV-C layouts, Table II's
three passes; Caffe readings for rounding, groups and bias.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

# (N, C, H, W, K, R, S, stride, pad, group): strides 1-3, pads 0-2,
# groups 1-4, R != S, H != W, pad >= R, stride > R (uncovered input pixels),
# C/G = 1, filter covering the whole image.
SMALL_SHAPES = [
    (2, 4, 5, 6, 6, 3, 2, 2, 1, 2),
    (1, 3, 7, 7, 4, 3, 3, 1, 1, 1),
    (2, 6, 9, 8, 6, 5, 3, 3, 2, 3),
    (1, 2, 6, 6, 3, 1, 1, 2, 0, 1),
    (2, 2, 5, 5, 2, 2, 2, 3, 0, 1),
    (1, 2, 4, 5, 2, 1, 2, 1, 2, 2),
    (3, 4, 4, 4, 8, 4, 4, 1, 0, 4),
    (2, 3, 11, 10, 5, 4, 3, 2, 3, 1),
]


def _rand(shape, seed):
    """fp32 test arrays (values exactly representable, as on the GPU side)."""
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def _inputs(o, shape, seed=0):
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q = o.out_size(H, R, st, pad), o.out_size(W, S, st, pad)
    x = _rand((N, C, H, W), [seed, 0])
    w = _rand((K, C // G, R, S), [seed, 1])
    b = _rand((K,), [seed, 2])
    dy = _rand((N, K, P, Q), [seed, 3])
    return P, Q, x, w, b, dy


def _close(a, b, rtol=1e-12, atol=1e-12, what=""):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    err = np.abs(a - b)
    lim = atol + rtol * np.abs(b)
    assert np.all(err <= lim), f"{what}: max err {err.max()} (limit {lim.max()})"


# -------------------------------------------------------------- hand cases
def check_hand_cases(o):
    """Brute-force hand cases (tests/golden/hand_cases.json)."""
    cases = json.load(open(os.path.join(GOLDEN, "hand_cases.json")))["cases"]
    for c in cases:
        shape = c["shape"]
        N, C, H, W, K, R, S, st, pad, G = shape
        P, Q = o.out_size(H, R, st, pad), o.out_size(W, S, st, pad)
        x = np.array(c["x"], np.float32).reshape(N, C, H, W)
        w = np.array(c["w"], np.float32).reshape(K, C // G, R, S)
        b = None if c["b"] is None else np.array(c["b"], np.float32)
        dy = np.ones((N, K, P, Q), np.float32)
        y, _ = o.conv_fwd(shape, x, w, b)
        assert y.ravel().tolist() == c["y"], (c["name"], "y", y.ravel())
        dx, _ = o.conv_bwd_data(shape, dy, w)
        assert dx.ravel().tolist() == c["dx"], (c["name"], "dx", dx.ravel())
        dw, _, db, _ = o.conv_bwd_weight(shape, x, dy)
        assert dw.ravel().tolist() == c["dw"], (c["name"], "dw", dw.ravel())
        assert db.ravel().tolist() == c["db"], (c["name"], "db", db.ravel())


# --------------------------------------------------------------- geometry
OUT_SIZES = [
    # (in, filter, stride, pad, expected): AlexNet conv1 227 -> 55 (exact);
    # ResNet stem 224 -> 112 and 1x1 stride-2 56 -> 28 need floor rounding;
    # "same" 3x3 pad 1; 5x5 pad 2; window larger than the padded input -> 0.
    (227, 11, 4, 0, 55), (224, 7, 2, 3, 112), (56, 1, 2, 0, 28),
    (224, 3, 1, 1, 224), (27, 5, 1, 2, 27), (13, 3, 1, 1, 13), (4, 3, 2, 1, 2),
    (5, 2, 3, 0, 2), (3, 5, 1, 0, 0), (3, 5, 1, 1, 1), (1, 1, 1, 0, 1),
]


def check_out_size(o):
    for n_in, f, st, pad, want in OUT_SIZES:
        got = o.out_size(n_in, f, st, pad)
        assert got == want, (n_in, f, st, pad, got, want)


# ------------------------------------------------------ GEMM special cases
def check_gemm_1x1(o):
    """A 1x1, stride-1, unpadded conv is a per-image GEMM per group:
    y[n] = W x[n] + b, dx[n] = W^T dy[n], dW = sum_n dy[n] x[n]^T."""
    for shape in [(2, 6, 3, 5, 4, 1, 1, 1, 0, 1), (3, 6, 4, 2, 9, 1, 1, 1, 0, 3)]:
        N, C, H, W, K, _, _, _, _, G = shape
        P, Q, x, w, b, dy = _inputs(o, shape, 7)
        Cg, Kg = C // G, K // G
        X = x.astype(np.float64).reshape(N, C, H * W)
        D = dy.astype(np.float64).reshape(N, K, H * W)
        Wm = w.astype(np.float64).reshape(K, Cg)
        y_ref = np.empty((N, K, H * W))
        dx_ref = np.empty((N, C, H * W))
        dw_ref = np.empty((K, Cg))
        for g in range(G):
            ks, cs = slice(g * Kg, (g + 1) * Kg), slice(g * Cg, (g + 1) * Cg)
            y_ref[:, ks] = np.matmul(Wm[ks], X[:, cs])
            dx_ref[:, cs] = np.matmul(Wm[ks].T, D[:, ks])
            dw_ref[ks] = sum(D[n, ks] @ X[n, cs].T for n in range(N))
        y_ref += b.astype(np.float64)[None, :, None]
        y, _ = o.conv_fwd(shape, x, w, b)
        _close(y.reshape(N, K, -1), y_ref, what="1x1 fwd")
        dx, _ = o.conv_bwd_data(shape, dy, w)
        _close(dx.reshape(N, C, -1), dx_ref, what="1x1 bwd_data")
        dw, _, db, _ = o.conv_bwd_weight(shape, x, dy)
        _close(dw.reshape(K, Cg), dw_ref, what="1x1 bwd_weight")
        _close(db, D.sum(axis=(0, 2)), what="1x1 db")


def check_fully_connected(o):
    """A filter as large as the unpadded image gives P = Q = 1: a fully
    connected layer, y[n] = W_flat x_flat[n] + b."""
    shape = (3, 4, 3, 2, 5, 3, 2, 1, 0, 1)
    N, C, H, W, K = shape[:5]
    P, Q, x, w, b, dy = _inputs(o, shape, 11)
    assert (P, Q) == (1, 1)
    Wf = w.astype(np.float64).reshape(K, -1)
    Xf = x.astype(np.float64).reshape(N, -1)
    y, _ = o.conv_fwd(shape, x, w, b)
    _close(y.reshape(N, K), Xf @ Wf.T + b.astype(np.float64), what="fc fwd")
    Df = dy.astype(np.float64).reshape(N, K)
    dx, _ = o.conv_bwd_data(shape, dy, w)
    _close(dx.reshape(N, -1), Df @ Wf, what="fc bwd_data")
    dw, _, _, _ = o.conv_bwd_weight(shape, x, dy)
    _close(dw.reshape(K, -1), Df.T @ Xf, what="fc bwd_weight")


# ------------------------------------------------ explicit plan (im2col)
def _im2col(x, R, S, st, pad, P, Q):
    """x [C,H,W] -> columns [C*R*S, P*Q] (the explicit plan of Sec. IV-B)."""
    C = x.shape[0]
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad)))
    cols = np.empty((C, R, S, P, Q))
    for r in range(R):
        for s in range(S):
            cols[:, r, s] = xp[:, r:r + st * (P - 1) + 1:st, s:s + st * (Q - 1) + 1:st]
    return cols.reshape(C * R * S, P * Q)


def _col2im(cols, C, H, W, R, S, st, pad, P, Q):
    """Adjoint of _im2col: scatter-add the columns back into the image."""
    xp = np.zeros((C, H + 2 * pad, W + 2 * pad))
    c4 = cols.reshape(C, R, S, P, Q)
    for r in range(R):
        for s in range(S):
            xp[:, r:r + st * (P - 1) + 1:st, s:s + st * (Q - 1) + 1:st] += c4[:, r, s]
    return xp[:, pad:pad + H, pad:pad + W]


def check_im2col_plan(o):
    """Forward = filter matrix x im2col columns (+ bias); backward-data =
    col2im of W^T dy; backward-weight = dy x columns^T, per image and group."""
    for seed, shape in enumerate(SMALL_SHAPES):
        N, C, H, W, K, R, S, st, pad, G = shape
        P, Q, x, w, b, dy = _inputs(o, shape, 100 + seed)
        Cg, Kg = C // G, K // G
        Wm = w.astype(np.float64).reshape(K, Cg * R * S)
        y_ref = np.empty((N, K, P * Q))
        dx_ref = np.empty((N, C, H, W))
        dw_ref = np.zeros((K, Cg * R * S))
        for n in range(N):
            for g in range(G):
                ks, cs = slice(g * Kg, (g + 1) * Kg), slice(g * Cg, (g + 1) * Cg)
                cols = _im2col(x[n, cs].astype(np.float64), R, S, st, pad, P, Q)
                d = dy[n, ks].astype(np.float64).reshape(Kg, P * Q)
                y_ref[n, ks] = Wm[ks] @ cols
                dx_ref[n, cs] = _col2im(Wm[ks].T @ d, Cg, H, W, R, S, st, pad, P, Q)
                dw_ref[ks] += d @ cols.T
        y_ref += b.astype(np.float64)[None, :, None]
        y, _ = o.conv_fwd(shape, x, w, b)
        _close(y.reshape(N, K, -1), y_ref, what=f"im2col fwd {shape}")
        dx, _ = o.conv_bwd_data(shape, dy, w)
        _close(dx, dx_ref, what=f"col2im bwd_data {shape}")
        dw, _, _, _ = o.conv_bwd_weight(shape, x, dy)
        _close(dw.reshape(K, -1), dw_ref, what=f"im2col bwd_weight {shape}")


# --------------------------------------------- independent library (torch)
def check_torch_cpu(o):
    """torch's CPU fp64 conv2d and its autograd gradients (an independent
    implementation of the same layer) agree with the oracle, including the
    abs-sums: conv of |x| with |w| plus |b|, and likewise for the grads."""
    import torch
    F = torch.nn.functional
    for seed, shape in enumerate(SMALL_SHAPES):
        N, C, H, W, K, R, S, st, pad, G = shape
        P, Q, x, w, b, dy = _inputs(o, shape, 200 + seed)
        tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
        tw = torch.tensor(w, dtype=torch.float64, requires_grad=True)
        tb = torch.tensor(b, dtype=torch.float64, requires_grad=True)
        ty = F.conv2d(tx, tw, tb, stride=st, padding=pad, groups=G)
        ty.backward(torch.tensor(dy, dtype=torch.float64))
        y, ay = o.conv_fwd(shape, x, w, b)
        _close(y, ty.detach().numpy(), what=f"torch fwd {shape}")
        dx, adx = o.conv_bwd_data(shape, dy, w)
        _close(dx, tx.grad.numpy(), what=f"torch dx {shape}")
        dw, adw, db, adb = o.conv_bwd_weight(shape, x, dy)
        _close(dw, tw.grad.numpy(), what=f"torch dw {shape}")
        _close(db, tb.grad.numpy(), what=f"torch db {shape}")
        ax = torch.tensor(np.abs(x), dtype=torch.float64, requires_grad=True)
        aw = torch.tensor(np.abs(w), dtype=torch.float64, requires_grad=True)
        ab = torch.tensor(np.abs(b), dtype=torch.float64)
        ayt = F.conv2d(ax, aw, ab, stride=st, padding=pad, groups=G)
        ayt.backward(torch.tensor(np.abs(dy), dtype=torch.float64))
        _close(ay, ayt.detach().numpy(), what=f"abs-sum y {shape}")
        _close(adx, ax.grad.numpy(), what=f"abs-sum dx {shape}")
        _close(adw, aw.grad.numpy(), what=f"abs-sum dw {shape}")
        _close(adb, np.abs(dy).astype(np.float64).sum(axis=(0, 2, 3)), what="abs-sum db")


# -------------------------------------------------------------- identities
def check_adjoint(o):
    """<conv(x,w), dy> = <x, bwd_data(dy,w)> = <w, bwd_weight(x,dy)>."""
    for seed, shape in enumerate(SMALL_SHAPES):
        P, Q, x, w, b, dy = _inputs(o, shape, 300 + seed)
        y, _ = o.conv_fwd(shape, x, w, None)
        dx, _ = o.conv_bwd_data(shape, dy, w)
        dw, _, _, _ = o.conv_bwd_weight(shape, x, dy)
        d = dy.astype(np.float64)
        l0 = float(np.sum(y * d))
        l1 = float(np.sum(x.astype(np.float64) * dx))
        l2 = float(np.sum(w.astype(np.float64) * dw))
        scale = float(np.sum(np.abs(y * d))) + 1e-300
        assert abs(l0 - l1) <= 1e-12 * scale, (shape, l0, l1)
        assert abs(l0 - l2) <= 1e-12 * scale, (shape, l0, l2)


def check_finite_differences(o):
    """L(x, w, b) = <conv(x,w)+b, dy> is linear in each argument, so central
    differences have no truncation error: they equal dx, dw and db up to
    fp64 rounding."""
    eps = 1e-3
    rng = np.random.default_rng(5)
    for seed, shape in enumerate(SMALL_SHAPES[:5]):
        P, Q, x, w, b, dy = _inputs(o, shape, 400 + seed)
        d = dy.astype(np.float64)

        def L(xx, ww, bb):
            yy, _ = o.conv_fwd(shape, xx, ww, bb)
            return float(np.sum(yy * d))

        x64, w64, b64 = (a.astype(np.float64) for a in (x, w, b))
        dx, _ = o.conv_bwd_data(shape, dy, w)
        dw, _, db, _ = o.conv_bwd_weight(shape, x, dy)
        for arr, grad, which in ((x64, dx, 0), (w64, dw, 1), (b64, db, 2)):
            for flat in rng.choice(arr.size, size=min(arr.size, 6), replace=False):
                plus, minus = arr.copy(), arr.copy()
                plus.flat[flat] += eps
                minus.flat[flat] -= eps
                args_p = [x64, w64, b64]
                args_m = [x64, w64, b64]
                args_p[which], args_m[which] = plus, minus
                fd = (L(*args_p) - L(*args_m)) / (2 * eps)
                g = grad.flat[flat]
                assert abs(fd - g) <= 1e-8 * (1 + abs(g)), (shape, which, flat, fd, g)


def check_delta_filter(o):
    """A filter with one unit tap copies a shifted input (zeros where the
    shift leaves the image); its backward-data copies dy back."""
    N, C, H, W, K, R, S, st, pad = 2, 3, 6, 7, 3, 3, 3, 1, 1
    shape = (N, C, H, W, K, R, S, st, pad, 1)
    P, Q, x, _, _, dy = _inputs(o, shape, 500)
    r0, s0 = 2, 0
    w = np.zeros((K, C, R, S), np.float32)
    perm = [2, 0, 1]                         # y channel k copies x channel perm[k]
    for k in range(K):
        w[k, perm[k], r0, s0] = 1.0
    y, _ = o.conv_fwd(shape, x, w, None)
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    for k in range(K):
        want = xp[:, perm[k], r0:r0 + P, s0:s0 + Q]
        assert np.array_equal(y[:, k], want.astype(np.float64)), k
    dx, _ = o.conv_bwd_data(shape, dy, w)
    for k in range(K):
        buf = np.zeros((N, H + 2 * pad, W + 2 * pad))
        buf[:, r0:r0 + P, s0:s0 + Q] = dy[:, k]
        assert np.array_equal(dx[:, perm[k]], buf[:, pad:pad + H, pad:pad + W]), k


def check_group_split(o):
    """A G-group conv equals G independent convs on channel slices."""
    shape = (2, 6, 7, 6, 9, 3, 2, 2, 1, 3)
    N, C, H, W, K, R, S, st, pad, G = shape
    P, Q, x, w, b, dy = _inputs(o, shape, 600)
    y, _ = o.conv_fwd(shape, x, w, b)
    dx, _ = o.conv_bwd_data(shape, dy, w)
    dw, _, db, _ = o.conv_bwd_weight(shape, x, dy)
    Cg, Kg = C // G, K // G
    sub = (N, Cg, H, W, Kg, R, S, st, pad, 1)
    for g in range(G):
        cs, ks = slice(g * Cg, (g + 1) * Cg), slice(g * Kg, (g + 1) * Kg)
        ys, _ = o.conv_fwd(sub, x[:, cs], w[ks], b[ks])
        assert np.array_equal(ys, y[:, ks]), g
        dxs, _ = o.conv_bwd_data(sub, dy[:, ks], w[ks])
        assert np.array_equal(dxs, dx[:, cs]), g
        dws, _, dbs, _ = o.conv_bwd_weight(sub, x[:, cs], dy[:, ks])
        assert np.array_equal(dws, dw[ks]) and np.array_equal(dbs, db[ks]), g


def check_translation(o):
    """At stride 1, shifting the input shifts the output (away from borders)."""
    shape = (1, 2, 9, 10, 3, 3, 3, 1, 0, 1)
    P, Q, x, w, _, _ = _inputs(o, shape, 700)
    xs = np.zeros_like(x)
    xs[:, :, 1:, 2:] = x[:, :, :-1, :-2]
    y, _ = o.conv_fwd(shape, x, w, None)
    ys, _ = o.conv_fwd(shape, xs, w, None)
    _close(ys[:, :, 1 + 2:, 2 + 2:], y[:, :, 2:-1, 2:-2], what="translation")


def check_gather_matches_scatter(o):
    """Per-element gather forms equal the full scatter forms everywhere."""
    for seed, shape in enumerate(SMALL_SHAPES):
        P, Q, x, w, b, dy = _inputs(o, shape, 800 + seed)
        y, ay = o.conv_fwd(shape, x, w, b)
        v, av = o.conv_fwd_at(shape, x, w, b, np.arange(y.size))
        _close(v, y.ravel(), what="fwd_at")
        _close(av, ay.ravel(), what="fwd_at abs")
        dx, adx = o.conv_bwd_data(shape, dy, w)
        v, av = o.conv_bwd_data_at(shape, dy, w, np.arange(dx.size))
        _close(v, dx.ravel(), what=f"bwd_data_at {shape}")
        _close(av, adx.ravel(), what="bwd_data_at abs")
        dw, adw, db, adb = o.conv_bwd_weight(shape, x, dy)
        v, av = o.conv_bwd_weight_at(shape, x, dy, np.arange(dw.size))
        _close(v, dw.ravel(), what="bwd_weight_at")
        _close(av, adw.ravel(), what="bwd_weight_at abs")
        v, av = o.bias_grad(dy)
        _close(v, db, what="bias_grad")
        _close(av, adb, what="bias_grad abs")


ALL_CHECKS = [
    check_hand_cases, check_out_size, check_gemm_1x1, check_fully_connected,
    check_im2col_plan, check_torch_cpu, check_adjoint, check_finite_differences,
    check_delta_filter, check_group_split, check_translation,
    check_gather_matches_scatter,
]
