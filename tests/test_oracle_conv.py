"""Pins of the oracle's convolutions against things other than itself:
brute-force direct sums, closed forms, adjoint identities and torch fp64."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pulse_oracle as O


def _brute_conv3x3(a, w, b):
    B, H, W, I = a.shape
    Oc = w.shape[0]
    y = np.zeros((B, H, W, Oc))
    for n in range(B):
        for h in range(H):
            for x in range(W):
                for o in range(Oc):
                    s = float(b[o])
                    for dy in range(3):
                        for dx in range(3):
                            hh, ww = h + dy - 1, x + dx - 1
                            if 0 <= hh < H and 0 <= ww < W:
                                for i in range(I):
                                    s += float(w[o, dy, dx, i]) * float(a[n, hh, ww, i])
                    y[n, h, x, o] = s
    return y


def _brute_conv1x1(a, w, b):
    B, H, W, I = a.shape
    Oc = w.shape[0]
    y = np.zeros((B, H, W, Oc))
    for n in range(B):
        for h in range(H):
            for x in range(W):
                for o in range(Oc):
                    y[n, h, x, o] = b[o] + sum(w[o, i] * a[n, h, x, i] for i in range(I))
    return y


def test_conv3x3_brute_force():
    rng = np.random.default_rng(11)
    a = rng.standard_normal((2, 5, 4, 3))
    w = rng.standard_normal((2, 3, 3, 3))
    b = rng.standard_normal(2)
    np.testing.assert_allclose(O.conv3x3_fwd(a, w, b), _brute_conv3x3(a, w, b), rtol=0, atol=1e-12)


def test_conv1x1_brute_force():
    rng = np.random.default_rng(12)
    a = rng.standard_normal((1, 3, 4, 5))
    w = rng.standard_normal((3, 5))
    b = rng.standard_normal(3)
    np.testing.assert_allclose(O.conv1x1_fwd(a, w, b), _brute_conv1x1(a, w, b), rtol=0, atol=1e-12)


def test_conv3x3_delta_kernel_is_identity():
    rng = np.random.default_rng(13)
    C = 4
    a = rng.standard_normal((2, 6, 7, C))
    w = np.zeros((C, 3, 3, C))
    w[:, 1, 1, :] = np.eye(C)
    b = np.arange(C, dtype=float)
    np.testing.assert_array_equal(O.conv3x3_fwd(a, w, b), a + b)


def test_conv3x3_all_ones_counts_the_padding():
    # interior pixels see 9 taps, edge pixels 6, corner pixels 4
    I, Oc = 3, 2
    a = np.ones((1, 5, 6, I))
    w = np.ones((Oc, 3, 3, I))
    y = O.conv3x3_fwd(a, w, np.zeros(Oc))
    expect = np.full((5, 6), 9.0 * I)
    expect[0, :] = expect[-1, :] = expect[:, 0] = expect[:, -1] = 6.0 * I
    for h in (0, -1):
        for x in (0, -1):
            expect[h, x] = 4.0 * I
    for o in range(Oc):
        np.testing.assert_array_equal(y[0, :, :, o], expect)


def test_conv3x3_shifted_delta_moves_the_image():
    # tap (dy, dx) = (0, 2) reads a[h-1, w+1]
    rng = np.random.default_rng(14)
    a = rng.standard_normal((1, 5, 5, 1))
    w = np.zeros((1, 3, 3, 1))
    w[0, 0, 2, 0] = 1.0
    y = O.conv3x3_fwd(a, w, np.zeros(1))
    expect = np.zeros_like(a)
    expect[0, 1:, :-1, 0] = a[0, :-1, 1:, 0]
    np.testing.assert_array_equal(y, expect)


@pytest.mark.parametrize("shape", [(2, 5, 4, 3, 2), (1, 1, 1, 4, 3), (1, 2, 7, 2, 5)])
def test_conv3x3_adjoint_identities(shape):
    B, H, W, I, Oc = shape
    rng = np.random.default_rng(15)
    a = rng.standard_normal((B, H, W, I))
    w = rng.standard_normal((Oc, 3, 3, I))
    g = rng.standard_normal((B, H, W, Oc))
    y = O.conv3x3_fwd(a, w, np.zeros(Oc))
    lhs = np.sum(g * y)
    da = O.conv3x3_dgrad(g, w)
    dw, db = O.conv3x3_wgrad(g, a)
    assert abs(np.sum(da * a) - lhs) <= 1e-12 * max(1.0, abs(lhs)) * 10
    assert abs(np.sum(dw * w) - lhs) <= 1e-12 * max(1.0, abs(lhs)) * 10
    np.testing.assert_allclose(db, g.sum(axis=(0, 1, 2)), rtol=1e-13)


def test_conv1x1_adjoint_identities():
    rng = np.random.default_rng(16)
    a = rng.standard_normal((2, 3, 5, 4))
    w = rng.standard_normal((6, 4))
    g = rng.standard_normal((2, 3, 5, 6))
    lhs = np.sum(g * O.conv1x1_fwd(a, w, np.zeros(6)))
    dw, db = O.conv1x1_wgrad(g, a)
    assert abs(np.sum(O.conv1x1_dgrad(g, w) * a) - lhs) <= 1e-11
    assert abs(np.sum(dw * w) - lhs) <= 1e-11


def test_conv3x3_dgrad_brute_force():
    # da[n,h,w,i] = sum w[o,dy,dx,i] * g[n,h-dy+1,w-dx+1,o] written out
    rng = np.random.default_rng(17)
    B, H, W, I, Oc = 1, 4, 3, 2, 3
    g = rng.standard_normal((B, H, W, Oc))
    w = rng.standard_normal((Oc, 3, 3, I))
    da = np.zeros((B, H, W, I))
    for h in range(H):
        for x in range(W):
            for i in range(I):
                s = 0.0
                for o in range(Oc):
                    for dy in range(3):
                        for dx in range(3):
                            hh, ww = h - dy + 1, x - dx + 1
                            if 0 <= hh < H and 0 <= ww < W:
                                s += w[o, dy, dx, i] * g[0, hh, ww, o]
                da[0, h, x, i] = s
    np.testing.assert_allclose(O.conv3x3_dgrad(g, w), da, rtol=0, atol=1e-12)


def test_conv_against_torch_fp64():
    rng = np.random.default_rng(18)
    a = rng.standard_normal((2, 7, 6, 5))
    w = rng.standard_normal((4, 3, 3, 5))
    b = rng.standard_normal(4)
    at = torch.tensor(a).permute(0, 3, 1, 2).requires_grad_(True)
    wt = torch.tensor(w).permute(0, 3, 1, 2).contiguous().requires_grad_(True)
    bt = torch.tensor(b).requires_grad_(True)
    yt = F.conv2d(at, wt, bt, padding=1)
    np.testing.assert_allclose(O.conv3x3_fwd(a, w, b), yt.permute(0, 2, 3, 1).detach().numpy(),
                               rtol=1e-12, atol=1e-12)
    g = rng.standard_normal((2, 7, 6, 4))
    yt.backward(torch.tensor(g).permute(0, 3, 1, 2))
    dw, db = O.conv3x3_wgrad(g, a)
    np.testing.assert_allclose(O.conv3x3_dgrad(g, w), at.grad.permute(0, 2, 3, 1).numpy(),
                               rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12)
