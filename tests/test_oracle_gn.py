"""Pins of the oracle's GroupNorm, SiLU and timestep projection: invariants,
special cases that reduce to other norms, torch fp64 and finite differences."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pulse_oracle as O


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("C,G", [(12, 3), (8, 8), (6, 1), (30, 10)])
def test_gn_normalised_moments(C, G):
    x = 3.0 + 2.0 * _rand((2, 5, 4, C), 1)
    eps = 1e-5
    z, (xhat, rstd) = O.group_norm_fwd(x, np.ones(C), np.zeros(C), G, eps)
    xg = xhat.reshape(2, 20, G, C // G)
    assert np.abs(xg.mean(axis=(1, 3))).max() < 1e-12
    v = x.reshape(2, 20, G, C // G).var(axis=(1, 3))
    np.testing.assert_allclose(xg.var(axis=(1, 3)), v / (v + eps), rtol=1e-12)
    np.testing.assert_array_equal(z, xhat)


def test_gn_groups_equal_channels_is_instance_norm():
    x = _rand((2, 4, 5, 6), 2)
    z, _ = O.group_norm_fwd(x, np.ones(6), np.zeros(6), 6, 1e-5)
    ref = F.instance_norm(torch.tensor(x).permute(0, 3, 1, 2), eps=1e-5)
    np.testing.assert_allclose(z, ref.permute(0, 2, 3, 1).numpy(), rtol=1e-10, atol=1e-12)


def test_gn_one_group_is_layer_norm():
    x = _rand((3, 4, 5, 6), 3)
    z, _ = O.group_norm_fwd(x, np.ones(6), np.zeros(6), 1, 1e-5)
    ref = F.layer_norm(torch.tensor(x), (4, 5, 6), eps=1e-5)
    np.testing.assert_allclose(z, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_gn_fwd_bwd_against_torch():
    C, G = 12, 4
    x = _rand((2, 3, 5, C), 4)
    ga = 1 + 0.1 * _rand(C, 5)
    be = 0.1 * _rand(C, 6)
    g = _rand((2, 3, 5, C), 7)
    xt = torch.tensor(x).permute(0, 3, 1, 2).requires_grad_(True)
    gat = torch.tensor(ga).requires_grad_(True)
    bet = torch.tensor(be).requires_grad_(True)
    zt = F.group_norm(xt, G, gat, bet, eps=1e-5)
    zt.backward(torch.tensor(g).permute(0, 3, 1, 2))
    z, aux = O.group_norm_fwd(x, ga, be, G, 1e-5)
    dx, dga, dbe = O.group_norm_bwd(g, aux, ga, G)
    np.testing.assert_allclose(z, zt.permute(0, 2, 3, 1).detach().numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dga, gat.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dbe, bet.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_gn_backward_invariants():
    C, G = 12, 3
    x = _rand((2, 4, 4, C), 8)
    ga = 1 + 0.1 * _rand(C, 9)
    g = _rand((2, 4, 4, C), 10)
    # sum over a group of dx vanishes for any eps
    _, aux = O.group_norm_fwd(x, ga, np.zeros(C), G, 1e-5)
    dx, _, _ = O.group_norm_bwd(g, aux, ga, G)
    assert np.abs(dx.reshape(2, 16, G, 4).sum(axis=(1, 3))).max() < 1e-12
    # with eps = 0 the sum of dx * xhat vanishes too
    _, aux0 = O.group_norm_fwd(x, ga, np.zeros(C), G, 0.0)
    dx0, _, _ = O.group_norm_bwd(g, aux0, ga, G)
    s = (dx0 * aux0[0]).reshape(2, 16, G, 4).sum(axis=(1, 3))
    assert np.abs(s).max() < 1e-11


def test_gn_backward_finite_difference():
    C, G = 6, 2
    x = _rand((1, 3, 3, C), 11)
    ga = 1 + 0.1 * _rand(C, 12)
    be = 0.1 * _rand(C, 13)
    g = _rand((1, 3, 3, C), 14)
    _, aux = O.group_norm_fwd(x, ga, be, G, 1e-5)
    dx, dga, dbe = O.group_norm_bwd(g, aux, ga, G)
    h = 1e-6
    f = lambda xx, gg, bb: np.sum(g * O.group_norm_fwd(xx, gg, bb, G, 1e-5)[0])
    for idx in [(0, 0, 0, 0), (0, 1, 2, 3), (0, 2, 1, 5)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        assert abs((f(xp, ga, be) - f(xm, ga, be)) / (2 * h) - dx[idx]) < 1e-7
    for c in range(C):
        gp, gm = ga.copy(), ga.copy()
        gp[c] += h
        gm[c] -= h
        assert abs((f(x, gp, be) - f(x, gm, be)) / (2 * h) - dga[c]) < 1e-7


def test_silu_identities():
    assert O.silu(0.0) == 0.0
    assert O.silu_grad(0.0) == 0.5
    x = _rand(50, 15) * 4
    np.testing.assert_allclose(O.silu(x) - O.silu(-x), x, rtol=1e-13, atol=1e-14)
    h = 1e-6
    np.testing.assert_allclose((O.silu(x + h) - O.silu(x - h)) / (2 * h), O.silu_grad(x), atol=1e-8)
    np.testing.assert_allclose(O.silu(x), F.silu(torch.tensor(x)).numpy(), rtol=1e-13)


def test_temb_projection_against_torch():
    rng = np.random.default_rng(16)
    temb = rng.standard_normal((3, 8))
    wl = rng.standard_normal((5, 8))
    bl = rng.standard_normal(5)
    de = rng.standard_normal((3, 5))
    tt = torch.tensor(temb).requires_grad_(True)
    wt = torch.tensor(wl).requires_grad_(True)
    bt = torch.tensor(bl).requires_grad_(True)
    e = F.linear(F.silu(tt), wt, bt)
    e.backward(torch.tensor(de))
    np.testing.assert_allclose(O.temb_fwd(temb, wl, bl), e.detach().numpy(), rtol=1e-12)
    dwl, dbl, dtemb = O.temb_bwd(de, temb, wl)
    np.testing.assert_allclose(dwl, wt.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(dbl, bt.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(dtemb, tt.grad.numpy(), rtol=1e-11, atol=1e-13)
