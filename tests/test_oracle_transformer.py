"""Pins of the transformer-stage oracle (oracle/transformer_oracle.py):
torch fp64 autograd of an independently written block and stage, central
finite differences, and closed-form special cases of LayerNorm, GELU and
attention."""

import math

import numpy as np
import pytest
import torch

from oracle import transformer_oracle as T
from paper_2606_19163_amd import configs, synth


def _desc(**kw):
    d = configs.t_tiny()
    d.update(dtype=configs.F32, **kw)
    return d


def _torch_block(x, p, heads, eps):
    """The pre-norm block written with torch's own ops."""
    import torch.nn.functional as F
    B, L, C = x.shape
    d = C // heads
    a = F.layer_norm(x, (C,), p["ln1.g"], p["ln1.b"], eps)
    qkv = F.linear(a, p["qkv.W"], p["qkv.b"])
    q, k, v = qkv.split(C, dim=-1)
    sh = lambda t: t.reshape(B, L, heads, d).transpose(1, 2)
    att = torch.softmax(sh(q) @ sh(k).transpose(-1, -2) / math.sqrt(d), dim=-1) @ sh(v)
    h = x + F.linear(att.transpose(1, 2).reshape(B, L, C), p["proj.W"], p["proj.b"])
    a2 = F.layer_norm(h, (C,), p["ln2.g"], p["ln2.b"], eps)
    m = F.gelu(F.linear(a2, p["fc1.W"], p["fc1.b"]), approximate="none")
    return h + F.linear(m, p["fc2.W"], p["fc2.b"])


def _torch_stage(desc, params, b):
    P = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in params.items()}
    x = torch.tensor(b["x"], dtype=torch.float64, requires_grad=True)
    u = torch.tensor(b["u"], dtype=torch.float64, requires_grad=True)
    H, eps, ne = desc["heads"], desc["eps"], desc["n_enc"]
    sub = lambda pre: {k[len(pre):]: v for k, v in P.items() if k.startswith(pre)}
    h, skips = x, []
    for k in range(ne):
        h = _torch_block(h, sub(f"enc{k}."), H, eps)
        skips.append(h)
    v = u
    for k in range(desc["n_dec"]):
        p = sub(f"dec{k}.")
        s = torch.nn.functional.linear(torch.cat([v, skips[ne - 1 - k]], dim=-1), p["skip.W"],
                                       p["skip.b"])
        v = _torch_block(s, p, H, eps)
    loss = (h * torch.tensor(b["g_enc"], dtype=torch.float64)).sum() + \
        (v * torch.tensor(b["g_dec"], dtype=torch.float64)).sum()
    loss.backward()
    return h.detach().numpy(), v.detach().numpy(), x.grad.numpy(), u.grad.numpy(), \
        {k: t.grad.numpy() for k, t in P.items()}


@pytest.mark.parametrize("ne,nd", [(1, 1), (2, 2), (2, 1)])
def test_stage_matches_torch_autograd(ne, nd):
    desc = _desc(n_enc=ne, n_dec=nd)
    params, b = synth.make_tstage(desc, 3)
    r = T.tstage_run(desc, params, b["x"], b["u"], b["g_enc"], b["g_dec"])
    ye, yd, dx, du, g = _torch_stage(desc, params, b)
    np.testing.assert_allclose(r["y_enc"], ye, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(r["y_dec"], yd, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(r["dx"], dx, rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(r["du"], du, rtol=1e-9, atol=1e-9)
    assert set(r["grads"]) == set(g)
    for k in g:
        np.testing.assert_allclose(r["grads"][k], g[k], rtol=1e-9, atol=1e-9, err_msg=k)
    fo = T.tstage_forward_only(desc, params, b["x"], b["u"])
    np.testing.assert_allclose(fo["y_dec"], r["y_dec"], rtol=0, atol=0)


def test_finite_differences():
    desc = _desc(batch=1, tokens=5, width=8, heads=2)
    params, b = synth.make_tstage(desc, 11)
    params = {k: v.astype(np.float64) for k, v in params.items()}
    r = T.tstage_run(desc, params, b["x"], b["u"], b["g_enc"], b["g_dec"])

    def loss(pp, x, u):
        f = T.tstage_forward_only(desc, pp, x, u)
        return float((f["y_enc"] * b["g_enc"]).sum() + (f["y_dec"] * b["g_dec"]).sum())

    rng = np.random.default_rng(0)
    eps = 1e-6
    x = b["x"].astype(np.float64)
    u = b["u"].astype(np.float64)
    for _ in range(6):
        i = tuple(rng.integers(0, s) for s in x.shape)
        for arr, grad, name in ((x, r["dx"], "x"), (u, r["du"], "u")):
            a0 = arr[i]
            arr[i] = a0 + eps
            lp = loss(params, x, u)
            arr[i] = a0 - eps
            lm = loss(params, x, u)
            arr[i] = a0
            assert (lp - lm) / (2 * eps) == pytest.approx(grad[i], rel=1e-5, abs=1e-7), name
    for name in ("enc0.qkv.W", "enc0.ln2.g", "dec0.skip.W", "dec0.fc1.b", "dec0.proj.W"):
        w = params[name]
        j = tuple(rng.integers(0, s) for s in w.shape)
        w0 = w[j]
        w[j] = w0 + eps
        lp = loss(params, x, u)
        w[j] = w0 - eps
        lm = loss(params, x, u)
        w[j] = w0
        assert (lp - lm) / (2 * eps) == pytest.approx(r["grads"][name][j], rel=1e-5, abs=1e-7), name


def test_layer_norm_invariants():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 7, 24)) * 3 + 2
    y, (xh, rstd) = T.layer_norm_fwd(x, np.ones(24), np.zeros(24), 1e-5)
    np.testing.assert_allclose(y.mean(axis=-1), 0, atol=1e-12)
    v = x.var(axis=-1)
    np.testing.assert_allclose(y.var(axis=-1), v / (v + 1e-5), rtol=1e-12)
    dy, g = rng.standard_normal(y.shape), rng.standard_normal(24)
    dx, dg, db = T.layer_norm_bwd(dy, (xh, rstd), g)
    # the output ignores a shift of a token: the gradient sums to zero
    np.testing.assert_allclose(dx.sum(axis=-1), 0, atol=1e-10)
    # with eps = 0 it also ignores a scaling: the gradient is orthogonal to x
    y0, c0 = T.layer_norm_fwd(x, np.ones(24), np.zeros(24), 0.0)
    dx0, _, _ = T.layer_norm_bwd(dy, c0, g)
    np.testing.assert_allclose((dx0 * x).sum(axis=-1), 0, atol=1e-9)
    np.testing.assert_allclose(db, dy.sum(axis=(0, 1)), rtol=1e-12)
    np.testing.assert_allclose(dg, (dy * xh).sum(axis=(0, 1)), rtol=1e-12)


def test_gelu_values():
    z = np.array([-3.0, -1.0, 0.0, 0.5, 2.0])
    # z * Phi(z) with Phi from math.erf
    want = np.array([t * 0.5 * (1 + math.erf(t / math.sqrt(2))) for t in z])
    np.testing.assert_allclose(T.gelu(z), want, rtol=1e-14)
    assert T.gelu(np.array(0.0)) == 0.0
    assert T.gelu_grad(np.array(0.0)) == 0.5
    np.testing.assert_allclose(T.gelu(z) - T.gelu(-z), z, rtol=1e-14)
    h = 1e-6
    np.testing.assert_allclose(T.gelu_grad(z), (T.gelu(z + h) - T.gelu(z - h)) / (2 * h),
                               rtol=1e-8)


def test_attention_special_cases():
    rng = np.random.default_rng(2)
    B, L, C, H = 2, 6, 8, 2
    qkv = rng.standard_normal((B, L, 3 * C))
    # zero queries: every token attends uniformly -> the mean of v over keys
    z = qkv.copy()
    z[..., :C] = 0
    o, _ = T.attention_fwd(z, H)
    np.testing.assert_allclose(o, np.broadcast_to(z[..., 2 * C:].mean(axis=1, keepdims=True),
                                                  o.shape), rtol=1e-12)
    # one token: attention returns its own v
    o1, _ = T.attention_fwd(qkv[:, :1], H)
    np.testing.assert_allclose(o1, qkv[:, :1, 2 * C:], rtol=1e-12)
