"""CPU oracle for a skip-collocated stage of transformer blocks (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The
product package never imports it, and the GPU path shares no code with it.

What is computed
----------------
The paper's method applies to UNet-like denoisers whose long skips join
encoder and decoder blocks, including the transformer-block models it
evaluates (UViT, Hunyuan-DiT; Sec. II-A, Sec. VII).  As for the ResBlock
stage, one device holds an encoder group whose block outputs are cached as
skips and the decoder group that consumes them (Sec. IV-B, Sec. V-B):

* encoder half: x_k = Block_k(x_{k-1}), each x_k stored in skip slot k;
* decoder half: v_k = Block^d_k(Skip_k([v_{k-1} || skip[slot]])), where
  Skip_k is a linear layer over the token-wise concatenation (upstream
  channels first) and the slots pair in mirror order (the last cached skip
  feeds the first decoder block);
* backward: the exact vector-Jacobian product of
  L = <g_enc, y_enc> + <g_dec, y_dec> with respect to x, u and every
  parameter; a cached x_k receives gradient from its encoder consumer and,
  through the locally buffered skip gradient, from its decoder consumer.

The paper does not define the block; the one used here is the pre-norm
transformer block of the UViT family:

    h = x + Proj(MHA(LN1(x)))      MHA: softmax(q k^T / sqrt(d)) v per head
    y = h + Fc2(GELU(Fc1(LN2(h))))

Readings taken where the paper is silent: LayerNorm over the channels of each
token, biased variance, eps inside the square root; the qkv projection, the
output projection, both MLP layers and the skip linear carry biases; heads
split the channels in order (head j owns channels [j d, (j + 1) d) of q, k
and v, with q, k, v stacked in that order along the qkv output); GELU is the
exact erf form; the MLP is 4x wide; no time or class tokens, dropout or
attention masking.  Layouts: tokens [B, L, C]; linear weights [out, in].

Every function is the plain definition written out; the library primitives
used as steps are matrix products, exp, erf and sums.
"""

from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

F64 = np.float64


# ---------------------------------------------------------------------------
# pieces
# ---------------------------------------------------------------------------

def layer_norm_fwd(x, g, b, eps):
    """y = (x - mean) / sqrt(var + eps) * g + b over the last axis."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xh = (x - mu) * rstd
    return xh * g + b, (xh, rstd)


def layer_norm_bwd(dy, cache, g):
    """dx, dg, db of the LayerNorm above."""
    xh, rstd = cache
    dy = np.asarray(dy, F64)
    C = xh.shape[-1]
    dxh = dy * g
    dx = rstd * (dxh - dxh.mean(axis=-1, keepdims=True)
                 - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    axes = tuple(range(dy.ndim - 1))
    return dx, (dy * xh).sum(axis=axes), dy.sum(axis=axes)


def gelu(z):
    """z * Phi(z) with the standard normal CDF Phi."""
    return z * 0.5 * (1.0 + erf(z / math.sqrt(2.0)))


def gelu_grad(z):
    """Phi(z) + z * phi(z)."""
    return 0.5 * (1.0 + erf(z / math.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / math.sqrt(2 * math.pi)


def linear_fwd(x, w, b):
    """y[..., o] = b[o] + sum_i w[o, i] x[..., i]."""
    return np.asarray(x, F64) @ np.asarray(w, F64).T + b


def linear_bwd(dy, x, w):
    """dx, dw, db of the linear layer above."""
    dy = np.asarray(dy, F64)
    x = np.asarray(x, F64)
    O, I = dy.shape[-1], x.shape[-1]
    d2, x2 = dy.reshape(-1, O), x.reshape(-1, I)
    return dy @ np.asarray(w, F64), d2.T @ x2, d2.sum(axis=0)


def attention_fwd(qkv, heads):
    """Multi-head attention of q, k, v stacked along the last axis of qkv
    [B, L, 3C]: o[b, i, head] = sum_j softmax_j(q_i . k_j / sqrt(d)) v_j."""
    B, L, C3 = qkv.shape
    C = C3 // 3
    d = C // heads
    q = qkv[..., :C].reshape(B, L, heads, d).transpose(0, 2, 1, 3)
    k = qkv[..., C:2 * C].reshape(B, L, heads, d).transpose(0, 2, 1, 3)
    v = qkv[..., 2 * C:].reshape(B, L, heads, d).transpose(0, 2, 1, 3)
    s = q @ k.transpose(0, 1, 3, 2) / math.sqrt(d)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    o = p @ v
    return o.transpose(0, 2, 1, 3).reshape(B, L, C), (q, k, v, p)


def attention_bwd(do, cache, heads):
    """d(qkv) of the attention above."""
    q, k, v, p = cache
    B, H, L, d = q.shape
    do = np.asarray(do, F64).reshape(B, L, H, d).transpose(0, 2, 1, 3)
    dv = p.transpose(0, 1, 3, 2) @ do
    dp = do @ v.transpose(0, 1, 3, 2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True)) / math.sqrt(d)
    dq = ds @ k
    dk = ds.transpose(0, 1, 3, 2) @ q
    back = lambda t: t.transpose(0, 2, 1, 3).reshape(B, L, H * d)
    return np.concatenate([back(dq), back(dk), back(dv)], axis=-1)


# ---------------------------------------------------------------------------
# the block
# ---------------------------------------------------------------------------

def block_fwd(x, p, heads, eps):
    """One pre-norm transformer block; returns (y, cache)."""
    x = np.asarray(x, F64)
    a, c1 = layer_norm_fwd(x, p["ln1.g"], p["ln1.b"], eps)
    qkv = linear_fwd(a, p["qkv.W"], p["qkv.b"])
    o, ca = attention_fwd(qkv, heads)
    h = x + linear_fwd(o, p["proj.W"], p["proj.b"])
    a2, c2 = layer_norm_fwd(h, p["ln2.g"], p["ln2.b"], eps)
    z = linear_fwd(a2, p["fc1.W"], p["fc1.b"])
    m = gelu(z)
    y = h + linear_fwd(m, p["fc2.W"], p["fc2.b"])
    return y, dict(x=x, a=a, c1=c1, qkv=qkv, o=o, ca=ca, h=h, a2=a2, c2=c2, z=z, m=m)


def block_bwd(dy, c, p, heads):
    """(dx, grads) of block_fwd."""
    g = {}
    dy = np.asarray(dy, F64)
    dm, g["fc2.W"], g["fc2.b"] = linear_bwd(dy, c["m"], p["fc2.W"])
    dz = dm * gelu_grad(c["z"])
    da2, g["fc1.W"], g["fc1.b"] = linear_bwd(dz, c["a2"], p["fc1.W"])
    dh_ln, g["ln2.g"], g["ln2.b"] = layer_norm_bwd(da2, c["c2"], p["ln2.g"])
    dh = dy + dh_ln
    do, g["proj.W"], g["proj.b"] = linear_bwd(dh, c["o"], p["proj.W"])
    dqkv = attention_bwd(do, c["ca"], heads)
    da, g["qkv.W"], g["qkv.b"] = linear_bwd(dqkv, c["a"], p["qkv.W"])
    dx_ln, g["ln1.g"], g["ln1.b"] = layer_norm_bwd(da, c["c1"], p["ln1.g"])
    return dh + dx_ln, g


BLOCK_PARAMS = ("ln1.g", "ln1.b", "qkv.W", "qkv.b", "proj.W", "proj.b",
                "ln2.g", "ln2.b", "fc1.W", "fc1.b", "fc2.W", "fc2.b")


def _sub(params, prefix):
    return {k[len(prefix):]: np.asarray(v, F64) for k, v in params.items()
            if k.startswith(prefix)}


# ---------------------------------------------------------------------------
# the stage
# ---------------------------------------------------------------------------

def tstage_run(desc, params, x, u, g_enc, g_dec):
    """Forward and backward of one collocated transformer stage.

    ``desc``: dict with batch, tokens, width, heads, eps, n_enc, n_dec.
    ``params``: "enc{k}.NAME" for NAME in BLOCK_PARAMS, "dec{k}.NAME" and
    "dec{k}.skip.W" [C, 2C], "dec{k}.skip.b".  Encoder block k fills skip
    slot k; decoder block k reads slot n_enc - 1 - k.

    Returns y_enc, y_dec, dx, du, grads, skips {slot: x_k}, dskips {slot:
    buffered gradient of x_k from the decoder}.
    """
    H, eps = int(desc["heads"]), float(desc["eps"])
    ne, nd = int(desc["n_enc"]), int(desc["n_dec"])
    C = int(desc["width"])
    h = np.asarray(x, F64)
    skips, enc_c = {}, []
    for k in range(ne):
        h, c = block_fwd(h, _sub(params, f"enc{k}."), H, eps)
        enc_c.append(c)
        skips[k] = h
    y_enc = h
    v = np.asarray(u, F64)
    dec_c = []
    for k in range(nd):
        p = _sub(params, f"dec{k}.")
        cat = np.concatenate([v, skips[ne - 1 - k]], axis=-1)
        s = linear_fwd(cat, p["skip.W"], p["skip.b"])
        v, c = block_fwd(s, p, H, eps)
        dec_c.append((cat, c))
    y_dec = v
    grads = {}
    dskips = {}
    dv = np.asarray(g_dec, F64)
    for k in reversed(range(nd)):
        p = _sub(params, f"dec{k}.")
        cat, c = dec_c[k]
        ds, g = block_bwd(dv, c, p, H)
        dcat, g["skip.W"], g["skip.b"] = linear_bwd(ds, cat, p["skip.W"])
        for n, val in g.items():
            grads[f"dec{k}.{n}"] = val
        dv = dcat[..., :C]
        dskips[ne - 1 - k] = dcat[..., C:]
    du = dv
    dh = np.asarray(g_enc, F64)
    for k in reversed(range(ne)):
        if k in dskips:
            dh = dh + dskips[k]
        dh, g = block_bwd(dh, enc_c[k], _sub(params, f"enc{k}."), H)
        for n, val in g.items():
            grads[f"enc{k}.{n}"] = val
    return dict(y_enc=y_enc, y_dec=y_dec, dx=dh, du=du, grads=grads, skips=skips,
                dskips=dskips)


def tstage_forward_only(desc, params, x, u):
    """y_enc, y_dec of tstage_run without the backward pass."""
    H, eps = int(desc["heads"]), float(desc["eps"])
    ne, nd = int(desc["n_enc"]), int(desc["n_dec"])
    h = np.asarray(x, F64)
    skips = {}
    for k in range(ne):
        h, _ = block_fwd(h, _sub(params, f"enc{k}."), H, eps)
        skips[k] = h
    v = np.asarray(u, F64)
    for k in range(nd):
        p = _sub(params, f"dec{k}.")
        s = linear_fwd(np.concatenate([v, skips[ne - 1 - k]], axis=-1), p["skip.W"],
                       p["skip.b"])
        v, _ = block_fwd(s, p, H, eps)
    return dict(y_enc=h, y_dec=v)
