"""CPU oracle for one skip-collocated Pulse pipeline stage (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The GPU
product path never routes through it and shares no code with it: the only
thing both sides consume is the seeded data produced by
``paper_2606_19163_amd.synth`` (which holds none of the method's arithmetic),
passed in as plain arrays.

What is computed
----------------
Pulse places the encoder blocks of a UNet denoiser and their skip-connected
decoder partners on one device (Sec. IV-B, the symmetric placement rule that
sends an op in partition q to partition p-q+1), keeps the skip activations in
local buffers during the forward pass, reuses them for the decoder and for the
backward pass, and keeps the skip *gradients* in local buffers too
(Sec. I and Sec. III, Overview).  With S = 2D stages every device holds one
encoder stage and its mirrored decoder stage (Sec. V-B).  This module computes
exactly what such a stage computes on its device:

* encoder half: x_k = ResBlock_k(x_{k-1}), each cached x_k (and optionally the
  stage input x_0) stored in a skip slot;
* decoder half: v_k = ResBlock^d_k(concat_c(v_{k-1}, skip[slot_k])), upstream
  channels first;
* backward: the exact vector-Jacobian product of
  L = <g_enc, y_enc> + <g_dec, y_dec> with respect to the stage input x, the
  upstream input u, the timestep embedding and every parameter.  A cached x_k
  receives gradient from its encoder consumer and from its decoder consumer;
  the decoder's share is the locally buffered skip gradient.

The paper does not define the block arithmetic (Sec. II-A only says that the
blocks hold attention and ResNet layers).  The ResBlock used here is the
SD-style block: GroupNorm -> SiLU -> 3x3 conv (+ timestep-embedding add) ->
GroupNorm -> SiLU -> 3x3 conv, plus a residual that is the identity when the
channel count is unchanged and a 1x1 conv otherwise.  Readings taken where
the paper is silent:

* every conv, the shortcut and the timestep linear carry a bias; GroupNorm
  uses the biased variance with eps inside the square root, per sample, and
  its groups follow the concatenated channel index (a group may straddle the
  upstream/skip boundary);
* zero padding is applied to the conv input after GroupNorm + SiLU;
* the residual is an unscaled sum; no dropout;
* the timestep path is SiLU, then Linear with bias, added after conv1 and
  broadcast over the image -- parity unpinned: nothing in the paper fixes
  this order, only torch (sharing the reading) checks it;
* skips pair in mirror order (the last cached skip feeds the first decoder
  block), following the symmetric placement rule; which tensors are cached
  (e.g. the stage input of the 32x32 stage) is a descriptor choice -- parity
  unpinned for the same reason.

Every function is the plain definition written out; the only library
primitives used as steps are matrix products (the channel sum of one
convolution tap), elementwise exp and sums.  Layouts: activations NHWC
[B, H, W, C]; 3x3 conv weights OHWI [O, 3, 3, I]; 1x1 weights [O, I]; the
timestep linear [O, D].
"""

from __future__ import annotations

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# elementwise
# ---------------------------------------------------------------------------

def silu(z):
    """SiLU(z) = z * sigmoid(z) = z / (1 + exp(-z))."""
    z = np.asarray(z, dtype=F64)
    return z / (1.0 + np.exp(-z))


def silu_grad(z):
    """d SiLU / dz = s * (1 + z * (1 - s)) with s = sigmoid(z)."""
    z = np.asarray(z, dtype=F64)
    s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


# ---------------------------------------------------------------------------
# GroupNorm
# ---------------------------------------------------------------------------

def group_norm_fwd(x, gamma, beta, groups, eps):
    """GroupNorm over NHWC.

    Group g holds channels [g*C/G, (g+1)*C/G).  For every sample n and group g
    the mean and the *biased* variance run over all H*W*C/G elements;
    z = (x - mean) / sqrt(var + eps) * gamma[c] + beta[c].

    Returns (z, aux) where aux = (xhat, rstd) is what the backward needs.
    """
    x = np.asarray(x, dtype=F64)
    B, H, W, C = x.shape
    if C % groups != 0:
        raise ValueError(f"channels {C} not divisible by groups {groups}")
    cg = C // groups
    xg = x.reshape(B, H * W, groups, cg)
    mean = xg.mean(axis=(1, 3))                                   # [B, G]
    dev = xg - mean[:, None, :, None]
    var = (dev * dev).mean(axis=(1, 3))                            # biased
    rstd = 1.0 / np.sqrt(var + eps)                                # [B, G]
    xhat = (dev * rstd[:, None, :, None]).reshape(B, H, W, C)
    z = xhat * np.asarray(gamma, F64) + np.asarray(beta, F64)
    return z, (xhat, rstd)


def group_norm_bwd(dz, aux, gamma, groups):
    """Backward of :func:`group_norm_fwd`.

    dxhat = dz * gamma;  dgamma[c] = sum dz * xhat;  dbeta[c] = sum dz;
    dx = rstd * (dxhat - mean_g(dxhat) - xhat * mean_g(dxhat * xhat)),
    the means running over the same H*W*C/G elements as the forward.
    """
    xhat, rstd = aux
    dz = np.asarray(dz, dtype=F64)
    B, H, W, C = dz.shape
    cg = C // groups
    dgamma = (dz * xhat).sum(axis=(0, 1, 2))
    dbeta = dz.sum(axis=(0, 1, 2))
    dxhat = (dz * np.asarray(gamma, F64)).reshape(B, H * W, groups, cg)
    xh = xhat.reshape(B, H * W, groups, cg)
    m1 = dxhat.mean(axis=(1, 3))[:, None, :, None]
    m2 = (dxhat * xh).mean(axis=(1, 3))[:, None, :, None]
    dx = rstd[:, None, :, None] * (dxhat - m1 - xh * m2)
    return dx.reshape(B, H, W, C), dgamma, dbeta


# ---------------------------------------------------------------------------
# convolutions (stride 1; 3x3 with zero padding 1 applied to the conv input)
# ---------------------------------------------------------------------------

def _pad1(a):
    B, H, W, C = a.shape
    p = np.zeros((B, H + 2, W + 2, C), dtype=F64)
    p[:, 1:H + 1, 1:W + 1, :] = a
    return p


def conv3x3_fwd(a, w, b):
    """y[n,h,w,o] = b[o] + sum_{dy,dx,i} w[o,dy,dx,i] * a[n,h+dy-1,w+dx-1,i],
    a taken as zero outside the image (cross-correlation, stride 1, pad 1)."""
    a = np.asarray(a, F64)
    w = np.asarray(w, F64)
    B, H, W, I = a.shape
    O = w.shape[0]
    ap = _pad1(a)
    y = np.zeros((B * H * W, O), dtype=F64)
    for dy in range(3):
        for dx in range(3):
            tap = ap[:, dy:dy + H, dx:dx + W, :].reshape(-1, I)
            y += tap @ w[:, dy, dx, :].T
    y += np.asarray(b, F64)
    return y.reshape(B, H, W, O)


def conv3x3_dgrad(dy_, w):
    """da[n,h,w,i] = sum_{o,dy,dx} w[o,dy,dx,i] * dY[n,h-dy+1,w-dx+1,o],
    dY taken as zero outside the image."""
    dy_ = np.asarray(dy_, F64)
    w = np.asarray(w, F64)
    B, H, W, O = dy_.shape
    I = w.shape[3]
    gp = _pad1(dy_)
    da = np.zeros((B * H * W, I), dtype=F64)
    for dy in range(3):
        for dx in range(3):
            # dY[h - dy + 1] lives at padded row h - dy + 2
            tap = gp[:, 2 - dy:2 - dy + H, 2 - dx:2 - dx + W, :].reshape(-1, O)
            da += tap @ w[:, dy, dx, :]
    return da.reshape(B, H, W, I)


def conv3x3_wgrad(dy_, a):
    """dw[o,dy,dx,i] = sum_{n,h,w} dY[n,h,w,o] * a[n,h+dy-1,w+dx-1,i];
    db[o] = sum_{n,h,w} dY[n,h,w,o]."""
    dy_ = np.asarray(dy_, F64)
    a = np.asarray(a, F64)
    B, H, W, O = dy_.shape
    I = a.shape[3]
    ap = _pad1(a)
    g2 = dy_.reshape(-1, O)
    dw = np.zeros((O, 3, 3, I), dtype=F64)
    for dy in range(3):
        for dx in range(3):
            tap = ap[:, dy:dy + H, dx:dx + W, :].reshape(-1, I)
            dw[:, dy, dx, :] = g2.T @ tap
    return dw, g2.sum(axis=0)


def conv1x1_fwd(a, w, b):
    """y[n,h,w,o] = b[o] + sum_i w[o,i] * a[n,h,w,i]."""
    a = np.asarray(a, F64)
    B, H, W, I = a.shape
    y = a.reshape(-1, I) @ np.asarray(w, F64).T + np.asarray(b, F64)
    return y.reshape(B, H, W, -1)


def conv1x1_dgrad(dy_, w):
    """da[n,h,w,i] = sum_o w[o,i] * dY[n,h,w,o]."""
    dy_ = np.asarray(dy_, F64)
    B, H, W, O = dy_.shape
    return (dy_.reshape(-1, O) @ np.asarray(w, F64)).reshape(B, H, W, -1)


def conv1x1_wgrad(dy_, a):
    """dw[o,i] = sum_{n,h,w} dY[n,h,w,o] * a[n,h,w,i]; db[o] = sum dY."""
    dy_ = np.asarray(dy_, F64)
    a = np.asarray(a, F64)
    O = dy_.shape[3]
    I = a.shape[3]
    g2 = dy_.reshape(-1, O)
    return g2.T @ a.reshape(-1, I), g2.sum(axis=0)


# ---------------------------------------------------------------------------
# timestep-embedding projection
# ---------------------------------------------------------------------------

def temb_fwd(temb, wl, bl):
    """e[n,o] = bl[o] + sum_d wl[o,d] * SiLU(temb[n,d])."""
    return silu(temb) @ np.asarray(wl, F64).T + np.asarray(bl, F64)


def temb_bwd(de, temb, wl):
    """Backward of :func:`temb_fwd`: (dwl, dbl, dtemb)."""
    de = np.asarray(de, F64)
    temb = np.asarray(temb, F64)
    dwl = de.T @ silu(temb)
    dbl = de.sum(axis=0)
    dtemb = (de @ np.asarray(wl, F64)) * silu_grad(temb)
    return dwl, dbl, dtemb


# ---------------------------------------------------------------------------
# ResBlock
# ---------------------------------------------------------------------------

def has_conv_shortcut(c_in, c_out):
    """The residual is the identity when the channel count is unchanged and a
    1x1 conv (with bias) otherwise."""
    return c_in != c_out


def resblock_fwd(x, p, temb, groups, eps):
    """out = S(x) + Conv3(SiLU(GN2(h1)); W2, b2),
    h1 = Conv3(SiLU(GN1(x)); W1, b1) + e[n, :],  e = Linear(SiLU(temb)).

    ``p`` maps the names W1 b1 Wl bl g1 be1 g2 be2 W2 b2 (and Ws bs when the
    shortcut is a conv) to arrays.  Returns (out, cache)."""
    x = np.asarray(x, F64)
    c_in = x.shape[3]
    c_out = p["W1"].shape[0]
    z1, gn1 = group_norm_fwd(x, p["g1"], p["be1"], groups, eps)
    a1 = silu(z1)
    e = temb_fwd(temb, p["Wl"], p["bl"])                           # [B, O]
    h1 = conv3x3_fwd(a1, p["W1"], p["b1"]) + e[:, None, None, :]
    z2, gn2 = group_norm_fwd(h1, p["g2"], p["be2"], groups, eps)
    a2 = silu(z2)
    h2 = conv3x3_fwd(a2, p["W2"], p["b2"])
    if has_conv_shortcut(c_in, c_out):
        sc = conv1x1_fwd(x, p["Ws"], p["bs"])
    else:
        sc = x
    out = sc + h2
    cache = dict(x=x, z1=z1, gn1=gn1, a1=a1, h1=h1, z2=z2, gn2=gn2, a2=a2,
                 temb=np.asarray(temb, F64))
    return out, cache


def resblock_bwd(dout, cache, p, groups):
    """Exact backward of :func:`resblock_fwd`.  Returns (dx, grads, dtemb)
    with grads keyed like ``p``."""
    dout = np.asarray(dout, F64)
    x = cache["x"]
    c_in = x.shape[3]
    c_out = p["W1"].shape[0]
    g = {}
    # h2 = Conv3(a2)
    g["W2"], g["b2"] = conv3x3_wgrad(dout, cache["a2"])
    da2 = conv3x3_dgrad(dout, p["W2"])
    dz2 = da2 * silu_grad(cache["z2"])
    dh1, g["g2"], g["be2"] = group_norm_bwd(dz2, cache["gn2"], p["g2"], groups)
    # h1 = Conv3(a1) + e
    de = dh1.sum(axis=(1, 2))                                      # [B, O]
    g["Wl"], g["bl"], dtemb = temb_bwd(de, cache["temb"], p["Wl"])
    g["W1"], g["b1"] = conv3x3_wgrad(dh1, cache["a1"])
    da1 = conv3x3_dgrad(dh1, p["W1"])
    dz1 = da1 * silu_grad(cache["z1"])
    dx, g["g1"], g["be1"] = group_norm_bwd(dz1, cache["gn1"], p["g1"], groups)
    # residual
    if has_conv_shortcut(c_in, c_out):
        g["Ws"], g["bs"] = conv1x1_wgrad(dout, x)
        dx = dx + conv1x1_dgrad(dout, p["Ws"])
    else:
        dx = dx + dout
    return dx, g, dtemb


# ---------------------------------------------------------------------------
# the stage
# ---------------------------------------------------------------------------

def _block_params(params, prefix):
    n = len(prefix)
    return {k[n:]: v for k, v in params.items() if k.startswith(prefix)}


def stage_run(desc, params, x, u, temb, g_enc, g_dec):
    """Forward and backward of one collocated stage.

    ``desc``: dict with batch, height, width, groups, eps, temb_dim,
    enc = [{c_in, c_out, skip_slot_out}], dec = [{c_up, c_skip, c_out,
    skip_slot_in}], input_skip_slot (-1 when the stage input is not cached).
    ``params``: dict "enc{k}.NAME" / "dec{k}.NAME" -> array.

    Returns a dict with y_enc, y_dec, dx, du, dtemb, grads (same keys as
    params), skips {slot: activation} and dskips {slot: gradient}.
    """
    G = int(desc["groups"])
    eps = float(desc["eps"])
    x = np.asarray(x, F64)
    u = np.asarray(u, F64)
    temb = np.asarray(temb, F64)
    skips = {}
    in_slot = int(desc.get("input_skip_slot", -1))
    if in_slot >= 0:
        skips[in_slot] = x

    # ---- encoder forward: every cached block output goes to its slot
    enc_caches = []
    h = x
    for k, blk in enumerate(desc["enc"]):
        p = _block_params(params, f"enc{k}.")
        h, c = resblock_fwd(h, p, temb, G, eps)
        enc_caches.append(c)
        if blk["skip_slot_out"] >= 0:
            skips[int(blk["skip_slot_out"])] = h
    y_enc = h

    # ---- decoder forward: upstream channels first, then the skip
    dec_caches = []
    v = u
    for k, blk in enumerate(desc["dec"]):
        p = _block_params(params, f"dec{k}.")
        s = skips[int(blk["skip_slot_in"])]
        v, c = resblock_fwd(np.concatenate([v, s], axis=3), p, temb, G, eps)
        dec_caches.append(c)
    y_dec = v

    # ---- decoder backward: split the input gradient, buffer the skip part
    grads = {}
    dtemb = np.zeros_like(temb)
    dskips = {s: np.zeros_like(a) for s, a in skips.items()}
    dv = np.asarray(g_dec, F64)
    for k in reversed(range(len(desc["dec"]))):
        blk = desc["dec"][k]
        p = _block_params(params, f"dec{k}.")
        dcat, gk, dt = resblock_bwd(dv, dec_caches[k], p, G)
        for name, val in gk.items():
            grads[f"dec{k}.{name}"] = val
        dtemb += dt
        c_up = int(blk["c_up"])
        dv = dcat[..., :c_up]
        dskips[int(blk["skip_slot_in"])] += dcat[..., c_up:]
    du = dv

    # ---- encoder backward: add the locally buffered skip gradient
    dh = np.asarray(g_enc, F64)
    for k in reversed(range(len(desc["enc"]))):
        blk = desc["enc"][k]
        if blk["skip_slot_out"] >= 0:
            dh = dh + dskips[int(blk["skip_slot_out"])]
        p = _block_params(params, f"enc{k}.")
        dh, gk, dt = resblock_bwd(dh, enc_caches[k], p, G)
        for name, val in gk.items():
            grads[f"enc{k}.{name}"] = val
        dtemb += dt
    if in_slot >= 0:
        dh = dh + dskips[in_slot]
    dx = dh

    return dict(y_enc=y_enc, y_dec=y_dec, dx=dx, du=du, dtemb=dtemb,
                grads=grads, skips=skips, dskips=dskips)


def stage_forward_only(desc, params, x, u, temb):
    """Forward outputs only (y_enc, y_dec, skips); used for sampled checks."""
    G = int(desc["groups"])
    eps = float(desc["eps"])
    x = np.asarray(x, F64)
    skips = {}
    in_slot = int(desc.get("input_skip_slot", -1))
    if in_slot >= 0:
        skips[in_slot] = x
    h = x
    for k, blk in enumerate(desc["enc"]):
        h, _ = resblock_fwd(h, _block_params(params, f"enc{k}."), temb, G, eps)
        if blk["skip_slot_out"] >= 0:
            skips[int(blk["skip_slot_out"])] = h
    v = np.asarray(u, F64)
    for k, blk in enumerate(desc["dec"]):
        s = skips[int(blk["skip_slot_in"])]
        v, _ = resblock_fwd(np.concatenate([v, s], axis=3),
                            _block_params(params, f"dec{k}."), temb, G, eps)
    return dict(y_enc=h, y_dec=v, skips=skips)


# ---------------------------------------------------------------------------
# the decoder block without a materialised concat
# ---------------------------------------------------------------------------

def resblock_fwd_two_source(v, s, p, temb, groups, eps):
    """The decoder ResBlock on [v || s] computed from the two sources apart.

    GroupNorm groups follow the concatenated channel index (a group may hold
    channels of both sources), so the statistics gather from both.  A conv
    over the concatenation is the sum of the convs over each source with the
    matching slice of the input-channel axis of the weights.  Used to pin
    that reading the two sources separately is the same map as the explicit
    concatenation.  Returns out only."""
    v = np.asarray(v, F64)
    s = np.asarray(s, F64)
    B, H, W, cu = v.shape
    cs = s.shape[3]
    C = cu + cs
    cg = C // groups
    # statistics per (n, g) gathered from whichever source holds the channel
    mean = np.zeros((B, groups))
    var = np.zeros((B, groups))
    for g in range(groups):
        lo, hi = g * cg, (g + 1) * cg
        parts = []
        if lo < cu:
            parts.append(v[..., lo:min(hi, cu)].reshape(B, -1))
        if hi > cu:
            parts.append(s[..., max(lo, cu) - cu:hi - cu].reshape(B, -1))
        allv = np.concatenate(parts, axis=1)
        mean[:, g] = allv.mean(axis=1)
        var[:, g] = ((allv - mean[:, g:g + 1]) ** 2).mean(axis=1)
    rstd = 1.0 / np.sqrt(var + eps)
    gidx = np.arange(C) // cg

    def act(src, c0):
        cidx = gidx[c0:c0 + src.shape[3]]
        m = mean[:, cidx][:, None, None, :]
        r = rstd[:, cidx][:, None, None, :]
        ga = p["g1"][c0:c0 + src.shape[3]]
        be = p["be1"][c0:c0 + src.shape[3]]
        return silu((src - m) * r * ga + be)

    w1 = np.asarray(p["W1"], F64)
    e = temb_fwd(temb, p["Wl"], p["bl"])
    h1 = (conv3x3_fwd(act(v, 0), w1[..., :cu], p["b1"])
          + conv3x3_fwd(act(s, cu), w1[..., cu:], np.zeros_like(p["b1"]))
          + e[:, None, None, :])
    z2, _ = group_norm_fwd(h1, p["g2"], p["be2"], groups, eps)
    h2 = conv3x3_fwd(silu(z2), p["W2"], p["b2"])
    ws = np.asarray(p["Ws"], F64)
    sc = (conv1x1_fwd(v, ws[:, :cu], p["bs"])
          + conv1x1_fwd(s, ws[:, cu:], np.zeros_like(p["bs"])))
    return sc + h2
