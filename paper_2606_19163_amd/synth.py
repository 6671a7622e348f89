"""Seeded synthetic inputs for a stage (shared by the tests, the bench and the
oracle's callers; it holds none of the stage's arithmetic).

Draw order (numpy PCG64 ``default_rng(seed)``, fp32 ``standard_normal``):
parameters block by block in descriptor order (encoder then decoder; in a
block W1 b1 Wl bl g1 be1 g2 be2 W2 b2 [Ws bs]), then x, u, temb, g_enc,
g_dec.

Scaling: a weight of fan-in F is N(0, 1/F) in the variance sense (std
F**-0.5); its bias uses the same F.  F is 9*C_in for a 3x3 conv (C_in counts
both concatenated sources), C_in for a 1x1 conv and the embedding width for
the timestep linear.  GroupNorm gains are 1 + 0.1*N(0,1) and shifts
0.1*N(0,1) so the affine path is exercised.  Activations, embeddings and
upstream gradients are N(0,1).

For bf16 stages every draw is rounded to bf16 (round to nearest, ties to
even) and the *decoded* values are what both the oracle and the device see.
"""

from __future__ import annotations

import numpy as np

from . import configs as _cfg


def bf16_bits(a):
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    r = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_decode(bits):
    """bf16 bit patterns (uint16) -> fp32 values."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def round_bf16(a):
    return bf16_decode(bf16_bits(a))


def _fan_in(name, shape):
    leaf = name.split(".")[-1]
    if leaf in ("W1", "W2"):
        return shape[1] * shape[2] * shape[3]
    if leaf == "Ws":
        return shape[1]
    if leaf == "Wl":
        return shape[1]
    return None


def make_params(desc, rng):
    """Parameters as a dict name -> fp32 array (bf16-representable for bf16
    stages)."""
    names = _cfg.param_names(desc)
    shapes = dict(names)
    out = {}
    last_fan = {}
    for name, shape in names:
        leaf = name.split(".")[-1]
        blk = name.rsplit(".", 1)[0]
        z = rng.standard_normal(shape, dtype=np.float32)
        if leaf in ("W1", "W2", "Ws", "Wl"):
            f = _fan_in(name, shape)
            last_fan[(blk, leaf)] = f
            v = z / np.float32(np.sqrt(f))
        elif leaf in ("b1", "b2", "bs", "bl"):
            wname = {"b1": "W1", "b2": "W2", "bs": "Ws", "bl": "Wl"}[leaf]
            f = _fan_in(blk + "." + wname, shapes[blk + "." + wname])
            v = z / np.float32(np.sqrt(f))
        elif leaf in ("g1", "g2"):
            v = np.float32(1.0) + np.float32(0.1) * z
        else:  # be1, be2
            v = np.float32(0.1) * z
        out[name] = v.astype(np.float32)
    if desc["dtype"] == _cfg.BF16:
        out = {k: round_bf16(v) for k, v in out.items()}
    return out


def make_boundary(desc, rng):
    """x, u, temb, g_enc, g_dec as fp32 arrays (bf16-representable for bf16
    stages)."""
    B, H, W = desc["batch"], desc["height"], desc["width"]
    shapes = dict(
        x=(B, H, W, desc["enc"][0]["c_in"]),
        u=(B, H, W, desc["dec"][0]["c_up"]),
        temb=(B, desc["temb_dim"]),
        g_enc=(B, H, W, desc["enc"][-1]["c_out"]),
        g_dec=(B, H, W, desc["dec"][-1]["c_out"]),
    )
    out = {}
    for k in ("x", "u", "temb", "g_enc", "g_dec"):
        out[k] = rng.standard_normal(shapes[k], dtype=np.float32)
    if desc["dtype"] == _cfg.BF16:
        out = {k: round_bf16(v) for k, v in out.items()}
    return out


def make_all(desc, seed):
    """(params, boundary) for one stage, drawn from ``default_rng(seed)``."""
    rng = np.random.default_rng(seed)
    params = make_params(desc, rng)
    boundary = make_boundary(desc, rng)
    return params, boundary


def make_wave(levels, seed, n_mb):
    """Parameters per level, then boundary tensors per (level, microbatch),
    all from one ``default_rng(seed)`` stream."""
    rng = np.random.default_rng(seed)
    params = [make_params(d, rng) for d in levels]
    bounds = [[make_boundary(d, rng) for _ in range(n_mb)] for d in levels]
    return params, bounds


def make_tstage(desc, seed):
    """(params, boundary) of a transformer stage from ``default_rng(seed)``:
    parameters in tparam_names order (a weight [out, in] is N(0, 1/in), its
    bias uses the same fan-in; LayerNorm gains 1 + 0.1 N(0,1), shifts
    0.1 N(0,1)), then x, u, g_enc, g_dec [B, L, C] ~ N(0,1); bf16-rounded
    for bf16 stages."""
    rng = np.random.default_rng(seed)
    names = _cfg.tparam_names(desc)
    shapes = dict(names)
    params = {}
    for name, shape in names:
        leaf = name.split(".")[-1]
        z = rng.standard_normal(shape, dtype=np.float32)
        if leaf == "W":
            v = z / np.float32(np.sqrt(shape[1]))
        elif leaf == "b" and not name.split(".")[-2].startswith("ln"):
            fan = shapes[name[:-1] + "W"][1]
            v = z / np.float32(np.sqrt(fan))
        elif leaf == "g":
            v = np.float32(1.0) + np.float32(0.1) * z
        else:
            v = np.float32(0.1) * z
        params[name] = v.astype(np.float32)
    shp = (desc["batch"], desc["tokens"], desc["width"])
    bound = {k: rng.standard_normal(shp, dtype=np.float32) for k in ("x", "u", "g_enc", "g_dec")}
    if desc["dtype"] == _cfg.BF16:
        params = {k: round_bf16(v) for k, v in params.items()}
        bound = {k: round_bf16(v) for k, v in bound.items()}
    return params, bound
