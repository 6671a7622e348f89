"""Pins of the oracle's whole stage (forward + vector-Jacobian product):
finite differences in fp64, torch autograd over a torch.nn.functional
composition, the two-source decoder block against the explicit concat, and
the skip-gradient paths."""

import copy

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pulse_oracle as O
from paper_2606_19163_amd import configs, synth


def tiny_desc(c=4, c_skip=None, groups=2, hw=4, width=None, batch=1, dt=8, n_blocks=1):
    d = configs._pair_stage(batch, hw, c, groups, dt, "f32", n_blocks=n_blocks)
    if width is not None:
        d["width"] = width
    if c_skip is not None:
        # decoder reads a narrower skip: cache the stage input of width c_skip
        d["enc"] = [dict(c_in=c_skip, c_out=c, skip_slot_out=0)]
        d["dec"] = [dict(c_up=c, c_skip=c, c_out=c, skip_slot_in=0),
                    dict(c_up=c, c_skip=c_skip, c_out=c, skip_slot_in=1)]
        d["input_skip_slot"] = 1
    return d


def f64(dct):
    return {k: np.asarray(v, np.float64) for k, v in dct.items()}


def loss(desc, params, b):
    out = O.stage_forward_only(desc, params, b["x"], b["u"], b["temb"])
    return np.sum(b["g_enc"] * out["y_enc"]) + np.sum(b["g_dec"] * out["y_dec"])


# --------------------------------------------------------------------------
# finite differences
# --------------------------------------------------------------------------

def _fd_check(desc, seed, n_samples=6, h=1e-6, tol=1e-6):
    params, b = synth.make_all(desc, seed)
    params, b = f64(params), f64(b)
    res = O.stage_run(desc, params, b["x"], b["u"], b["temb"], b["g_enc"], b["g_dec"])
    rng = np.random.default_rng(seed + 100)
    worst = 0.0

    def check(analytic, perturb):
        nonlocal worst
        lp = perturb(+h)
        lm = perturb(-h)
        fd = (lp - lm) / (2 * h)
        err = abs(fd - analytic) / max(1e-3, abs(fd), abs(analytic))
        worst = max(worst, err)

    for name in ("x", "u", "temb"):
        grad = {"x": res["dx"], "u": res["du"], "temb": res["dtemb"]}[name]
        for _ in range(n_samples):
            idx = tuple(rng.integers(0, s) for s in b[name].shape)

            def pert(d, name=name, idx=idx):
                bb = copy.deepcopy(b)
                bb[name][idx] += d
                return loss(desc, params, bb)
            check(grad[idx], pert)
    for pname in params:
        for _ in range(max(1, n_samples // 2)):
            idx = tuple(rng.integers(0, s) for s in params[pname].shape)

            def pert(d, pname=pname, idx=idx):
                pp = dict(params)
                pp[pname] = params[pname].copy()
                pp[pname][idx] += d
                return loss(desc, pp, b)
            check(res["grads"][pname][idx], pert)
    assert worst <= tol, worst


def test_fd_one_pair():
    _fd_check(tiny_desc(), seed=1)


def test_fd_two_pairs_ragged_width():
    _fd_check(tiny_desc(c=4, groups=2, hw=3, width=5, n_blocks=2), seed=2)


def test_fd_straddling_groups_and_cached_input():
    # second decoder block reads (4 || 2) = 6 channels in 2 groups of 3:
    # group 1 holds channel 3 of the upstream source and both skip channels
    _fd_check(tiny_desc(c=4, c_skip=2, groups=2), seed=3)


# --------------------------------------------------------------------------
# torch autograd on an independent functional composition
# --------------------------------------------------------------------------

def _torch_stage(desc, params, b):
    G, eps = desc["groups"], desc["eps"]
    P = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in params.items()}
    T = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in b.items()}

    def block(xin, pre):
        def w3(name):
            return P[pre + name].permute(0, 3, 1, 2)
        xin_c = xin.permute(0, 3, 1, 2)
        a1 = F.silu(F.group_norm(xin_c, G, P[pre + "g1"], P[pre + "be1"], eps))
        e = F.linear(F.silu(T["temb"]), P[pre + "Wl"], P[pre + "bl"])
        h1 = F.conv2d(a1, w3("W1"), P[pre + "b1"], padding=1) + e[:, :, None, None]
        a2 = F.silu(F.group_norm(h1, G, P[pre + "g2"], P[pre + "be2"], eps))
        h2 = F.conv2d(a2, w3("W2"), P[pre + "b2"], padding=1)
        if pre + "Ws" in P:
            sc = F.conv2d(xin_c, P[pre + "Ws"][:, :, None, None], P[pre + "bs"])
        else:
            sc = xin_c
        return (sc + h2).permute(0, 2, 3, 1)

    skips = {}
    if desc["input_skip_slot"] >= 0:
        skips[desc["input_skip_slot"]] = T["x"]
    h = T["x"]
    for k, blk in enumerate(desc["enc"]):
        h = block(h, f"enc{k}.")
        if blk["skip_slot_out"] >= 0:
            skips[blk["skip_slot_out"]] = h
    v = T["u"]
    for k, blk in enumerate(desc["dec"]):
        v = block(torch.cat([v, skips[blk["skip_slot_in"]]], dim=3), f"dec{k}.")
    L = (T["g_enc"] * h).sum() + (T["g_dec"] * v).sum()
    L.backward()
    return h.detach().numpy(), v.detach().numpy(), T, P


@pytest.mark.parametrize("which", ["tiny", "l64s", "l32s", "l16s"])
def test_stage_against_torch_autograd(which):
    if which == "tiny":
        desc = configs.tiny()
        desc["batch"], desc["height"], desc["width"] = 1, 6, 5
    elif which == "l64s":
        desc = configs._pair_stage(2, 4, 8, 4, 16, "f32")
    elif which == "l32s":
        desc = configs.l32()
        desc.update(batch=2, height=4, width=3, groups=4, temb_dim=16, dtype="f32")
        for blk in desc["enc"]:
            blk["c_in"], blk["c_out"] = blk["c_in"] // 40, blk["c_out"] // 40
        for blk in desc["dec"]:
            blk["c_up"], blk["c_skip"], blk["c_out"] = (blk["c_up"] // 40, blk["c_skip"] // 40,
                                                         blk["c_out"] // 40)
    else:
        desc = configs._pair_stage(2, 2, 16, 4, 16, "f32")
    params, b = synth.make_all(desc, 7)
    params, b = f64(params), f64(b)
    res = O.stage_run(desc, params, b["x"], b["u"], b["temb"], b["g_enc"], b["g_dec"])
    y_enc, y_dec, T, P = _torch_stage(desc, params, b)
    tol = dict(rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(res["y_enc"], y_enc, **tol)
    np.testing.assert_allclose(res["y_dec"], y_dec, **tol)
    np.testing.assert_allclose(res["dx"], T["x"].grad.numpy(), **tol)
    np.testing.assert_allclose(res["du"], T["u"].grad.numpy(), **tol)
    np.testing.assert_allclose(res["dtemb"], T["temb"].grad.numpy(), **tol)
    for k in params:
        np.testing.assert_allclose(res["grads"][k], P[k].grad.numpy(), err_msg=k, **tol)


# --------------------------------------------------------------------------
# concat-free decoder block, skip-gradient paths
# --------------------------------------------------------------------------

@pytest.mark.parametrize("cu,cs,G", [(4, 4, 2), (4, 2, 2), (6, 3, 3), (8, 4, 4)])
def test_two_source_block_equals_explicit_concat(cu, cs, G):
    rng = np.random.default_rng(cu * 10 + cs)
    desc = dict(groups=G, eps=1e-5)
    co = cu
    C = cu + cs
    p = {"W1": rng.standard_normal((co, 3, 3, C)), "b1": rng.standard_normal(co),
         "Wl": rng.standard_normal((co, 5)), "bl": rng.standard_normal(co),
         "g1": 1 + 0.1 * rng.standard_normal(C), "be1": 0.1 * rng.standard_normal(C),
         "g2": 1 + 0.1 * rng.standard_normal(co), "be2": 0.1 * rng.standard_normal(co),
         "W2": rng.standard_normal((co, 3, 3, co)), "b2": rng.standard_normal(co),
         "Ws": rng.standard_normal((co, C)), "bs": rng.standard_normal(co)}
    v = rng.standard_normal((2, 4, 5, cu))
    s = 2.0 + rng.standard_normal((2, 4, 5, cs))
    temb = rng.standard_normal((2, 5))
    ref, _ = O.resblock_fwd(np.concatenate([v, s], 3), p, temb, G, desc["eps"])
    two = O.resblock_fwd_two_source(v, s, p, temb, G, desc["eps"])
    np.testing.assert_allclose(two, ref, rtol=1e-11, atol=1e-11)


def test_skip_gradient_vanishes_without_decoder_cotangent():
    desc = configs._pair_stage(1, 4, 4, 2, 8, "f32")
    params, b = synth.make_all(desc, 21)
    params, b = f64(params), f64(b)
    b["g_dec"] = np.zeros_like(b["g_dec"])
    res = O.stage_run(desc, params, b["x"], b["u"], b["temb"], b["g_enc"], b["g_dec"])
    for s, d in res["dskips"].items():
        assert np.all(d == 0.0)
    assert np.all(res["du"] == 0.0)
    # with no encoder cotangent the encoder gradient is the skip path alone
    b2 = dict(b)
    b2["g_dec"] = np.random.default_rng(3).standard_normal(b["g_dec"].shape)
    b2["g_enc"] = np.zeros_like(b["g_enc"])
    res2 = O.stage_run(desc, params, b2["x"], b2["u"], b2["temb"], b2["g_enc"], b2["g_dec"])
    assert np.abs(res2["dx"]).max() > 0
    assert any(np.abs(d).max() > 0 for d in res2["dskips"].values())


def test_chained_single_device_gradient():
    # D = 1: the decoder's upstream input is the encoder's own output, so the
    # full gradient w.r.t. x is dx of a second pass whose encoder cotangent
    # also carries du.  Compared with finite differences of the composition.
    desc = configs._pair_stage(1, 3, 4, 2, 6, "f32", n_blocks=2)
    params, b = synth.make_all(desc, 22)
    params, b = f64(params), f64(b)

    def composed(x):
        y_enc = O.stage_forward_only(desc, params, x, b["u"], b["temb"])["y_enc"]
        out = O.stage_forward_only(desc, params, x, y_enc, b["temb"])
        return np.sum(b["g_enc"] * out["y_enc"]) + np.sum(b["g_dec"] * out["y_dec"])

    y_enc = O.stage_forward_only(desc, params, b["x"], b["u"], b["temb"])["y_enc"]
    r1 = O.stage_run(desc, params, b["x"], y_enc, b["temb"], b["g_enc"], b["g_dec"])
    r2 = O.stage_run(desc, params, b["x"], y_enc, b["temb"], b["g_enc"] + r1["du"],
                     b["g_dec"])
    rng = np.random.default_rng(5)
    h = 1e-6
    for _ in range(8):
        idx = tuple(rng.integers(0, s) for s in b["x"].shape)
        xp, xm = b["x"].copy(), b["x"].copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (composed(xp) - composed(xm)) / (2 * h)
        assert abs(fd - r2["dx"][idx]) <= 1e-6 * max(1.0, abs(fd))
