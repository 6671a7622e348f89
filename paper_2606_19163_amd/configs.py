"""Stage descriptors for the synthetic SD-shaped workloads.

A descriptor is a plain dict (the Python twin of ``pulse_stage_desc`` in
``include/pulse_stage.h``).  Each stage is one collocated pair: the encoder
ResBlocks of pipeline stage q and the mirrored decoder ResBlocks of stage
2D-1-q that read their skips (symmetric placement, Sec. IV-B; S = 2D,
Sec. V-B).  Skip slots pair up last-in-first-out: the last cached encoder
output feeds the first decoder block.

Workloads (shapes of the SD UNet levels; the paper's own SDv2 widths are not
given, so these stand in for its workload):

* ``tiny``   fp32, B=2, 16x16, C=32, 8 groups, t-emb 128: one encoder block
  32->32 caching its output, one decoder block (32 || 32) -> 32.
* ``l64``    bf16, B=8, 64x64, C=320: 2 encoder blocks 320->320 each caching
  its output, 2 decoder blocks (320 || 320) -> 320.  The headline stage.
* ``l32``    bf16, B=8, 32x32: encoder 320->640 (1x1 shortcut) and 640->640;
  decoder (640 || 640) -> 640 and (640 || 320) -> 640.  The 320-channel skip
  of the second decoder block is the stage input, which is therefore cached.
* ``l16`` / ``l8``  bf16, B=16, 16x16 / 8x8, C=1280, the ``l64`` structure at
  1280 channels.
* ``wave``   bf16: the four levels (64x64x320, 32x32x640, 16x16x1280,
  8x8x1280) at B=8 as four stage objects, 4 microbatches in flight.
"""

from __future__ import annotations

import copy

F32 = "f32"
BF16 = "bf16"


def _pair_stage(batch, hw, c, groups, temb_dim, dtype, n_blocks=2):
    enc = [dict(c_in=c, c_out=c, skip_slot_out=k) for k in range(n_blocks)]
    dec = [dict(c_up=c, c_skip=c, c_out=c, skip_slot_in=n_blocks - 1 - k)
           for k in range(n_blocks)]
    return dict(batch=batch, height=hw, width=hw, groups=groups, eps=1e-5,
                temb_dim=temb_dim, dtype=dtype, enc=enc, dec=dec,
                input_skip_slot=-1, max_inflight=1)


def tiny():
    d = _pair_stage(2, 16, 32, 8, 128, F32, n_blocks=1)
    return d


def l64(batch=8):
    return _pair_stage(batch, 64, 320, 32, 1280, BF16)


def l32(batch=8):
    enc = [dict(c_in=320, c_out=640, skip_slot_out=-1),
           dict(c_in=640, c_out=640, skip_slot_out=0)]
    dec = [dict(c_up=640, c_skip=640, c_out=640, skip_slot_in=0),
           dict(c_up=640, c_skip=320, c_out=640, skip_slot_in=1)]
    return dict(batch=batch, height=32, width=32, groups=32, eps=1e-5,
                temb_dim=1280, dtype=BF16, enc=enc, dec=dec,
                input_skip_slot=1, max_inflight=1)


def l16(batch=16):
    return _pair_stage(batch, 16, 1280, 32, 1280, BF16)


def l8(batch=16):
    return _pair_stage(batch, 8, 1280, 32, 1280, BF16)


def wave_levels(batch=8, inflight=4):
    """The four stage objects of the full collocated stage under the wave
    order, each allowed ``inflight`` microbatches."""
    levels = [l64(batch), l32(batch), l16(batch), l8(batch)]
    for d in levels:
        d["max_inflight"] = inflight
    return levels


CONFIGS = {
    "tiny": tiny,
    "l64": l64,
    "l32": l32,
    "l16": l16,
    "l8": l8,
}

SEEDS = {"tiny": 0, "l64": 2, "l32": 3, "l16": 4, "l8": 4, "wave": 5}


def get(name, **kw):
    return copy.deepcopy(CONFIGS[name](**kw))


def shrink(desc, batch=None, hw=None, width=None):
    """A copy of ``desc`` with a smaller batch / spatial extent (same
    channel structure), for parity cases that the oracle finishes quickly."""
    d = copy.deepcopy(desc)
    if batch is not None:
        d["batch"] = batch
    if hw is not None:
        d["height"] = hw
        d["width"] = hw if width is None else width
    elif width is not None:
        d["width"] = width
    return d


def slot_channels(desc):
    """Channel count of every skip slot, from the block that fills it."""
    out = {}
    if desc.get("input_skip_slot", -1) >= 0:
        out[int(desc["input_skip_slot"])] = int(desc["enc"][0]["c_in"])
    for b in desc["enc"]:
        if b["skip_slot_out"] >= 0:
            out[int(b["skip_slot_out"])] = int(b["c_out"])
    return out


def param_names(desc):
    """Parameter names and shapes in generation order: encoder blocks then
    decoder blocks; in a block W1 b1 Wl bl g1 be1 g2 be2 W2 b2 [Ws bs]."""
    out = []
    dt = int(desc["temb_dim"])
    blocks = [("enc", k, b["c_in"], b["c_out"]) for k, b in enumerate(desc["enc"])]
    blocks += [("dec", k, b["c_up"] + b["c_skip"], b["c_out"])
               for k, b in enumerate(desc["dec"])]
    for half, k, ci, co in blocks:
        pre = f"{half}{k}."
        out += [(pre + "W1", (co, 3, 3, ci)), (pre + "b1", (co,)),
                (pre + "Wl", (co, dt)), (pre + "bl", (co,)),
                (pre + "g1", (ci,)), (pre + "be1", (ci,)),
                (pre + "g2", (co,)), (pre + "be2", (co,)),
                (pre + "W2", (co, 3, 3, co)), (pre + "b2", (co,))]
        if ci != co:
            out += [(pre + "Ws", (co, ci)), (pre + "bs", (co,))]
    return out


# ---- transformer-block stages -----------------------------------------------

T_BLOCK = ("ln1.g", "ln1.b", "qkv.W", "qkv.b", "proj.W", "proj.b",
           "ln2.g", "ln2.b", "fc1.W", "fc1.b", "fc2.W", "fc2.b")


def _tstage(batch, tokens, width, heads, n_enc, n_dec, dtype=BF16):
    return dict(kind="transformer", batch=batch, tokens=tokens, width=width, heads=heads,
                eps=1e-5, mlp=4, n_enc=n_enc, n_dec=n_dec, dtype=dtype, max_inflight=1)


def t_tiny():
    """Small transformer stage: 2 x 64 tokens of 128 channels, 2 heads of 64."""
    return _tstage(2, 64, 128, 2, 1, 1)


def t768(batch=16):
    """UViT-like stage: 256 tokens (a 32x32 latent in 2x2 patches) of 768
    channels, 12 heads of 64, 2 encoder and 2 decoder blocks."""
    return _tstage(batch, 256, 768, 12, 2, 2)


def t1408(batch=8):
    """Hunyuan-DiT-like stage: 1024 tokens (a 64x64x4 latent in 2x2 patches)
    of 1408 channels, split into 22 heads of 64 (the attention kernels' head
    dimension), a 4x MLP, 1 encoder and 1 decoder block."""
    return _tstage(batch, 1024, 1408, 22, 1, 1)


CONFIGS["t_tiny"] = t_tiny
CONFIGS["t768"] = t768
CONFIGS["t1408"] = t1408
SEEDS["t_tiny"] = 6
SEEDS["t768"] = 7
SEEDS["t1408"] = 8


def tparam_names(desc):
    """Transformer-stage parameter names and shapes in generation order:
    encoder blocks, then decoder blocks (skip linear first)."""
    C, M = desc["width"], desc["width"] * desc["mlp"]
    shapes = {"ln1.g": (C,), "ln1.b": (C,), "qkv.W": (3 * C, C), "qkv.b": (3 * C,),
              "proj.W": (C, C), "proj.b": (C,), "ln2.g": (C,), "ln2.b": (C,),
              "fc1.W": (M, C), "fc1.b": (M,), "fc2.W": (C, M), "fc2.b": (C,)}
    out = []
    for k in range(desc["n_enc"]):
        out += [(f"enc{k}.{n}", shapes[n]) for n in T_BLOCK]
    for k in range(desc["n_dec"]):
        out += [(f"dec{k}.skip.W", (C, 2 * C)), (f"dec{k}.skip.b", (C,))]
        out += [(f"dec{k}.{n}", shapes[n]) for n in T_BLOCK]
    return out
