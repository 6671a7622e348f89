"""Skip-aware partition and hybrid tuning of transformer-block diffusion
models (UViT, Hunyuan-DiT).

    python -m paper_2606_19163_amd.uvit_plan [--model uvit|hdit] [--batch B]
                                             [--reps 20] [--tune]

The models keep the layout of Sec. II-A and Sec. VII: encoder blocks, an
optional middle block and decoder blocks, with a long skip from encoder
block i to decoder block n_in - 1 - i (mirror order; the decoder block
applies its skip linear over [upstream || skip] first).
  uvit: 8 + 1 + 8 blocks of width 768, 12 heads, 256 tokens (a 32x32 latent
        in 2x2 patches), timed at batch 16;
  hdit: 20 + 20 blocks (no middle block) of width 1408 in 22 heads of 64,
        1024 tokens (a 64x64 latent in 2x2 patches), timed at batch 32 (the
        microbatch of the paper's partition figure).
Every block's forward time is measured on this GPU through the transformer
stage ABI: a one-block-each stage, HIP events around the ENC forward (an
encoder or the middle block) or around the DEC forward (skip linear +
block).  The partitioner (pulse_partition, Sec. IV-B) splits the sequence
for 2 and 4 devices beside the block-wise split and reports the
point-to-point traffic of the collocated plan against a sequential pipeline
(Sec. II-C); with --tune the hybrid tuner (Sec. VI) runs on
per-microbatch-size times.
"""

from __future__ import annotations

import argparse
import json

from . import configs, synth
from . import tstage as TS
from .unet_plan import partition_report, tune_choices

MODELS = {
    "uvit": dict(width=768, heads=12, tokens=256, mlp=4, n_in=8, mid=True, batch=16,
                 tune_bs=(1, 2, 4, 8, 16)),
    "hdit": dict(width=1408, heads=22, tokens=1024, mlp=4, n_in=20, mid=False, batch=32,
                 tune_bs=(1, 2, 4, 8, 16, 32)),
}


def uvit_ops(n_in=8, mid=True):
    """(names, kinds, skips): ops in model order, kind "enc" for encoder and
    middle blocks, "dec" for decoder blocks, skips as op-index pairs."""
    names = [f"in{i}" for i in range(n_in)] + (["mid"] if mid else []) + \
        [f"out{i}" for i in range(n_in)]
    kinds = ["enc"] * (n_in + (1 if mid else 0)) + ["dec"] * n_in
    first_out = n_in + (1 if mid else 0)
    skips = [(i, first_out + n_in - 1 - i) for i in range(n_in)]  # in_i -> out_(n_in-1-i)
    return names, kinds, skips


def time_forward(kind, batch, reps=20, warmup=3, seed=0, model=None):
    """Median forward time (s) of one encoder block ("enc") or one decoder
    block with its skip linear ("dec") at `batch` images."""
    import torch
    m = model or MODELS["uvit"]
    desc = configs._tstage(batch, m["tokens"], m["width"], m["heads"], 1, 1)
    desc["mlp"] = m["mlp"]
    params, b = synth.make_tstage(desc, seed)
    st = TS.TStage(desc)
    st.set_params(params)
    x, u = st.to_dev(b["x"]), st.to_dev(b["u"])
    times = []
    for r in range(warmup + reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if kind == "enc":
            a.record()
            st.forward(TS.ENC, 0, x)
            e.record()
        else:
            st.forward(TS.ENC, 0, x)
            a.record()
            st.forward(TS.DEC, 0, u)
            e.record()
        e.synchronize()
        st.release(0)
        if r >= warmup:
            times.append(a.elapsed_time(e) * 1e-3)
    times.sort()
    return times[len(times) // 2]


def param_bytes(kind, model=None):
    """Parameters of one block at 2 bytes each (the memory model's
    half-precision weights)."""
    m = model or MODELS["uvit"]
    C, R = m["width"], m["mlp"] * m["width"]
    n = 4 * C + 3 * C * C + 3 * C + C * C + C + R * C + R + C * R + C
    if kind == "dec":
        n += 2 * C * C + C
    return 2.0 * n


def act_bytes_per_sample(kind, model=None):
    """bf16 activations the stage keeps per sample for a block's backward:
    per token the block input, a, qkv, o, h, a2 (8 widths) and z, GELU(z)
    (2 MLP widths), plus the skip linear's upstream input for a decoder
    block."""
    m = model or MODELS["uvit"]
    C, R = m["width"], m["mlp"] * m["width"]
    per_token = 8 * C + 2 * R + (C if kind == "dec" else 0)
    return 2.0 * m["tokens"] * per_token


def out_bytes_per_sample(model=None):
    m = model or MODELS["uvit"]
    return 2.0 * m["tokens"] * m["width"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", choices=sorted(MODELS), default="uvit")
    ap.add_argument("--batch", type=int, default=None,
                    help="microbatch of the partition (default: the model's)")
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--tune", action="store_true",
                    help="also time the blocks at each microbatch size up to the model's and "
                         "run the hybrid tuner for 8, 16 and 32 devices at two memory limits")
    args = ap.parse_args()
    import torch
    torch.cuda.set_device(0)
    m = MODELS[args.model]
    batch = args.batch or m["batch"]
    names, kinds, skips = uvit_ops(m["n_in"], m["mid"])
    t_kind = {k: time_forward(k, batch, args.reps, model=m) for k in ("enc", "dec")}
    for k, v in t_kind.items():
        print(f"# {k} block at batch {batch}: {v * 1e6:.1f} us", flush=True)
    t_f = [t_kind[k] for k in kinds]
    m_a = [batch * out_bytes_per_sample(m)] * len(names)
    out = partition_report(names, t_f, m_a, skips, batch)
    out["model"] = {"name": args.model, "width": m["width"], "heads": m["heads"],
                    "tokens": m["tokens"], "mlp": m["mlp"],
                    "blocks": [m["n_in"], 1 if m["mid"] else 0, m["n_in"]]}
    if args.tune:
        bs = tuple(b for b in m["tune_bs"] if b <= batch)
        rows = []
        for b in bs:
            tk = {k: time_forward(k, b, args.reps, model=m) for k in ("enc", "dec")}
            rows.append([tk[k] for k in kinds])
            print(f"# b={b}: enc {tk['enc'] * 1e6:.0f} us, dec {tk['dec'] * 1e6:.0f} us",
                  flush=True)
        out["tune"] = tune_choices(bs, rows, [param_bytes(k, m) for k in kinds],
                                   [act_bytes_per_sample(k, m) for k in kinds],
                                   [out_bytes_per_sample(m)] * len(kinds), skips)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
