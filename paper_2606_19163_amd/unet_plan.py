"""Skip-aware partition of a UNet built from the four measured stage levels.

    python -m paper_2606_19163_amd.unet_plan [--batch 8] [--reps 20]

The UNet is the sixteen ResBlocks of the 64x64x320, 32x32x640, 16x16x1280
and 8x8x1280 levels in model order (encoder blocks of each level going down,
then decoder blocks coming up), with the long skips of those levels: each
decoder block reads the encoder output its level caches for it, and the
second 32x32 decoder block reads the 32x32 level's input, the output of the
last 64x64 encoder block.  Every block's forward time is measured on this
GPU through the stage ABI (a one-block stage per ResBlock shape, HIP events
around the forward call), every block's output size is its bf16 activation.
The partitioner (pulse_partition, Sec. IV-B) then splits the sequence for
2 and 4 devices, beside the block-wise split (equal ResBlocks per stage),
and one JSON line reports both.
"""

from __future__ import annotations

import argparse
import json

from . import configs, plan, synth
from . import stage as S

XGMI_BYTES_PER_S = 153e9   # one MI355X xGMI link
T_LAT_S = 10e-6            # per-transfer latency taken for the link


def unet_ops(batch=8):
    """(ops, skips): ops in model order as dicts (name, half, level desc,
    block), skips as op-index pairs."""
    levels = [("64", configs.l64(batch)), ("32", configs.l32(batch)),
              ("16", configs.l16(batch)), ("8", configs.l8(batch))]
    ops, enc_index, slot_owner = [], {}, {}
    for name, d in levels:
        for k, b in enumerate(d["enc"]):
            enc_index[(name, k)] = len(ops)
            ops.append(dict(name=f"E{name}.{k}", half=S.ENC, level=d, block=b))
    skips = []
    prev_level_out = None  # op whose output enters the level
    for name, d in levels:
        owner = {}
        if d.get("input_skip_slot", -1) >= 0:
            owner[d["input_skip_slot"]] = prev_level_out
        for k, b in enumerate(d["enc"]):
            if b["skip_slot_out"] >= 0:
                owner[b["skip_slot_out"]] = enc_index[(name, k)]
        slot_owner[name] = owner
        prev_level_out = enc_index[(name, len(d["enc"]) - 1)]
    for name, d in reversed(levels):
        for k, b in enumerate(d["dec"]):
            i = len(ops)
            ops.append(dict(name=f"D{name}.{k}", half=S.DEC, level=d, block=b))
            src = slot_owner[name].get(b["skip_slot_in"])
            if src is not None:
                skips.append((src, i))
    return ops, skips


def out_bytes(op):
    d, b = op["level"], op["block"]
    return d["batch"] * d["height"] * d["width"] * b["c_out"] * 2


def block_stage(op):
    """A stage holding the op's block and the smallest partner the ABI needs
    (a decoder block reading the encoder block's output, or an encoder
    block producing the decoder block's skip)."""
    d, b = op["level"], op["block"]
    desc = {k: d[k] for k in ("batch", "height", "width", "groups", "eps", "temb_dim", "dtype")}
    desc["input_skip_slot"] = -1
    desc["max_inflight"] = 1
    if op["half"] == S.ENC:
        desc["enc"] = [dict(c_in=b["c_in"], c_out=b["c_out"], skip_slot_out=0)]
        desc["dec"] = [dict(c_up=b["c_out"], c_skip=b["c_out"], c_out=b["c_out"],
                            skip_slot_in=0)]
    else:
        desc["enc"] = [dict(c_in=b["c_skip"], c_out=b["c_skip"], skip_slot_out=0)]
        desc["dec"] = [dict(c_up=b["c_up"], c_skip=b["c_skip"], c_out=b["c_out"],
                            skip_slot_in=0)]
    return desc


def time_forward(op, reps=20, warmup=3, seed=0):
    """Median forward time (s) of the op's block at its level's batch."""
    import torch
    desc = block_stage(op)
    params, b = synth.make_all(desc, seed)
    st = S.Stage(desc)
    st.set_params(params)
    db = {k: st.to_dev(v) for k, v in b.items()}
    times = []
    for r in range(warmup + reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if op["half"] == S.ENC:
            a.record()
            st.forward(S.ENC, 0, db["x"], db["temb"])
            e.record()
        else:
            st.forward(S.ENC, 0, db["x"], db["temb"])
            a.record()
            st.forward(S.DEC, 0, db["u"], db["temb"])
            e.record()
        e.synchronize()
        st.release(0)
        if r >= warmup:
            times.append(a.elapsed_time(e) * 1e-3)
    times.sort()
    return times[len(times) // 2]


def param_bytes(op):
    """Bytes of the block's parameters at 2 bytes each (the half-precision
    weights the memory model's factor 7 counts)."""
    d, b = op["level"], op["block"]
    c_in = b["c_in"] if op["half"] == S.ENC else b["c_up"] + b["c_skip"]
    c_out = b["c_out"]
    n = 9 * c_in * c_out + c_out            # conv1
    n += d["temb_dim"] * c_out + c_out      # timestep linear
    n += 2 * c_in + 2 * c_out               # GroupNorm affines
    n += 9 * c_out * c_out + c_out          # conv2
    if c_in != c_out:
        n += c_in * c_out + c_out           # 1x1 shortcut
    return 2.0 * n


def act_bytes_per_sample(op):
    """Bytes the stage keeps per sample for the block's backward: its
    GroupNorm+SiLU input a1 (all input channels), h1, a2 and the output, in
    bf16."""
    d, b = op["level"], op["block"]
    c_in = b["c_in"] if op["half"] == S.ENC else b["c_up"] + b["c_skip"]
    return 2.0 * d["height"] * d["width"] * (c_in + 3 * b["c_out"])


def out_bytes_per_sample(op):
    d, b = op["level"], op["block"]
    return 2.0 * d["height"] * d["width"] * b["c_out"]


def blockwise_cuts(n, p):
    per = n // p
    return [per * (k + 1) - 1 for k in range(p - 1)]


def partition_report(names, t_f, m_a, skips, batch):
    """Balanced skip-aware partitions for 4 and 8 stages (with and without
    the communication term) beside the block-wise split, and the forward
    point-to-point bytes per sample of each collocated plan against a
    sequential pipeline on the same devices."""
    n = len(names)
    out = {"batch": batch, "ops": list(names), "forward_us": [round(t * 1e6, 2) for t in t_f],
           "skips": skips, "plans": []}
    for p in (4, 8):
        for lam in (0.0, 1.0):
            kw = dict(lam=lam, t_lat=T_LAT_S, b_inter=XGMI_BYTES_PER_S)
            cuts, cost = plan.partition(t_f, m_a, skips, p, **kw)
            _, _, sc = plan.partition_cost(t_f, m_a, skips, p, cuts, **kw)
            bw = blockwise_cuts(n, p)
            bcost, bvalid, bsc = plan.partition_cost(t_f, m_a, skips, p, bw, **kw)
            # forward point-to-point bytes per sample: this collocated plan
            # against a sequential pipeline of p / 2 stages balanced on the
            # same forward times (skips forwarded stage to stage)
            D = p // 2
            per = 1.0 / batch
            pulse_b = plan.comm_volume(m_a, skips, p, cuts, True) * per
            seq_cuts, _ = plan.partition(t_f, m_a, [], D) if D % 2 == 0 else \
                (blockwise_cuts(n, D), 0.0)
            seq_b = plan.comm_volume(m_a, skips, D, seq_cuts, False) * per
            out["plans"].append({
                "stages": p, "devices": D, "lambda": lam,
                "comm_mb_per_sample": {"sequential": round(seq_b / 1e6, 3),
                                       "sequential_cuts": seq_cuts,
                                       "collocated": round(pulse_b / 1e6, 3),
                                       "reduction_pct": round(100 * (1 - pulse_b / seq_b), 1)},
                "balanced": {"cuts": cuts, "max_stage_us": round(cost * 1e6, 2),
                             "stage_us": [round(v * 1e6, 2) for v in sc]},
                "blockwise": {"cuts": bw, "valid": bvalid,
                              "max_stage_us": round(max(bsc) * 1e6, 2),
                              "stage_us": [round(v * 1e6, 2) for v in bsc]},
                "reduction_pct": round(100.0 * (1.0 - cost / max(bsc)), 1),
            })
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--tune", action="store_true",
                    help="also time every block at microbatch 1, 2, 4, 8, 16 and run the "
                         "hybrid tuner for 8, 16 and 32 devices at two memory limits")
    args = ap.parse_args()
    import torch
    torch.cuda.set_device(0)
    ops, skips = unet_ops(args.batch)
    t_f = []
    for op in ops:
        t_f.append(time_forward(op, args.reps))
        print(f"# {op['name']}: {t_f[-1] * 1e6:.1f} us", flush=True)
    m_a = [float(out_bytes(op)) for op in ops]
    out = partition_report([o["name"] for o in ops], t_f, m_a, skips, args.batch)
    if args.tune:
        out["tune"] = tune_report(args.reps)
    print(json.dumps(out), flush=True)


B_INTER_NODE = 50e9    # one 400 Gb/s network port per device between nodes
B_INTRA_NODE = 300e9   # ring all-reduce over the xGMI mesh of one node
M_LIMITS = (288e9, 6e9)  # HBM3E per MI355X, and a tight budget that binds


def tune_report(reps, bs=(1, 2, 4, 8, 16)):
    ops, skips = unet_ops(8)
    t_f = []
    for b in bs:
        row = []
        for op in ops:
            o = dict(op, level=dict(op["level"], batch=b))
            row.append(time_forward(o, reps))
        t_f.append(row)
        print(f"# b={b}: " + " ".join(f"{v * 1e6:.0f}" for v in row), flush=True)
    m_theta = [param_bytes(o) for o in ops]
    m_a = [act_bytes_per_sample(o) for o in ops]
    m_o = [out_bytes_per_sample(o) for o in ops]
    return tune_choices(bs, t_f, m_theta, m_a, m_o, skips)


def tune_choices(bs, t_f, m_theta, m_a, m_o, skips):
    """The hybrid tuner (Sec. VI) for 8, 16 and 32 devices at each memory
    limit, from per-op forward times t_f[b_index][op] and byte counts."""
    res = {"bs": list(bs), "forward_us": [[round(v * 1e6, 2) for v in r] for r in t_f],
           "b_inter": B_INTER_NODE, "b_intra": B_INTRA_NODE, "t_lat": T_LAT_S,
           "choices": []}
    for m_limit in M_LIMITS:
        for N in (8, 16, 32):
            best, rows = plan.tune(N, list(bs), t_f, m_theta, m_a, m_o, skips, lam=1.0,
                                   t_lat=T_LAT_S, b_inter=B_INTER_NODE, b_intra=B_INTRA_NODE,
                                   m_limit=m_limit)
            res["choices"].append({"devices": N, "m_limit": m_limit, "best": best,
                                   "rows": rows})
    return res


if __name__ == "__main__":
    main()
