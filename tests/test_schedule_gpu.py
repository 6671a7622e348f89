"""The per-device schedule executor on the device: D skip-collocated stages
(one per device of a D-device pipeline, all on this GPU) wired into one
model -- encoder outputs feed the next device's encoder, decoder outputs the
previous device's decoder, and the gradients flow back the same way -- and
driven step by step through the wave schedule with pulse_sched_run_device.
Every boundary tensor and accumulated weight gradient equals bitwise what
one-microbatch-at-a-time runs of the same chain give, and for the fp32
configuration the composed model matches the oracle (the stage oracle
applied partition by partition)."""

import numpy as np
import pytest

from oracle import pulse_oracle as po
from paper_2606_19163_amd import configs, synth
from paper_2606_19163_amd import stage as S

from gpu_util import log, rel_l2

pytestmark = pytest.mark.gpu

OUTS = ("y_enc", "y_dec", "dx", "du")


def _bytes(t):
    import torch
    return t.contiguous().view(torch.uint8).cpu().numpy().tobytes()


def _pipeline(desc, D, M, seed):
    """Stages and wired per-(device, microbatch) io dicts.  Device d holds
    encoder partition d and decoder partition 2D-1-d."""
    import torch
    params, bounds = synth.make_wave([desc] * D, seed, M)
    sts = []
    for d in range(D):
        st = S.Stage(desc)
        st.set_params(params[d])
        st.zero_grads()
        sts.append(st)
    io = [[{} for _ in range(M)] for _ in range(D)]
    c_enc = desc["enc"][-1]["c_out"]
    c_dec = desc["dec"][-1]["c_out"]
    for d in range(D):
        for m in range(M):
            e = io[d][m]
            e["y_enc"] = sts[d].act(c_enc)
            e["y_dec"] = sts[d].act(c_dec)
            e["dx"] = sts[d].act(desc["enc"][0]["c_in"])
            e["du"] = sts[d].act(desc["dec"][0]["c_up"])
            e["dtemb"] = torch.zeros((desc["batch"], desc["temb_dim"]), dtype=torch.float32,
                                     device="cuda")
    host = []
    for m in range(M):
        b = bounds[0][m]
        host.append(dict(x=b["x"], temb=b["temb"], g_dec=b["g_dec"]))
    for m in range(M):
        temb = sts[0].to_dev(host[m]["temb"])
        for d in range(D):
            e = io[d][m]
            e["temb"] = temb
            e["x"] = sts[0].to_dev(host[m]["x"]) if d == 0 else io[d - 1][m]["y_enc"]
            e["u"] = io[d + 1][m]["y_dec"] if d + 1 < D else e["y_enc"]
            e["g_dec"] = sts[0].to_dev(host[m]["g_dec"]) if d == 0 else io[d - 1][m]["du"]
            e["g_enc"] = io[d + 1][m]["dx"] if d + 1 < D else e["du"]
    return sts, io, params, host


def _sequential(sts, io, D, M):
    """The same chain, one microbatch at a time, through the stage calls."""
    for m in range(M):
        for d in range(D):
            e = io[d][m]
            sts[d].forward(S.ENC, m, e["x"], e["temb"], out=e["y_enc"])
        for d in reversed(range(D)):
            e = io[d][m]
            sts[d].forward(S.DEC, m, e["u"], e["temb"], out=e["y_dec"])
        for d in range(D):
            e = io[d][m]
            sts[d].backward(S.DEC, m, e["g_dec"], din=e["du"], dtemb=e["dtemb"])
        for d in reversed(range(D)):
            e = io[d][m]
            sts[d].backward(S.ENC, m, e["g_enc"], din=e["dx"], dtemb=e["dtemb"])


def _snapshot(sts, io, D, M):
    import torch
    torch.cuda.synchronize()
    out = {}
    for d in range(D):
        out[("grads", d)] = _bytes(sts[d].grads)
        for m in range(M):
            for k in OUTS + ("dtemb",):
                out[(k, d, m)] = _bytes(io[d][m][k])
    return out


def _scheduled(sts, io, D, M, table):
    T = len(table[0])
    for t in range(T):
        for d in range(D):
            S.sched_run_device(sts[d], D, d, M, table, io[d], t0=t, t1=t + 1)


@pytest.mark.parametrize("name,D,M", [("l64", 2, 3), ("l64", 3, 4), ("tiny", 2, 3)])
def test_scheduled_pipeline_matches_sequential(name, D, M):
    import torch
    desc = configs.shrink(configs.get(name), batch=2, hw=8) if name != "tiny" \
        else configs.tiny()
    desc["max_inflight"] = M
    table, exact = S.sched_build(D, M)
    log(f"case schedule {name} D={D} M={M} T={len(table[0])} exact={exact}")
    sts, io, params, host = _pipeline(desc, D, M, configs.SEEDS["wave"] + D)
    _scheduled(sts, io, D, M, table)
    for st in sts:
        assert st.inflight() == 0
    got = _snapshot(sts, io, D, M)
    # the same chain, microbatch by microbatch
    for d in range(D):
        sts[d].zero_grads()
        for m in range(M):
            for k in OUTS:
                io[d][m][k].zero_()
            io[d][m]["dtemb"].zero_()
    _sequential(sts, io, D, M)
    ref = _snapshot(sts, io, D, M)
    bad = [k for k in got if got[k] != ref[k]]
    assert not bad, bad[:8]

    if desc["dtype"] != configs.F32:
        return
    # the composed model against the oracle, partition by partition
    log(f"case schedule {name}: oracle composition")
    zeros_u = np.zeros((desc["batch"], desc["height"], desc["width"],
                        desc["dec"][0]["c_up"]))
    zeros_e = np.zeros((desc["batch"], desc["height"], desc["width"],
                        desc["enc"][-1]["c_out"]))
    gsum = [None] * D
    for m in range(M):
        temb = host[m]["temb"]
        x = [None] * D
        y_enc = [None] * D
        for d in range(D):
            x[d] = host[m]["x"] if d == 0 else y_enc[d - 1]
            y_enc[d] = po.stage_forward_only(desc, params[d], x[d], zeros_u, temb)["y_enc"]
        u = [None] * D
        y_dec = [None] * D
        for d in reversed(range(D)):
            u[d] = y_dec[d + 1] if d + 1 < D else y_enc[d]
            y_dec[d] = po.stage_forward_only(desc, params[d], x[d], u[d], temb)["y_dec"]
        # decoder backward chain (does not depend on g_enc)
        g_dec = [None] * D
        du = [None] * D
        for d in range(D):
            g_dec[d] = host[m]["g_dec"] if d == 0 else du[d - 1]
            du[d] = po.stage_run(desc, params[d], x[d], u[d], temb, zeros_e, g_dec[d])["du"]
        dx = [None] * D
        for d in reversed(range(D)):
            g_enc = dx[d + 1] if d + 1 < D else du[d]
            r = po.stage_run(desc, params[d], x[d], u[d], temb, g_enc, g_dec[d])
            dx[d] = r["dx"]
            want = dict(y_enc=y_enc[d], y_dec=y_dec[d], dx=r["dx"], du=r["du"],
                        dtemb=r["dtemb"])
            for k, v in want.items():
                g = io[d][m][k].float().cpu().numpy()
                e = rel_l2(g, v)
                assert e <= 1e-4, (d, m, k, e)
            gsum[d] = r["grads"] if gsum[d] is None else \
                {n: gsum[d][n] + r["grads"][n] for n in r["grads"]}
    for d in range(D):
        gd = sts[d].grads_dict()
        for n, v in gsum[d].items():
            e = rel_l2(gd[n], v)
            assert e <= 1e-4, (d, n, e)
