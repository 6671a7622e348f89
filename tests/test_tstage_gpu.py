"""GPU parity of the transformer-block stage (C ABI) against the fp64 oracle:
outputs, boundary gradients, every parameter gradient and the buffered skip
gradients, element by element (relative L2 within the bf16 bound)."""

import numpy as np
import pytest

from oracle import transformer_oracle as TO
from paper_2606_19163_amd import configs, synth
from paper_2606_19163_amd import tstage as TS

from gpu_util import log, rel_l2

pytestmark = pytest.mark.gpu

TOL = 2e-2  # bf16 storage of activations and weights, fp32 accumulation


def _mid():
    """Ragged tiles: 576 tokens (4.5 row tiles of 128), width 192 (3 heads;
    192- and 576-column GEMMs end in half tiles), 2 + 2 blocks."""
    d = configs._tstage(3, 192, 192, 3, 2, 2)
    return d


def _narrow():
    """128 tokens (the attention kernels' L = 128 instance), one image,
    width 256 in 4 heads, a 2x MLP, 1 + 1 blocks."""
    d = configs._tstage(1, 128, 256, 4, 1, 1)
    d["mlp"] = 2
    return d


def _t320():
    """320 tokens: the streamed attention kernels over five 64-token chunks
    (an odd count), one image, 2 heads, 1 + 1 blocks."""
    return configs._tstage(1, 320, 128, 2, 1, 1)


def _long():
    """1024 tokens per image (the Hunyuan-DiT-like sequence length), two
    images, width 256 in 4 heads, 1 + 1 blocks."""
    return configs._tstage(2, 1024, 256, 4, 1, 1)


def _t4096():
    """The longest sequence the stage takes: 4096 tokens, one image, 2 heads,
    1 + 1 blocks (32 forward chunks, 64 streamed backward chunks)."""
    return configs._tstage(1, 4096, 128, 2, 1, 1)


def _t1408_b2():
    """The Hunyuan-DiT-like stage at its full per-image shape (1024 tokens,
    width 1408 in 22 heads, MLP 5632) with two images (GEMMs that fit one
    round of tiles).  The "t1408" case runs the benchmarked batch of 8, whose
    GEMMs take the multi-round plan (128 x 192 conv tiles, 320 x 128
    weight-gradient tiles over 8192 tokens)."""
    return configs.t1408(batch=2)


CASES = {"t_tiny": (configs.t_tiny, 6), "t_mid": (_mid, 11), "t_narrow": (_narrow, 12),
         "t768": (configs.t768, 7), "t_320": (_t320, 13), "t_long": (_long, 14),
         "t_4096": (_t4096, 15), "t1408_b2": (_t1408_b2, 8), "t1408": (configs.t1408, 8)}


def run_gpu(desc, params, b, mbs=(0,)):
    import torch
    st = TS.TStage(desc)
    st.set_params(params)
    st.zero_grads()
    dev = {k: st.to_dev(v) for k, v in b.items()}
    res = {}
    for mb in mbs:
        ye = st.forward(TS.ENC, mb, dev["x"])
        yd = st.forward(TS.DEC, mb, dev["u"])
        du = st.backward(TS.DEC, mb, dev["g_dec"])
        dsk = {k: st.skip_grad(mb, k) for k in range(desc["n_enc"])}
        dx = st.backward(TS.ENC, mb, dev["g_enc"])
        torch.cuda.synchronize()
        res = dict(y_enc=ye.float().cpu().numpy(), y_dec=yd.float().cpu().numpy(),
                   du=du.float().cpu().numpy(), dx=dx.float().cpu().numpy(),
                   dskips={k: v.cpu().numpy() for k, v in dsk.items()})
    res["grads"] = st.grads_dict()
    assert st.inflight() == 0
    return res, st


def _compare(name, got, ref, scale=1.0):
    worst = 0.0
    for k in ("y_enc", "y_dec", "dx", "du"):
        e = rel_l2(got[k], ref[k])
        log(f"{name} {k}: rel {e:.3e}")
        assert e < TOL, (k, e)
    for k in ref["dskips"]:
        e = rel_l2(got["dskips"][k], ref["dskips"][k])
        log(f"{name} dskip[{k}]: rel {e:.3e}")
        assert e < TOL, ("dskip", k, e)
    for k, v in ref["grads"].items():
        e = rel_l2(got["grads"][k], scale * np.asarray(v))
        worst = max(worst, e)
        assert e < TOL, (k, e)
    log(f"{name} worst parameter-gradient rel {worst:.3e}")


@pytest.mark.parametrize("name", list(CASES))
def test_tstage_matches_oracle(name):
    make, seed = CASES[name]
    d = make()
    log(f"case {name}: batch {d['batch']} tokens {d['tokens']} width {d['width']} "
        f"heads {d['heads']} blocks {d['n_enc']}+{d['n_dec']}")
    p, b = synth.make_tstage(d, seed)
    ref = TO.tstage_run(d, p, b["x"], b["u"], b["g_enc"], b["g_dec"])
    got, _ = run_gpu(d, p, b)
    _compare(name, got, ref)


def test_gradients_accumulate_over_microbatches():
    d = configs.t_tiny()
    d["max_inflight"] = 2
    p, b = synth.make_tstage(d, 6)
    ref = TO.tstage_run(d, p, b["x"], b["u"], b["g_enc"], b["g_dec"])
    got, _ = run_gpu(d, p, b, mbs=(3, 5))
    _compare("two microbatches", got, ref, scale=2.0)


def test_interleaved_microbatches_keep_their_skips():
    """Two microbatches in flight with different inputs, run in a pipeline
    order (F_enc 0, F_enc 1, F_dec 1, F_dec 0, B_dec 0, B_dec 1, B_enc 1,
    B_enc 0): each microbatch's outputs and gradients match its own oracle."""
    import torch
    d = configs.t_tiny()
    d["max_inflight"] = 2
    p, b0 = synth.make_tstage(d, 6)
    _, b1 = synth.make_tstage(d, 16)
    refs = [TO.tstage_run(d, p, bb["x"], bb["u"], bb["g_enc"], bb["g_dec"]) for bb in (b0, b1)]
    st = TS.TStage(d)
    st.set_params(p)
    st.zero_grads()
    dev = [{k: st.to_dev(v) for k, v in bb.items()} for bb in (b0, b1)]
    ye = [st.forward(TS.ENC, m, dev[m]["x"]) for m in (0, 1)]
    yd = [None, None]
    yd[1] = st.forward(TS.DEC, 1, dev[1]["u"])
    yd[0] = st.forward(TS.DEC, 0, dev[0]["u"])
    du = [st.backward(TS.DEC, m, dev[m]["g_dec"]) for m in (0, 1)]
    dx = [None, None]
    dx[1] = st.backward(TS.ENC, 1, dev[1]["g_enc"])
    dx[0] = st.backward(TS.ENC, 0, dev[0]["g_enc"])
    torch.cuda.synchronize()
    for m in (0, 1):
        for k, t in (("y_enc", ye[m]), ("y_dec", yd[m]), ("du", du[m]), ("dx", dx[m])):
            e = rel_l2(t.float().cpu().numpy(), refs[m][k])
            log(f"mb {m} {k}: rel {e:.3e}")
            assert e < TOL, (m, k, e)
    g = st.grads_dict()
    for k in refs[0]["grads"]:
        e = rel_l2(g[k], np.asarray(refs[0]["grads"][k]) + np.asarray(refs[1]["grads"][k]))
        assert e < TOL, (k, e)


@pytest.mark.parametrize("tile", range(4))
def test_tstage_every_conv_tile(tile, monkeypatch):
    """Every conv-mode tile shape (128x160, 128x128, 128x192, 64x128 with
    three stages) on the token-major linear layers (ragged rows and
    columns)."""
    monkeypatch.setenv("PULSE_TCONV_TILE", str(tile))
    d = _mid()
    p, b = synth.make_tstage(d, 11)
    ref = TO.tstage_run(d, p, b["x"], b["u"], b["g_enc"], b["g_dec"])
    got, _ = run_gpu(d, p, b)
    _compare(f"conv tile {tile}", got, ref)


@pytest.mark.parametrize("tile", [20, 21])
def test_tstage_every_wgrad_tile(tile, monkeypatch):
    monkeypatch.setenv("PULSE_TWGRAD_TILE", str(tile))
    d = _mid()
    p, b = synth.make_tstage(d, 11)
    ref = TO.tstage_run(d, p, b["x"], b["u"], b["g_enc"], b["g_dec"])
    got, _ = run_gpu(d, p, b)
    _compare(f"wgrad tile {tile}", got, ref)


@pytest.mark.parametrize("D,M", [(2, 3), (3, 4)])
def test_scheduled_transformer_pipeline(D, M):
    """D transformer stages on this GPU wired as the devices of a D-device
    pipeline (encoder outputs feed the next device's encoder, decoder
    outputs the previous device's decoder, gradients flow back), driven one
    step at a time through the wave schedule with pulse_tsched_run_device:
    every boundary tensor and weight gradient equals bitwise the
    microbatch-at-a-time run of the same chain, and the composed model
    matches the oracle applied partition by partition."""
    import torch
    from paper_2606_19163_amd import stage as S
    table, exact = S.sched_build(D, M)
    need = max(S.sched_inflight(D, M, table))
    log(f"case transformer schedule D={D} M={M} T={len(table[0])} in flight {need}")
    desc = configs.t_tiny()
    desc["max_inflight"] = need
    sts, params = [], []
    for d in range(D):
        p, _ = synth.make_tstage(desc, 40 + d)
        st = TS.TStage(desc)
        st.set_params(p)
        st.zero_grads()
        sts.append(st)
        params.append(p)
    host = [synth.make_tstage(desc, 80 + m)[1] for m in range(M)]
    io = [[{k: sts[d].act() for k in ("y_enc", "y_dec", "dx", "du")} for _ in range(M)]
          for d in range(D)]
    for m in range(M):
        for d in range(D):
            e = io[d][m]
            e["x"] = sts[0].to_dev(host[m]["x"]) if d == 0 else io[d - 1][m]["y_enc"]
            e["u"] = io[d + 1][m]["y_dec"] if d + 1 < D else e["y_enc"]
            e["g_dec"] = sts[0].to_dev(host[m]["g_dec"]) if d == 0 else io[d - 1][m]["du"]
            e["g_enc"] = io[d + 1][m]["dx"] if d + 1 < D else e["du"]

    def snap():
        torch.cuda.synchronize()
        out = {}
        for d in range(D):
            out[("grads", d)] = sts[d].grads.cpu().numpy().tobytes()
            for m in range(M):
                for k in ("y_enc", "y_dec", "dx", "du"):
                    out[(k, d, m)] = io[d][m][k].view(torch.uint16).cpu().numpy().tobytes()
        return out

    for t in range(len(table[0])):
        for d in range(D):
            TS.tsched_run_device(sts[d], D, d, M, table, io[d], t0=t, t1=t + 1)
    for st in sts:
        assert st.inflight() == 0
    got = snap()
    for d in range(D):
        sts[d].zero_grads()
    for m in range(M):
        for d in range(D):
            e = io[d][m]
            sts[d].forward(TS.ENC, m, e["x"], out=e["y_enc"])
        for d in reversed(range(D)):
            e = io[d][m]
            sts[d].forward(TS.DEC, m, e["u"], out=e["y_dec"])
        for d in range(D):
            e = io[d][m]
            sts[d].backward(TS.DEC, m, e["g_dec"], din=e["du"])
        for d in reversed(range(D)):
            e = io[d][m]
            sts[d].backward(TS.ENC, m, e["g_enc"], din=e["dx"])
    ref = snap()
    bad = [k for k in got if got[k] != ref[k]]
    assert not bad, bad[:8]
    # the composed model against the oracle (bf16 bound)
    zeros = np.zeros_like(host[0]["x"])
    for m in range(M):
        x, ye = [None] * D, [None] * D
        for d in range(D):
            x[d] = host[m]["x"] if d == 0 else ye[d - 1]
            ye[d] = TO.tstage_forward_only(desc, params[d], x[d], zeros)["y_enc"]
        u, yd = [None] * D, [None] * D
        for d in reversed(range(D)):
            u[d] = yd[d + 1] if d + 1 < D else ye[d]
            yd[d] = TO.tstage_forward_only(desc, params[d], x[d], u[d])["y_dec"]
        gd, du = [None] * D, [None] * D
        for d in range(D):
            gd[d] = host[m]["g_dec"] if d == 0 else du[d - 1]
            du[d] = TO.tstage_run(desc, params[d], x[d], u[d], zeros, gd[d])["du"]
        dx = [None] * D
        for d in reversed(range(D)):
            ge = dx[d + 1] if d + 1 < D else du[d]
            r = TO.tstage_run(desc, params[d], x[d], u[d], ge, gd[d])
            dx[d] = r["dx"]
            for k, v in (("y_enc", ye[d]), ("y_dec", yd[d]), ("du", r["du"]), ("dx", r["dx"])):
                e = rel_l2(io[d][m][k].float().cpu().numpy(), v)
                assert e < TOL, (d, m, k, e)


@pytest.mark.parametrize("name", ["t_tiny", "t_long"])
def test_tstage_reruns_are_bitwise_identical(name):
    """Every reduction of the stage (attention merges, LayerNorm and bias
    sums, split-K finalizes) runs in a fixed order, also with the parameter
    gradients on the side stream: two runs from zeroed gradients agree
    bitwise in every output, boundary gradient, skip gradient and parameter
    gradient (64 tokens: whole-tile backward; 1024: the streamed kernels)."""
    make, seed = CASES[name]
    d = make()
    p, b = synth.make_tstage(d, seed)
    first, _ = run_gpu(d, p, b)
    second, _ = run_gpu(d, p, b)
    for k in ("y_enc", "y_dec", "du", "dx"):
        assert np.array_equal(first[k], second[k]), k
    for k in first["dskips"]:
        assert np.array_equal(first["dskips"][k], second["dskips"][k]), ("dskip", k)
    for k in first["grads"]:
        assert np.array_equal(first["grads"][k], second["grads"][k]), k
    log(f"{name}: two runs bitwise identical")
