"""A whole stage step (forward and backward of both halves of one
microbatch) captured into a HIP graph and replayed gives the eager results
bitwise: the 64x64x320 ResBlock stage with the overlapped decoder backward
(its fork events are recorded events under capture) and the 768-wide
transformer stage.  Each replay runs after other eager work and a
synchronisation, and every replay is checked."""

import pytest

from paper_2606_19163_amd import configs, synth

from gpu_util import log

pytestmark = pytest.mark.gpu


def _replays_match(step, outs, st, label):
    import torch
    for _ in range(2):
        step()
    torch.cuda.synchronize()

    def snap():
        torch.cuda.synchronize()
        return [t.clone() for t in outs] + [st.grads.clone()]

    st.zero_grads()
    step()
    ref = snap()
    log(f"case graph {label}: capture")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.synchronize()
    for r in range(3):
        log(f"case graph {label}: replay {r}")
        st.zero_grads()
        torch.cuda.synchronize()
        g.replay()
        x = torch.ones(1 << 20, device="cuda")
        x.mul_(2.0)
        torch.cuda.synchronize()
        cur = snap()
        for i, (a, b) in enumerate(zip(ref, cur)):
            assert torch.equal(a, b), f"{label}: replay {r} differs in output {i}"


def test_resblock_stage_step_graph_replays_bitwise():
    import torch
    from paper_2606_19163_amd import stage as S
    d = configs.l64()
    params, b = synth.make_all(d, configs.SEEDS["l64"])
    st = S.Stage(d)
    st.set_params(params)
    st.overlap_bwd(True)
    dev = {k: st.to_dev(v) for k, v in b.items()}
    outs = [st.act(d["enc"][-1]["c_out"]), st.act(d["dec"][-1]["c_out"]),
            st.act(d["enc"][0]["c_in"]), st.act(d["dec"][0]["c_up"])]
    dtemb = torch.zeros((d["batch"], d["temb_dim"]), device="cuda")
    outs.append(dtemb)

    def step():
        st.forward(S.ENC, 0, dev["x"], dev["temb"], out=outs[0])
        st.forward(S.DEC, 0, dev["u"], dev["temb"], out=outs[1])
        st.backward(S.DEC, 0, dev["g_dec"], din=outs[3], dtemb=dtemb)
        st.backward(S.ENC, 0, dev["g_enc"], din=outs[2], dtemb=dtemb)

    def step_zero_dtemb():
        dtemb.zero_()
        step()

    _replays_match(step_zero_dtemb, outs, st, "l64")


def test_transformer_stage_step_graph_replays_bitwise():
    from paper_2606_19163_amd import tstage as TS
    d = configs.get("t768")
    params, b = synth.make_tstage(d, configs.SEEDS["t768"])
    st = TS.TStage(d)
    st.set_params(params)
    dev = {k: st.to_dev(v) for k, v in b.items()}
    outs = [st.act() for _ in range(4)]

    def step():
        st.forward(TS.ENC, 0, dev["x"], out=outs[0])
        st.forward(TS.DEC, 0, dev["u"], out=outs[1])
        st.backward(TS.DEC, 0, dev["g_dec"], din=outs[3])
        st.backward(TS.ENC, 0, dev["g_enc"], din=outs[2])

    _replays_match(step, outs, st, "t768")
