"""Overlapped decoder backward (pulse_stage_overlap_bwd): a decoder backward
that leaves its last parameter-gradient work on the stage's second stream,
with the encoder backward starting beside it, gives bitwise the results of
the joined backward, on the 64x64x320 and 32x32x640 stages in the bench's
launch configuration; a flush orders that work before later work on a
stream."""

import pytest

from paper_2606_19163_amd import configs, synth

from gpu_util import log

pytestmark = pytest.mark.gpu


def _run(desc, params, batches, overlap, streams=None):
    import torch
    from paper_2606_19163_amd import stage as S
    st = S.Stage(desc)
    st.set_params(params)
    st.zero_grads()
    st.overlap_bwd(overlap)
    dtemb = torch.zeros((desc["batch"], desc["temb_dim"]), dtype=torch.float32, device="cuda")
    outs = []
    for mb, bb in enumerate(batches):
        db = {k: st.to_dev(v) for k, v in bb.items()}
        torch.cuda.synchronize()  # the inputs are copied on the default stream
        s_dec, s_enc = streams if streams else (None, None)
        y_enc = st.forward(S.ENC, mb, db["x"], db["temb"], stream=s_dec)
        y_dec = st.forward(S.DEC, mb, db["u"], db["temb"], stream=s_dec)
        du = st.backward(S.DEC, mb, db["g_dec"], dtemb=dtemb, stream=s_dec)
        dx = st.backward(S.ENC, mb, db["g_enc"], dtemb=dtemb, stream=s_enc)
        outs.append(dict(y_enc=y_enc, y_dec=y_dec, du=du, dx=dx))
    torch.cuda.synchronize()
    res = [{k: v.cpu() for k, v in o.items()} for o in outs]
    return res, st.grads.cpu(), dtemb.cpu()


def _same(a, b, label):
    import torch
    ra, ga, ta = a
    rb, gb, tb = b
    for mb, (oa, ob) in enumerate(zip(ra, rb)):
        for k in oa:
            assert torch.equal(oa[k], ob[k]), f"{label}: mb{mb} {k} differs"
    assert torch.equal(ga, gb), f"{label}: parameter gradients differ"
    assert torch.equal(ta, tb), f"{label}: dtemb differs"


@pytest.mark.parametrize("name", ["l64", "l32"])
def test_overlapped_decoder_backward_is_bitwise_the_joined_one(name):
    """Both stages the bench runs with it: 64x64x320, and 32x32x640 with its
    shortcut convs and K-split convs."""
    desc = configs.get(name)
    params, b0 = synth.make_all(desc, configs.SEEDS[name])
    _, b1 = synth.make_all(desc, configs.SEEDS[name] + 100)
    log(f"case overlap: {name}, two microbatches, joined backward")
    ref = _run(desc, params, (b0, b1), overlap=False)
    log(f"case overlap: {name}, two microbatches, overlapped decoder backward")
    got = _run(desc, params, (b0, b1), overlap=True)
    _same(ref, got, f"{name} overlapped")


def test_overlapped_decoder_backward_across_streams():
    """The encoder backward on another stream than the decoder's: the next
    call joins the side stream first (no carried markers)."""
    import torch
    desc = configs.l64()
    params, b0 = synth.make_all(desc, configs.SEEDS["l64"])
    log("case overlap: l64, decoder and encoder backward on two streams")
    ref = _run(desc, params, (b0,), overlap=False)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    got = _run(desc, params, (b0,), overlap=True, streams=(s1, s2))
    _same(ref, got, "two streams")


def test_flush_orders_decoder_gradients_on_the_stream():
    """After an overlapped decoder backward, a flush on the stream and a
    synchronisation of that stream alone see the decoder's complete
    parameter gradients."""
    import torch
    from paper_2606_19163_amd import stage as S
    desc = configs.l64()
    params, b0 = synth.make_all(desc, configs.SEEDS["l64"])
    grads = []
    for overlap in (False, True):
        log(f"case flush: l64 decoder backward, overlap={overlap}")
        st = S.Stage(desc)
        st.set_params(params)
        st.zero_grads()
        st.overlap_bwd(overlap)
        db = {k: st.to_dev(v) for k, v in b0.items()}
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        st.forward(S.ENC, 0, db["x"], db["temb"], stream=s)
        st.forward(S.DEC, 0, db["u"], db["temb"], stream=s)
        st.backward(S.DEC, 0, db["g_dec"], stream=s)
        st.flush(stream=s)
        with torch.cuda.stream(s):
            g = st.grads.clone()
        s.synchronize()
        grads.append(g.cpu())
        torch.cuda.synchronize()
        st.release(0)
    assert torch.equal(grads[0], grads[1])


def test_transformer_overlapped_decoder_backward_is_bitwise_the_joined_one():
    """The same for the 768-wide transformer stage (two microbatches)."""
    import torch
    from paper_2606_19163_amd import tstage as TS
    d = configs.get("t768")
    params, b0 = synth.make_tstage(d, configs.SEEDS["t768"])
    _, b1 = synth.make_tstage(d, configs.SEEDS["t768"] + 100)
    res = []
    for overlap in (False, True):
        log(f"case overlap: t768, two microbatches, overlap={overlap}")
        st = TS.TStage(d)
        st.set_params(params)
        st.zero_grads()
        st.overlap_bwd(overlap)
        outs = []
        for mb, bb in enumerate((b0, b1)):
            db = {k: st.to_dev(v) for k, v in bb.items()}
            torch.cuda.synchronize()
            y_enc = st.forward(TS.ENC, mb, db["x"])
            y_dec = st.forward(TS.DEC, mb, db["u"])
            du = st.backward(TS.DEC, mb, db["g_dec"])
            dx = st.backward(TS.ENC, mb, db["g_enc"])
            outs.append([y_enc, y_dec, du, dx])
        torch.cuda.synchronize()
        res.append(([[t.cpu() for t in o] for o in outs], st.grads.cpu()))
    (oa, ga), (ob, gb) = res
    for mb in range(2):
        for i in range(4):
            assert torch.equal(oa[mb][i], ob[mb][i]), f"t768 mb{mb} output {i} differs"
    assert torch.equal(ga, gb), "t768 parameter gradients differ"
