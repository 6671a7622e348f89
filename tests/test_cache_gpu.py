"""Bit-exact properties of the skip cache and the microbatch bookkeeping on
the device: put/take round trips, the cached skip is the encoder output,
reruns are identical, and microbatches in flight together (the wave order:
all forwards, then backwards in reverse) give exactly what isolated runs
give."""

import numpy as np
import pytest

from paper_2606_19163_amd import configs, synth
from paper_2606_19163_amd import stage as S

from gpu_util import device_boundary, log

pytestmark = pytest.mark.gpu


def _bytes(t):
    import torch
    return t.contiguous().view(torch.uint8).cpu().numpy().tobytes()


def test_put_take_roundtrip_bitwise():
    import torch
    desc = configs.shrink(configs.l64(), batch=2, hw=8)
    st = S.Stage(desc)
    g = torch.Generator(device="cpu").manual_seed(0)
    src = torch.randint(0, 65535, (2, 8, 8, 320), generator=g, dtype=torch.int32)
    src = src.to(torch.int16).view(torch.bfloat16).cuda()
    st.put(7, 1, src)
    assert st.state(7, 1) == S.ACT_PRESENT
    out = st.take(7, 1, S.SKIP_ACT)
    torch.cuda.synchronize()
    assert _bytes(out) == _bytes(src)
    assert st.inflight() == 0


def _wave_setup(desc, seed):
    params, b = synth.make_all(desc, seed)
    st = S.Stage(desc)
    st.set_params(params)
    return st, params


def test_encoder_output_is_the_cached_skip_and_reruns_match():
    import torch
    desc = configs.shrink(configs.l64(), batch=2, hw=16)
    st, _ = _wave_setup(desc, 2)
    _, b = synth.make_all(desc, 2)
    db = device_boundary(st, b)
    y1 = st.forward(S.ENC, 0, db["x"], db["temb"])
    skip = st.take(0, 1, S.SKIP_ACT)
    torch.cuda.synchronize()
    assert _bytes(y1) == _bytes(skip)
    st.put(0, 1, skip)
    y_dec = st.forward(S.DEC, 0, db["u"], db["temb"])
    du = st.backward(S.DEC, 0, db["g_dec"])
    dx = st.backward(S.ENC, 0, db["g_enc"])
    g1 = st.grads.clone()
    st.zero_grads()
    out2 = S.run_microbatch(st, 1, db)
    torch.cuda.synchronize()
    assert _bytes(out2["y_enc"]) == _bytes(y1)
    assert _bytes(out2["y_dec"]) == _bytes(y_dec)
    assert _bytes(out2["du"]) == _bytes(du)
    assert _bytes(out2["dx"]) == _bytes(dx)
    assert _bytes(st.grads) == _bytes(g1)


@pytest.mark.parametrize("name", ["l64", "l32"])
def test_wave_order_matches_isolated_microbatches(name):
    """4 microbatches in flight: all forward passes first, then the backward
    passes in reverse order.  Per-microbatch outputs equal isolated runs
    bitwise, and the gradients accumulated over the wave equal a sequential
    replay in the same accumulation order bitwise."""
    import torch
    desc = configs.shrink(configs.get(name), batch=2, hw=8)
    desc["max_inflight"] = 4
    params, bounds = synth.make_wave([desc], configs.SEEDS["wave"], 4)
    st = S.Stage(desc)
    st.set_params(params[0])
    dbs = [device_boundary(st, bb) for bb in bounds[0]]
    log(f"case wave {name}: forward all, backward reverse")
    y = {}
    for m in range(4):
        y[("e", m)] = st.forward(S.ENC, m, dbs[m]["x"], dbs[m]["temb"])
        y[("d", m)] = st.forward(S.DEC, m, dbs[m]["u"], dbs[m]["temb"])
    assert st.inflight() == 4
    for m in reversed(range(4)):
        y[("du", m)] = st.backward(S.DEC, m, dbs[m]["g_dec"])
        y[("dx", m)] = st.backward(S.ENC, m, dbs[m]["g_enc"])
    torch.cuda.synchronize()
    wave_grads = _bytes(st.grads)
    # isolated, same accumulation order (3, 2, 1, 0)
    st.zero_grads()
    for m in reversed(range(4)):
        out = S.run_microbatch(st, 100 + m, dbs[m])
        torch.cuda.synchronize()
        assert _bytes(out["y_enc"]) == _bytes(y[("e", m)]), m
        assert _bytes(out["y_dec"]) == _bytes(y[("d", m)]), m
        assert _bytes(out["du"]) == _bytes(y[("du", m)]), m
        assert _bytes(out["dx"]) == _bytes(y[("dx", m)]), m
    assert _bytes(st.grads) == wave_grads
    assert st.inflight() == 0


def test_state_errors_enqueue_nothing():
    import torch
    desc = configs.shrink(configs.l64(), batch=1, hw=8)
    st, _ = _wave_setup(desc, 2)
    x = st.act(320)
    with pytest.raises(S.PulseError) as e:
        st.forward(S.DEC, 0, x, torch.zeros((1, 1280), dtype=torch.bfloat16, device="cuda"))
    assert e.value.status == S.E_STATE
    with pytest.raises(S.PulseError) as e:
        st.backward(S.ENC, 0, x)
    assert e.value.status == S.E_STATE
    assert st.inflight() == 0


@pytest.mark.parametrize("level", [0, 1, 2, 3])
def test_full_size_wave_order_matches_isolated_microbatches(level):
    """The wave workload's launch configuration at full size: one level of
    the four (64x64x320, 32x32x640, 16x16x1280, 8x8x1280 at batch 8) with 4
    microbatches in flight, all forward passes, then the backward passes in
    reverse.  Every per-microbatch output equals an isolated run bitwise, and
    so do the accumulated gradients.  (Isolated runs of each level at batch 8,
    in this launch configuration, are compared with the oracle by
    ``test_parity_gpu.py::test_full_size``.)"""
    import torch
    desc = configs.wave_levels()[level]
    name = ["l64", "l32", "l16", "l8"][level]
    params, bounds = synth.make_wave([desc], configs.SEEDS["wave"] + level, 4)
    st = S.Stage(desc)
    st.set_params(params[0])
    dbs = [device_boundary(st, bb) for bb in bounds[0]]
    log(f"case full-size wave level {name}: B={desc['batch']} {desc['height']}x{desc['width']}")
    y = {}
    for m in range(4):
        y[("e", m)] = st.forward(S.ENC, m, dbs[m]["x"], dbs[m]["temb"])
        y[("d", m)] = st.forward(S.DEC, m, dbs[m]["u"], dbs[m]["temb"])
    assert st.inflight() == 4
    for m in reversed(range(4)):
        y[("du", m)] = st.backward(S.DEC, m, dbs[m]["g_dec"])
        y[("dx", m)] = st.backward(S.ENC, m, dbs[m]["g_enc"])
    torch.cuda.synchronize()
    wave_grads = _bytes(st.grads)
    st.zero_grads()
    for m in reversed(range(4)):
        out = S.run_microbatch(st, 100 + m, dbs[m])
        torch.cuda.synchronize()
        for k, t in (("e", "y_enc"), ("d", "y_dec"), ("du", "du"), ("dx", "dx")):
            assert torch.equal(out[t].view(torch.int16), y[(k, m)].view(torch.int16)), (m, t)
    assert _bytes(st.grads) == wave_grads
    assert st.inflight() == 0


def test_calls_on_alternating_streams_match_one_stream():
    """Every call shares the stage's scratch buffers, so a call on a stream
    other than the previous call's waits for that call's work first: the
    four calls of a microbatch alternating between two side streams give
    bitwise what the same calls give on one stream."""
    import torch
    desc = configs.shrink(configs.l64(), batch=2, hw=16)
    st, _ = _wave_setup(desc, 2)
    _, b = synth.make_all(desc, 2)
    db = device_boundary(st, b)
    st.zero_grads()
    ref = S.run_microbatch(st, 0, db)
    torch.cuda.synchronize()
    g_ref = _bytes(st.grads)
    st.zero_grads()
    outs = {k: torch.empty_like(v) for k, v in ref.items()}
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    log("case alternating streams: F_enc s1, F_dec s2, B_dec s1, B_enc s2")
    st.forward(S.ENC, 1, db["x"], db["temb"], out=outs["y_enc"], stream=s1)
    st.forward(S.DEC, 1, db["u"], db["temb"], out=outs["y_dec"], stream=s2)
    st.backward(S.DEC, 1, db["g_dec"], din=outs["du"], stream=s1)
    st.backward(S.ENC, 1, db["g_enc"], din=outs["dx"], stream=s2)
    torch.cuda.synchronize()
    for k in ref:
        assert _bytes(outs[k]) == _bytes(ref[k]), k
    assert _bytes(st.grads) == g_ref
    assert st.inflight() == 0
