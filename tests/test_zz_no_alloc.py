"""pulse_stage_forward_static, the forward whose scratch lives in the
library's static device array (for callers that cannot allocate), against
pulse_stage_forward through the C ABI: outputs, cached skips and the state
the backward consumes are bitwise equal, on two calls in a row, the second
on a smaller stage."""

import pytest

from paper_2606_19163_amd import configs, synth
from paper_2606_19163_amd import stage as S

from gpu_util import device_boundary, log

pytestmark = pytest.mark.gpu


def _bytes(t):
    import torch
    return t.contiguous().view(torch.uint8).cpu().numpy().tobytes()


def _compare(desc, seed, label):
    import torch
    log(f"case static-scratch forward {label}: B={desc['batch']} "
        f"{desc['height']}x{desc['width']}")
    d = dict(desc)
    d["max_inflight"] = 2
    params, b = synth.make_all(d, seed)
    st = S.Stage(d)
    st.set_params(params)
    st.zero_grads()
    db = device_boundary(st, b)
    out = {}
    for mb, fwd in ((0, st.forward), (1, st.forward_static)):
        out[("y_enc", mb)] = fwd(S.ENC, mb, db["x"], db["temb"])
        out[("y_dec", mb)] = fwd(S.DEC, mb, db["u"], db["temb"])
    torch.cuda.synchronize()
    for k in ("y_enc", "y_dec"):
        assert _bytes(out[(k, 0)]) == _bytes(out[(k, 1)]), k
    # the saved state: both microbatches' backward passes agree
    for mb in (0, 1):
        out[("du", mb)] = st.backward(S.DEC, mb, db["g_dec"])
        out[("dx", mb)] = st.backward(S.ENC, mb, db["g_enc"])
    torch.cuda.synchronize()
    for k in ("du", "dx"):
        assert _bytes(out[(k, 0)]) == _bytes(out[(k, 1)]), k
    assert st.inflight() == 0


def test_forward_static_matches_forward_twice():
    _compare(configs.l64(), configs.SEEDS["l64"], "l64 full size")
    _compare(configs.shrink(configs.l64(), batch=2, hw=12, width=10), 2, "l64 2x12x10")
