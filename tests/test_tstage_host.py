"""Host-side tests of the transformer-block stage's C ABI (no GPU):
descriptor validation, the documented parameter layout, the FLOP model and
the per-microbatch bookkeeping of dry-run stages (no device work)."""

import os

import numpy as np
import pytest

from paper_2606_19163_amd import configs
from paper_2606_19163_amd import stage as S
from paper_2606_19163_amd import tstage as TS


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_19163_amd import build
        build.build()
    yield


def _dry(desc):
    return TS.TStage(desc, dry_run=True)


@pytest.mark.parametrize("name", ["t_tiny", "t768"])
def test_param_layout_matches_config(name):
    d = configs.get(name)
    st = _dry(d)
    names = configs.tparam_names(d)
    assert list(st.layout) == [n for n, _ in names]  # documented order
    for n, shape in names:
        off, got = st.layout[n]
        assert got == shape, n
        assert off % 4 == 0
    spans = sorted((off, off + int(np.prod(s))) for off, s in st.layout.values())
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= st.n_params


def test_flops_model_t768():
    d = configs.t768()
    st = _dry(d)
    T, C, R, L = 16 * 256, 768, 3072, 256
    fwd_block = 2 * T * (3 * C * C + C * C + R * C + C * R) + 2 * 2 * T * L * C
    bwd_block = 2 * 2 * T * (3 * C * C + C * C + R * C + C * R) + 4 * 2 * T * L * C
    skip = 3 * 2 * T * 2 * C * C
    assert st.flops() == pytest.approx(4 * (fwd_block + bwd_block) + 2 * skip, rel=1e-12)


@pytest.mark.parametrize("bad", [
    dict(tokens=32), dict(tokens=4160), dict(tokens=96), dict(tokens=1000), dict(width=96),
    dict(width=2112, heads=33), dict(mlp=0), dict(mlp=9), dict(n_dec=2),
    dict(n_enc=0, n_dec=0), dict(max_inflight=0), dict(max_inflight=65), dict(eps=-1.0),
    dict(dtype=configs.F32), dict(batch=0), dict(batch=8193, tokens=128),
    dict(batch=4096, tokens=256, width=1024, heads=16, mlp=4),
])
def test_rejects_bad_descriptors(bad):
    d = configs.t_tiny()
    d.update(bad)
    with pytest.raises(S.PulseError) as e:
        _dry(d)
    assert e.value.status == S.E_SHAPE


@pytest.mark.parametrize("tokens", [320, 1024, 4096])
def test_accepts_long_sequences(tokens):
    """Token counts past 256 take the streamed attention kernels; any
    multiple of 64 up to 4096 is a valid stage."""
    d = configs.t_tiny()
    d.update(batch=1, tokens=tokens)
    st = _dry(d)
    assert st.L == tokens


def test_bookkeeping_order_and_capacity():
    d = configs.t_tiny()
    d["max_inflight"] = 2
    st = _dry(d)
    # decoder forward needs the encoder forward first
    with pytest.raises(S.PulseError) as e:
        st.forward(TS.DEC, 0, None)
    assert e.value.status == S.E_STATE
    st.forward(TS.ENC, 0, None)
    with pytest.raises(S.PulseError) as e:
        st.forward(TS.ENC, 0, None)  # twice
    assert e.value.status == S.E_STATE
    st.forward(TS.ENC, 1, None)
    with pytest.raises(S.PulseError) as e:
        st.forward(TS.ENC, 2, None)
    assert e.value.status == S.E_CACHE_FULL
    assert st.inflight() == 2
    # encoder backward before the decoder backward is out of order
    st.forward(TS.DEC, 0, None)
    with pytest.raises(S.PulseError) as e:
        st.backward(TS.ENC, 0, None)
    assert e.value.status == S.E_STATE
    with pytest.raises(S.PulseError) as e:
        st.backward(TS.DEC, 1, None)  # mb 1 has no decoder forward
    assert e.value.status == S.E_STATE
    st.backward(TS.DEC, 0, None)
    st.backward(TS.ENC, 0, None)
    assert st.inflight() == 1
    st.forward(TS.ENC, 7, None)  # the released row is reused
    assert st.inflight() == 2
    st.release(1)
    assert st.inflight() == 1
    st.reset()
    assert st.inflight() == 0


def test_dry_stage_binds_nothing():
    st = _dry(configs.t_tiny())
    assert st.ws_bytes == 0


def test_skip_grad_exists_only_between_the_two_backward_halves():
    import ctypes
    d = configs.t_tiny()
    st = _dry(d)
    L = TS.lib()

    def probe(mb, slot):
        return L.pulse_tstage_skip_grad(st.h, mb, slot, None, None)

    st.forward(TS.ENC, 4, None)
    st.forward(TS.DEC, 4, None)
    assert probe(4, 0) == S.E_CACHE_MISS       # before the decoder backward
    st.backward(TS.DEC, 4, None)
    assert probe(4, 0) == S.OK                 # buffered (dry run: no copy)
    assert probe(4, 1) == S.E_INVALID_ARG      # slot out of range (one encoder block)
    assert probe(5, 0) == S.E_CACHE_MISS       # unknown microbatch
    st.backward(TS.ENC, 4, None)
    assert probe(4, 0) == S.E_CACHE_MISS       # consumed by the encoder backward


def test_schedule_rows_drive_a_dry_transformer_stage():
    """Every device row of the collocated wave schedule runs through
    pulse_tsched_run_device in dry-run mode: the state machine accepts the
    schedule's order and every microbatch is released at the end; a cell of
    another device is rejected before anything runs."""
    from paper_2606_19163_amd import stage as S2
    for D, M in [(1, 3), (2, 3), (3, 4)]:
        table, _ = S2.sched_build(D, M)
        need = S2.sched_inflight(D, M, table)
        for d in range(D):
            desc = configs.t_tiny()
            desc["max_inflight"] = max(need)
            st = _dry(desc)
            TS.tsched_run_device(st, D, d, M, table)
            assert st.inflight() == 0
    table, _ = S2.sched_build(2, 2)
    st = _dry(configs.t_tiny())
    with pytest.raises(S.PulseError) as e:
        TS.tsched_run_device(st, 2, 0, 2, [table[1], table[1]])  # device 1's cells as row 0
    assert e.value.status == S.E_INVALID_ARG
    assert st.inflight() == 0


@pytest.mark.parametrize("batch,ok", [(1023, True), (1024, False)])
def test_activation_bytes_limit(batch, ok):
    """Width 2048 with an 8x MLP: the fc1 output holds 16384 bf16 values per
    token, so 65536 tokens reach 2^31 bytes exactly and are refused, while
    64 tokens fewer are accepted."""
    d = configs.t_tiny()
    d.update(batch=batch, tokens=64, width=2048, heads=32, mlp=8)
    if ok:
        _dry(d)
    else:
        with pytest.raises(S.PulseError) as e:
            _dry(d)
        assert e.value.status == S.E_SHAPE


@pytest.mark.parametrize("batch,ok", [(16384, True), (16385, False)])
def test_token_count_limit(batch, ok):
    """The GEMM kernels form token offsets as 24-bit products; the stage
    caps batch x tokens at 2^20."""
    d = configs.t_tiny()
    d.update(batch=batch, tokens=64)
    if ok:
        _dry(d)
    else:
        with pytest.raises(S.PulseError) as e:
            _dry(d)
        assert e.value.status == S.E_SHAPE
