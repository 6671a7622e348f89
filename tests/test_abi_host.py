"""Host-side tests of the C-ABI library (no GPU): it loads, exports every
function the header declares, validates descriptors, lays out parameters as
documented, and runs the skip-cache / microbatch bookkeeping exactly (dry-run
stages enqueue no device work)."""

import ctypes
import os

import pytest

from paper_2606_19163_amd import configs
from paper_2606_19163_amd import stage as S


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_19163_amd import build
        build.build()
    yield


def test_exports_every_header_function():
    names = S.header_functions()
    assert "pulse_stage_create" in names and "pulse_skip_cache_take" in names
    L = ctypes.CDLL(S.LIB_PATH)
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing


def _dry(desc):
    return S.Stage(desc, dry_run=True)


@pytest.mark.parametrize("name", ["tiny", "l64", "l32", "l16", "l8"])
def test_param_layout_matches_config(name):
    d = configs.get(name)
    st = _dry(d)
    expect = dict(configs.param_names(d))
    assert set(st.layout) == set(expect)
    for n, (off, shape) in st.layout.items():
        assert shape == expect[n], n
        assert off % 64 == 0
    # tensors do not overlap
    spans = sorted((off, off + int(__import__("numpy").prod(s))) for off, s in st.layout.values())
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= st.n_params


def test_flops_model_l64():
    st = _dry(configs.l64())
    # 2 encoder blocks 320->320 and 2 decoder blocks 640->320 at 8x64x64
    P = 8 * 64 * 64
    enc = 2 * P * 320 * 9 * 320 * 2 + 2 * 8 * 320 * 1280
    dec = 2 * P * 320 * 9 * 640 + 2 * P * 320 * 9 * 320 + 2 * P * 320 * 640 + 2 * 8 * 320 * 1280
    assert st.flops() == pytest.approx(3 * (2 * enc + 2 * dec), rel=1e-12)
    assert st.flops() == pytest.approx(1892.5e9, rel=1e-3)


def _expect_status(fn, status):
    with pytest.raises(S.PulseError) as e:
        fn()
    assert e.value.status == status, str(e.value)


def test_descriptor_validation():
    d = configs.l64()
    for mutate, status in [
        (lambda x: x.update(groups=7), S.E_SHAPE),
        (lambda x: x["enc"][1].update(c_in=640), S.E_SHAPE),
        (lambda x: x["dec"][0].update(skip_slot_in=5), S.E_SHAPE),
        (lambda x: x["dec"][1].update(skip_slot_in=1), S.E_SHAPE),  # slot read twice
        (lambda x: x["enc"][1].update(skip_slot_out=0), S.E_SHAPE),  # two producers
        (lambda x: x["dec"][0].update(c_skip=640), S.E_SHAPE),
        (lambda x: x.update(max_inflight=0), S.E_SHAPE),
        (lambda x: x["enc"][0].update(c_in=48), S.E_SHAPE),
    ]:
        dd = configs.get("l64")
        mutate(dd)
        _expect_status(lambda: _dry(dd), status)
    _dry(d)  # the unmodified descriptor is fine


def test_not_bound_errors_without_workspace():
    # a real (non dry-run) stage refuses to run before bind/sync; create and
    # validation need no GPU
    d = configs.tiny()
    cdesc, keep = S.make_desc(d)
    h = ctypes.c_void_p()
    L = S.lib()
    assert L.pulse_stage_create(ctypes.byref(cdesc), ctypes.byref(h)) == S.OK
    buf = ctypes.create_string_buffer(64)
    st = L.pulse_stage_forward(h, S.ENC, 0, ctypes.addressof(buf), ctypes.addressof(buf),
                               ctypes.addressof(buf), None)
    assert st == S.E_NOT_BOUND
    assert b"bound" in L.pulse_last_error()
    assert L.pulse_stage_inflight(h) == 0
    L.pulse_stage_destroy(h)


def test_microbatch_order_and_release():
    st = _dry(configs.l64())
    _expect_status(lambda: st.forward(S.DEC, 0, None, None), S.E_STATE)
    _expect_status(lambda: st.backward(S.DEC, 0, None), S.E_STATE)
    st.forward(S.ENC, 0, None, None)
    assert st.state(0, 0) == S.ACT_PRESENT and st.state(0, 1) == S.ACT_PRESENT
    _expect_status(lambda: st.forward(S.ENC, 0, None, None), S.E_STATE)
    _expect_status(lambda: st.backward(S.ENC, 0, None), S.E_STATE)
    _expect_status(lambda: st.backward(S.DEC, 0, None), S.E_STATE)
    st.forward(S.DEC, 0, None, None)
    _expect_status(lambda: st.forward(S.DEC, 0, None, None), S.E_STATE)
    _expect_status(lambda: st.backward(S.ENC, 0, None), S.E_STATE)
    st.backward(S.DEC, 0, None)
    assert st.state(0, 0) == S.ACT_PRESENT | S.GRAD_PRESENT
    st.backward(S.ENC, 0, None)
    assert st.inflight() == 0
    assert st.state(0, 0) == 0


def test_overlapped_backward_bookkeeping_matches_joined():
    """pulse_stage_overlap_bwd and pulse_stage_flush change no bookkeeping:
    a dry-run stage walks the same states with the switch on, and a flush
    is accepted at any point (it only orders work)."""
    st = _dry(configs.l64())
    st.overlap_bwd(True)
    st.flush()
    st.forward(S.ENC, 0, None, None)
    st.forward(S.DEC, 0, None, None)
    st.backward(S.DEC, 0, None)
    st.flush()
    assert st.state(0, 0) == S.ACT_PRESENT | S.GRAD_PRESENT
    st.backward(S.ENC, 0, None)
    assert st.inflight() == 0
    st.overlap_bwd(False)
    _expect_status(lambda: S._check(S.lib().pulse_stage_overlap_bwd(None, 1)), S.E_INVALID_ARG)
    _expect_status(lambda: S._check(S.lib().pulse_stage_flush(None, None)), S.E_INVALID_ARG)


def test_capacity_and_wave_order():
    d = configs.l64()
    d["max_inflight"] = 4
    st = _dry(d)
    for m in range(4):
        st.forward(S.ENC, m, None, None)
        st.forward(S.DEC, m, None, None)
    assert st.inflight() == 4
    _expect_status(lambda: st.forward(S.ENC, 9, None, None), S.E_CACHE_FULL)
    _expect_status(lambda: st.put(9, 0, None), S.E_CACHE_FULL)
    for m in reversed(range(4)):
        st.backward(S.DEC, m, None)
        st.backward(S.ENC, m, None)
    assert st.inflight() == 0
    st.forward(S.ENC, 9, None, None)  # rows are reusable
    assert st.inflight() == 1
    st.reset()
    assert st.inflight() == 0


def test_put_take_bookkeeping():
    st = _dry(configs.l64())
    # partial collocation: the skips come from elsewhere, no local encoder
    st.put(3, 0, None)
    _expect_status(lambda: st.put(3, 0, None), S.E_CACHE_OCCUPIED)
    _expect_status(lambda: st.forward(S.DEC, 3, None, None), S.E_CACHE_MISS)
    st.put(3, 1, None)
    st.forward(S.DEC, 3, None, None)
    st.backward(S.DEC, 3, None)
    _expect_status(lambda: st.backward(S.ENC, 3, None), S.E_STATE)
    for slot in (0, 1):
        st.take(3, slot, S.SKIP_GRAD)
        _expect_status(lambda: st.take(3, slot, S.SKIP_GRAD), S.E_CACHE_MISS)
    assert st.inflight() == 1
    st.take(3, 0, S.SKIP_ACT)
    st.take(3, 1, S.SKIP_ACT)
    assert st.inflight() == 0  # released with its last entry
    # a missing skip gradient blocks the encoder backward
    st.forward(S.ENC, 4, None, None)
    st.forward(S.DEC, 4, None, None)
    st.backward(S.DEC, 4, None)
    st.take(4, 1, S.SKIP_GRAD)
    _expect_status(lambda: st.backward(S.ENC, 4, None), S.E_CACHE_MISS)
    st.release(4)
    assert st.inflight() == 0
    _expect_status(lambda: st.take(4, 0, S.SKIP_ACT), S.E_CACHE_MISS)
    _expect_status(lambda: st.put(0, 7, None), S.E_INVALID_ARG)


def test_encoder_forward_refuses_occupied_slot():
    st = _dry(configs.l64())
    st.put(5, 1, None)
    _expect_status(lambda: st.forward(S.ENC, 5, None, None), S.E_CACHE_OCCUPIED)
    st.take(5, 1, S.SKIP_ACT)
    st.forward(S.ENC, 5, None, None)


def test_input_slot_bookkeeping_l32():
    st = _dry(configs.l32())
    st.forward(S.ENC, 0, None, None)
    assert st.state(0, 1) == S.ACT_PRESENT   # the stage input
    assert st.state(0, 0) == S.ACT_PRESENT   # the second block's output
    st.forward(S.DEC, 0, None, None)
    st.backward(S.DEC, 0, None)
    assert st.state(0, 1) & S.GRAD_PRESENT
    st.backward(S.ENC, 0, None)
    assert st.inflight() == 0


def test_pixel_count_limit():
    """The conv kernels form pixel offsets as 24-bit products: a stage of
    2^24 pixels is refused at create, with the pixel count named.  (The
    decoder's input gradient has at least 64 channels, so the 2 GiB tensor
    limit below already binds from 2^23 pixels on.)"""
    d = configs.shrink(configs.tiny(), batch=1, hw=4096, width=4096)
    with pytest.raises(S.PulseError) as e:
        _dry(d)
    assert e.value.status == S.E_SHAPE and "2^24" in str(e.value)


@pytest.mark.parametrize("width,ok", [(4095, True), (4096, False)])
def test_tensor_bytes_limit(width, ok):
    """Operands are addressed through buffer ranges of at most 2^31 - 1
    bytes: the widest [pixels][C] tensor, counted at 4 bytes per value (the
    fp32 skip gradients and partial sums), must stay below 2 GiB.  The tiny
    stage's widest tensor is the decoder's 64-channel input gradient, so
    2048 x 4096 pixels reach 2^31 bytes exactly."""
    d = configs.shrink(configs.tiny(), batch=1, hw=2048, width=width)
    if ok:
        _dry(d)
    else:
        _expect_status(lambda: _dry(d), S.E_SHAPE)


@pytest.mark.parametrize("dtype,ok", [(configs.BF16, True), (configs.F32, False)])
def test_weight_bytes_limit(dtype, ok):
    """A decoder conv2 copy with its shortcut appended, [8160][9*8160 + 8192],
    is 1.33 GB in bf16 and 2.66 GB in fp32: the fp32 stage is refused."""
    d = configs.tiny()
    d["dtype"] = dtype
    d["dec"][0].update(c_up=8160, c_out=8160)
    if ok:
        _dry(d)
    else:
        _expect_status(lambda: _dry(d), S.E_SHAPE)


def test_forward_static_scratch_limit():
    """The static-scratch forward takes stages whose forward scratch fits the
    library's array (the 64x64x320 stage at batch 8) and refuses larger ones
    (16x16x1280 at batch 16) before doing anything."""
    st = _dry(configs.l64())
    st.forward_static(S.ENC, 0, None, None)
    st.forward_static(S.DEC, 0, None, None)
    big = _dry(configs.l16())
    _expect_status(lambda: big.forward_static(S.ENC, 0, None, None), S.E_SHAPE)
    assert big.inflight() == 0
