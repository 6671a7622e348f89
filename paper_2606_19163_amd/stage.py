"""ctypes binding of ``libpulse_stage.so`` (see ``include/pulse_stage.h``).

Argument marshalling only: every step of the stage runs in the library's HIP
kernels.  torch supplies device memory (``data_ptr()``) and the stream
(``torch.cuda.current_stream().cuda_stream``).  Loading fails loudly when the
library has not been built; there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
import re

import numpy as np

from . import configs as _cfg

# PULSE_STAGE_LIB selects another build of the same library (the host
# sanitizer build of the tests); it must exist like the default one
LIB_PATH = os.environ.get("PULSE_STAGE_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libpulse_stage.so")
HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "pulse_stage.h")

OK, E_INVALID_ARG, E_SHAPE, E_STATE, E_CACHE_FULL, E_CACHE_MISS, E_CACHE_OCCUPIED, \
    E_NOT_BOUND, E_HIP = range(9)
STATUS_NAMES = ["OK", "INVALID_ARG", "SHAPE", "STATE", "CACHE_FULL", "CACHE_MISS",
                "CACHE_OCCUPIED", "NOT_BOUND", "HIP"]
F32, BF16 = 0, 1
ENC, DEC = 0, 1
SKIP_ACT, SKIP_GRAD = 0, 1
ACT_PRESENT, GRAD_PRESENT = 1, 2
FLAG_DRY_RUN = 1

_i32 = ctypes.c_int32
_vp = ctypes.c_void_p


class EncBlock(ctypes.Structure):
    _fields_ = [("c_in", _i32), ("c_out", _i32), ("skip_slot_out", _i32)]


class DecBlock(ctypes.Structure):
    _fields_ = [("c_up", _i32), ("c_skip", _i32), ("c_out", _i32), ("skip_slot_in", _i32)]


class StageDesc(ctypes.Structure):
    _fields_ = [("batch", _i32), ("height", _i32), ("width", _i32), ("groups", _i32),
                ("eps", ctypes.c_float), ("temb_dim", _i32), ("dtype", ctypes.c_int),
                ("n_enc", _i32), ("enc", ctypes.POINTER(EncBlock)),
                ("n_dec", _i32), ("dec", ctypes.POINTER(DecBlock)),
                ("input_skip_slot", _i32), ("max_inflight", _i32), ("flags", ctypes.c_uint32)]


class PulseError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES[status] if 0 <= status < 9 else status}: {msg}")
        self.status = status


_lib = None


def header_functions():
    """Names of the functions declared in the headers under include/."""
    import glob
    names = set()
    for h in sorted(glob.glob(os.path.join(os.path.dirname(HEADER), "*.h"))):
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(pulse_\w+)\s*\(", src))
    return sorted(names)


def lib():
    """The loaded library (torch is imported first so that the library binds
    to the HIP runtime torch already loaded)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2606_19163_amd.build`")
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        st = ctypes.c_int
        L.pulse_stage_create.argtypes = [ctypes.POINTER(StageDesc), ctypes.POINTER(_vp)]
        L.pulse_stage_create.restype = st
        L.pulse_stage_destroy.argtypes = [_vp]
        L.pulse_stage_destroy.restype = None
        L.pulse_stage_sizes.argtypes = [_vp, ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_size_t)]
        L.pulse_stage_sizes.restype = st
        L.pulse_stage_param_layout.argtypes = [_vp, _i32, ctypes.c_char_p,
                                               ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(_i32)]
        L.pulse_stage_param_layout.restype = st
        L.pulse_stage_bind.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_size_t]
        L.pulse_stage_bind.restype = st
        L.pulse_stage_sync_params.argtypes = [_vp, _vp]
        L.pulse_stage_sync_params.restype = st
        L.pulse_stage_forward.argtypes = [_vp, ctypes.c_int, _i32, _vp, _vp, _vp, _vp]
        L.pulse_stage_forward.restype = st
        L.pulse_stage_forward_static.argtypes = [_vp, ctypes.c_int, _i32, _vp, _vp, _vp, _vp]
        L.pulse_stage_forward_static.restype = st
        L.pulse_stage_backward.argtypes = [_vp, ctypes.c_int, _i32, _vp, _vp, _vp, _vp]
        L.pulse_stage_backward.restype = st
        L.pulse_skip_cache_put.argtypes = [_vp, _i32, _i32, _vp, _vp]
        L.pulse_skip_cache_put.restype = st
        L.pulse_skip_cache_take.argtypes = [_vp, _i32, _i32, ctypes.c_int, _vp, _vp]
        L.pulse_skip_cache_take.restype = st
        L.pulse_skip_cache_state.argtypes = [_vp, _i32, _i32, ctypes.POINTER(_i32)]
        L.pulse_skip_cache_state.restype = st
        L.pulse_stage_release.argtypes = [_vp, _i32]
        L.pulse_stage_release.restype = st
        L.pulse_stage_reset.argtypes = [_vp]
        L.pulse_stage_reset.restype = st
        L.pulse_stage_inflight.argtypes = [_vp]
        L.pulse_stage_inflight.restype = _i32
        L.pulse_stage_timing.argtypes = [_vp, _i32]
        L.pulse_stage_timing.restype = st
        L.pulse_stage_overlap_bwd.argtypes = [_vp, _i32]
        L.pulse_stage_overlap_bwd.restype = st
        L.pulse_stage_flush.argtypes = [_vp, _vp]
        L.pulse_stage_flush.restype = st
        L.pulse_stage_timing_read.argtypes = [_vp, ctypes.POINTER(ctypes.c_int64),
                                              ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_double)]
        L.pulse_stage_timing_read.restype = st
        L.pulse_stage_flops.argtypes = [_vp]
        L.pulse_stage_flops.restype = ctypes.c_double
        _ip = ctypes.POINTER(_i32)
        L.pulse_sched_build.argtypes = [_i32, _i32, _ip, _i32, _ip, _ip]
        L.pulse_sched_build.restype = st
        L.pulse_sched_check.argtypes = [_i32, _i32, _ip, _i32, _ip]
        L.pulse_sched_check.restype = st
        L.pulse_sched_inflight.argtypes = [_i32, _i32, _ip, _i32, _ip]
        L.pulse_sched_inflight.restype = st
        L.pulse_sched_run_device.argtypes = [_vp, _i32, _i32, _i32, _ip, _i32, _i32, _i32,
                                             ctypes.POINTER(MbIO), _vp]
        L.pulse_sched_run_device.restype = st
        L.pulse_mfma_probe.argtypes = [_i32, _i32, _i32, _vp, ctypes.POINTER(ctypes.c_double),
                                       _vp]
        L.pulse_mfma_probe.restype = st
        L.pulse_last_error.argtypes = []
        L.pulse_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status):
    if status != OK:
        raise PulseError(status, lib().pulse_last_error().decode())


def make_desc(desc, dry_run=False):
    """ctypes descriptor (and the arrays it points to) from a config dict."""
    enc = (EncBlock * len(desc["enc"]))(*[EncBlock(b["c_in"], b["c_out"], b["skip_slot_out"])
                                          for b in desc["enc"]])
    dec = (DecBlock * len(desc["dec"]))(*[DecBlock(b["c_up"], b["c_skip"], b["c_out"],
                                                   b["skip_slot_in"]) for b in desc["dec"]])
    d = StageDesc(batch=desc["batch"], height=desc["height"], width=desc["width"],
                  groups=desc["groups"], eps=desc["eps"], temb_dim=desc["temb_dim"],
                  dtype=BF16 if desc["dtype"] == _cfg.BF16 else F32,
                  n_enc=len(desc["enc"]), enc=enc, n_dec=len(desc["dec"]), dec=dec,
                  input_skip_slot=desc.get("input_skip_slot", -1),
                  max_inflight=desc.get("max_inflight", 1),
                  flags=FLAG_DRY_RUN if dry_run else 0)
    return d, (enc, dec)


def _stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class Stage:
    """One collocated stage.  ``desc`` is a config dict (see
    :mod:`paper_2606_19163_amd.configs`).  With ``dry_run`` only the
    bookkeeping runs (no device memory, no kernels)."""

    def __init__(self, desc, device="cuda", dry_run=False):
        self.desc = desc
        self.dry = dry_run
        self.h = _vp()
        cdesc, self._keep = make_desc(desc, dry_run)
        _check(lib().pulse_stage_create(ctypes.byref(cdesc), ctypes.byref(self.h)))
        n = ctypes.c_int64()
        ws = ctypes.c_size_t()
        _check(lib().pulse_stage_sizes(self.h, ctypes.byref(n), ctypes.byref(ws)))
        self.n_params = n.value
        self.ws_bytes = ws.value
        self.layout = self._read_layout()
        self.B, self.H, self.W = desc["batch"], desc["height"], desc["width"]
        self.slot_ch = _cfg.slot_channels(desc)
        self.params = self.grads = self.workspace = None
        if not dry_run:
            import torch
            self.torch_dtype = torch.bfloat16 if desc["dtype"] == _cfg.BF16 else torch.float32
            self.params = torch.zeros(self.n_params, dtype=torch.float32, device=device)
            self.grads = torch.zeros(self.n_params, dtype=torch.float32, device=device)
            self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
            _check(lib().pulse_stage_bind(self.h, _ptr(self.params), _ptr(self.grads),
                                          _ptr(self.workspace), self.ws_bytes))

    def __del__(self):
        try:
            if self.h:
                lib().pulse_stage_destroy(self.h)
                self.h = _vp()
        except Exception:
            pass

    # -- parameters -------------------------------------------------------
    def _read_layout(self):
        cnt = ctypes.c_int64()
        _check(lib().pulse_stage_param_layout(self.h, -1, None, ctypes.byref(cnt), None))
        out = {}
        for i in range(cnt.value):
            name = ctypes.create_string_buffer(64)
            off = ctypes.c_int64()
            shape = (_i32 * 4)()
            _check(lib().pulse_stage_param_layout(self.h, i, name, ctypes.byref(off), shape))
            out[name.value.decode()] = (off.value, tuple(s for s in shape if s > 0))
        return out

    def set_params(self, params, stream=None):
        """Upload fp32 master parameters (dict name -> array) and refresh the
        library's compute copies."""
        import torch
        flat = np.zeros(self.n_params, dtype=np.float32)
        for name, (off, shape) in self.layout.items():
            a = np.asarray(params[name], dtype=np.float32)
            assert a.shape == shape, (name, a.shape, shape)
            flat[off:off + a.size] = a.ravel()
        self.params.copy_(torch.from_numpy(flat))
        self.sync_params(stream)

    def sync_params(self, stream=None):
        _check(lib().pulse_stage_sync_params(self.h, None if self.dry else _stream_handle(stream)))

    def zero_grads(self):
        self.grads.zero_()

    def grads_dict(self):
        g = self.grads.cpu().numpy()
        return {n: g[o:o + int(np.prod(s))].reshape(s).copy() for n, (o, s) in self.layout.items()}

    # -- tensors ----------------------------------------------------------
    def act(self, C, device="cuda"):
        import torch
        return torch.empty((self.B, self.H, self.W, C), dtype=self.torch_dtype, device=device)

    def to_dev(self, a, device="cuda"):
        import torch
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(
            device=device, dtype=self.torch_dtype)

    # -- calls --------------------------------------------------------------
    def forward(self, half, mb, inp, temb, out=None, stream=None):
        if self.dry:
            _check(lib().pulse_stage_forward(self.h, half, mb, None, None, None, None))
            return None
        if out is None:
            C = self.desc["enc"][-1]["c_out"] if half == ENC else self.desc["dec"][-1]["c_out"]
            out = self.act(C)
        _check(lib().pulse_stage_forward(self.h, half, mb, _ptr(inp), _ptr(temb), _ptr(out),
                                         _stream_handle(stream)))
        return out

    def forward_static(self, half, mb, inp, temb, out=None, stream=None):
        """pulse_stage_forward_static: the forward with its scratch in the
        library's static device array (no allocation of any kind)."""
        if self.dry:
            _check(lib().pulse_stage_forward_static(self.h, half, mb, None, None, None, None))
            return None
        if out is None:
            C = self.desc["enc"][-1]["c_out"] if half == ENC else self.desc["dec"][-1]["c_out"]
            out = self.act(C)
        _check(lib().pulse_stage_forward_static(self.h, half, mb, _ptr(inp), _ptr(temb),
                                                _ptr(out), _stream_handle(stream)))
        return out

    def backward(self, half, mb, dout, din=None, dtemb=None, stream=None):
        if self.dry:
            _check(lib().pulse_stage_backward(self.h, half, mb, None, None, None, None))
            return None
        if din is None:
            C = self.desc["enc"][0]["c_in"] if half == ENC else self.desc["dec"][0]["c_up"]
            din = self.act(C)
        _check(lib().pulse_stage_backward(self.h, half, mb, _ptr(dout), _ptr(din), _ptr(dtemb),
                                          _stream_handle(stream)))
        return din

    def put(self, mb, slot, src, stream=None):
        _check(lib().pulse_skip_cache_put(self.h, mb, slot, None if self.dry else _ptr(src),
                                          None if self.dry else _stream_handle(stream)))

    def take(self, mb, slot, kind, dst=None, stream=None):
        if self.dry:
            _check(lib().pulse_skip_cache_take(self.h, mb, slot, kind, None, None))
            return None
        import torch
        if dst is None:
            dt = self.torch_dtype if kind == SKIP_ACT else torch.float32
            dst = torch.empty((self.B, self.H, self.W, self.slot_ch[slot]), dtype=dt,
                              device="cuda")
        _check(lib().pulse_skip_cache_take(self.h, mb, slot, kind, _ptr(dst),
                                           _stream_handle(stream)))
        return dst

    def state(self, mb, slot):
        s = _i32()
        _check(lib().pulse_skip_cache_state(self.h, mb, slot, ctypes.byref(s)))
        return s.value

    def release(self, mb):
        _check(lib().pulse_stage_release(self.h, mb))

    def reset(self):
        _check(lib().pulse_stage_reset(self.h))

    def inflight(self):
        return lib().pulse_stage_inflight(self.h)

    def flops(self):
        return lib().pulse_stage_flops(self.h)

    def overlap_bwd(self, enable):
        _check(lib().pulse_stage_overlap_bwd(self.h, 1 if enable else 0))

    def flush(self, stream=None):
        _check(lib().pulse_stage_flush(self.h, None if self.dry else _stream_handle(stream)))

    def timing(self, enable):
        _check(lib().pulse_stage_timing(self.h, 1 if enable else 0))

    def timing_read(self):
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        fl = ctypes.c_double()
        by = ctypes.c_double()
        _check(lib().pulse_stage_timing_read(self.h, ctypes.byref(n), ctypes.byref(ms),
                                             ctypes.byref(fl), ctypes.byref(by)))
        return n.value, ms.value, fl.value, by.value


class MbIO(ctypes.Structure):
    _fields_ = [("x", _vp), ("u", _vp), ("temb", _vp), ("g_enc", _vp), ("g_dec", _vp),
                ("y_enc", _vp), ("y_dec", _vp), ("dx", _vp), ("du", _vp), ("dtemb", _vp)]


def sched_build(D, M):
    """The wave schedule of (D, M): (table as a [D][T] list of lists of
    s*M+m or -1, exact flag)."""
    T = _i32()
    ex = _i32()
    _check(lib().pulse_sched_build(D, M, None, 0, ctypes.byref(T), ctypes.byref(ex)))
    buf = (_i32 * (D * T.value))()
    _check(lib().pulse_sched_build(D, M, buf, T.value, ctypes.byref(T), ctypes.byref(ex)))
    t = T.value
    return [[buf[d * t + i] for i in range(t)] for d in range(D)], bool(ex.value)


def sched_check(D, M, table):
    """Bit mask of violated schedule constraints (0: valid)."""
    T = len(table[0]) if table else 0
    buf = (_i32 * (D * T))(*[v for row in table for v in row])
    bad = _i32()
    _check(lib().pulse_sched_check(D, M, buf, T, ctypes.byref(bad)))
    return bad.value


def sched_inflight(D, M, table):
    """Peak microbatches in flight per device under the schedule."""
    T = len(table[0]) if table else 0
    buf = (_i32 * (D * T))(*[v for row in table for v in row])
    peak = (_i32 * D)()
    _check(lib().pulse_sched_inflight(D, M, buf, T, peak))
    return list(peak)


def sched_run_device(stage, D, d, M, table, io=None, t0=0, t1=None, stream=None):
    """Run steps [t0, t1) of device d's row of the schedule on ``stage``.
    ``io``: M dicts of device tensors (x, u, temb, g_enc, g_dec in; y_enc,
    y_dec, dx, du out; dtemb optional); None for a dry-run stage."""
    T = len(table[0])
    t1 = T if t1 is None else t1
    buf = (_i32 * (D * T))(*[v for row in table for v in row])
    arr = (MbIO * M)()
    keep = []
    if io is not None:
        for m in range(M):
            for k, _ in MbIO._fields_:
                t = io[m].get(k)
                setattr(arr[m], k, t.data_ptr() if t is not None else None)
                keep.append(t)
    s = None if stage.dry else _stream_handle(stream)
    _check(lib().pulse_sched_run_device(stage.h, D, d, M, buf, T, t0, t1, arr, s))


def mfma_probe(shape, blocks, iters, out, stream=None):
    """Launch the matrix-core throughput probe (see pulse_mfma_probe) on the
    current torch stream; returns the launch's FLOPs."""
    import torch
    fl = ctypes.c_double()
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    _check(lib().pulse_mfma_probe(shape, blocks, iters, out.data_ptr(), ctypes.byref(fl), s))
    return fl.value


def run_microbatch(stage, mb, b, dtemb=None):
    """F_enc, F_dec, B_dec, B_enc of one microbatch with boundary tensors
    ``b`` (device tensors x, u, temb, g_enc, g_dec).  Returns the outputs."""
    y_enc = stage.forward(ENC, mb, b["x"], b["temb"])
    y_dec = stage.forward(DEC, mb, b["u"], b["temb"])
    du = stage.backward(DEC, mb, b["g_dec"], dtemb=dtemb)
    dx = stage.backward(ENC, mb, b["g_enc"], dtemb=dtemb)
    return dict(y_enc=y_enc, y_dec=y_dec, du=du, dx=dx)
