"""ctypes binding of the transformer-block stage (``include/pulse_tstage.h``).

Argument marshalling only: every step runs in the library's HIP kernels, and
loading fails loudly when the library has not been built.
"""

from __future__ import annotations

import ctypes

import numpy as np

from . import configs as _cfg
from .stage import BF16, DEC, ENC, FLAG_DRY_RUN, MbIO, _check, _ptr, _stream_handle, lib as _lib

__all__ = ["TStageDesc", "TStage", "ENC", "DEC", "tsched_run_device"]

_i32 = ctypes.c_int32
_vp = ctypes.c_void_p
_bound = False


class TStageDesc(ctypes.Structure):
    _fields_ = [("batch", _i32), ("tokens", _i32), ("width", _i32), ("heads", _i32),
                ("mlp_ratio", _i32), ("eps", ctypes.c_float), ("dtype", ctypes.c_int),
                ("n_enc", _i32), ("n_dec", _i32), ("max_inflight", _i32),
                ("flags", ctypes.c_uint32)]


def lib():
    global _bound
    L = _lib()
    if not _bound:
        st = ctypes.c_int
        L.pulse_tstage_create.argtypes = [ctypes.POINTER(TStageDesc), ctypes.POINTER(_vp)]
        L.pulse_tstage_create.restype = st
        L.pulse_tstage_destroy.argtypes = [_vp]
        L.pulse_tstage_destroy.restype = None
        L.pulse_tstage_sizes.argtypes = [_vp, ctypes.POINTER(ctypes.c_int64),
                                         ctypes.POINTER(ctypes.c_size_t)]
        L.pulse_tstage_sizes.restype = st
        L.pulse_tstage_param_layout.argtypes = [_vp, _i32, ctypes.c_char_p,
                                                ctypes.POINTER(ctypes.c_int64),
                                                ctypes.POINTER(_i32)]
        L.pulse_tstage_param_layout.restype = st
        L.pulse_tstage_bind.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_size_t]
        L.pulse_tstage_bind.restype = st
        L.pulse_tstage_sync_params.argtypes = [_vp, _vp]
        L.pulse_tstage_sync_params.restype = st
        L.pulse_tstage_forward.argtypes = [_vp, ctypes.c_int, _i32, _vp, _vp, _vp]
        L.pulse_tstage_forward.restype = st
        L.pulse_tstage_backward.argtypes = [_vp, ctypes.c_int, _i32, _vp, _vp, _vp]
        L.pulse_tstage_backward.restype = st
        L.pulse_tstage_skip_grad.argtypes = [_vp, _i32, _i32, _vp, _vp]
        L.pulse_tstage_skip_grad.restype = st
        L.pulse_tstage_release.argtypes = [_vp, _i32]
        L.pulse_tstage_release.restype = st
        L.pulse_tstage_reset.argtypes = [_vp]
        L.pulse_tstage_reset.restype = st
        L.pulse_tstage_inflight.argtypes = [_vp]
        L.pulse_tstage_inflight.restype = _i32
        L.pulse_tstage_overlap_bwd.argtypes = [_vp, _i32]
        L.pulse_tstage_overlap_bwd.restype = st
        L.pulse_tstage_flush.argtypes = [_vp, _vp]
        L.pulse_tstage_flush.restype = st
        L.pulse_tstage_timing.argtypes = [_vp, _i32]
        L.pulse_tstage_timing.restype = st
        L.pulse_tstage_timing_read.argtypes = [_vp, ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(ctypes.c_double),
                                               ctypes.POINTER(ctypes.c_double),
                                               ctypes.POINTER(ctypes.c_double)]
        L.pulse_tstage_timing_read.restype = st
        L.pulse_tstage_flops.argtypes = [_vp]
        L.pulse_tstage_flops.restype = ctypes.c_double
        L.pulse_tsched_run_device.argtypes = [_vp, _i32, _i32, _i32, ctypes.POINTER(_i32), _i32,
                                              _i32, _i32, ctypes.POINTER(MbIO), _vp]
        L.pulse_tsched_run_device.restype = st
        _bound = True
    return L


def make_desc(desc, dry_run=False):
    return TStageDesc(batch=desc["batch"], tokens=desc["tokens"], width=desc["width"],
                      heads=desc["heads"], mlp_ratio=desc.get("mlp", 4), eps=desc["eps"],
                      dtype=BF16 if desc["dtype"] == _cfg.BF16 else 0,
                      n_enc=desc["n_enc"], n_dec=desc["n_dec"],
                      max_inflight=desc.get("max_inflight", 1),
                      flags=FLAG_DRY_RUN if dry_run else 0)


class TStage:
    """One collocated transformer-block stage (``desc``: a config dict of
    kind "transformer").  With ``dry_run`` only the bookkeeping runs."""

    def __init__(self, desc, device="cuda", dry_run=False):
        self.desc = desc
        self.dry = dry_run
        self.h = _vp()
        cdesc = make_desc(desc, dry_run)
        _check(lib().pulse_tstage_create(ctypes.byref(cdesc), ctypes.byref(self.h)))
        n = ctypes.c_int64()
        ws = ctypes.c_size_t()
        _check(lib().pulse_tstage_sizes(self.h, ctypes.byref(n), ctypes.byref(ws)))
        self.n_params = n.value
        self.ws_bytes = ws.value
        self.layout = self._read_layout()
        self.B, self.L, self.C = desc["batch"], desc["tokens"], desc["width"]
        self.params = self.grads = self.workspace = None
        if not dry_run:
            import torch
            self.params = torch.zeros(self.n_params, dtype=torch.float32, device=device)
            self.grads = torch.zeros(self.n_params, dtype=torch.float32, device=device)
            self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
            _check(lib().pulse_tstage_bind(self.h, _ptr(self.params), _ptr(self.grads),
                                           _ptr(self.workspace), self.ws_bytes))

    def __del__(self):
        try:
            if self.h:
                lib().pulse_tstage_destroy(self.h)
                self.h = _vp()
        except Exception:
            pass

    def _read_layout(self):
        cnt = ctypes.c_int64()
        _check(lib().pulse_tstage_param_layout(self.h, -1, None, ctypes.byref(cnt), None))
        out = {}
        for i in range(cnt.value):
            name = ctypes.create_string_buffer(64)
            off = ctypes.c_int64()
            shape = (_i32 * 4)()
            _check(lib().pulse_tstage_param_layout(self.h, i, name, ctypes.byref(off), shape))
            out[name.value.decode()] = (off.value, tuple(s for s in shape if s > 0))
        return out

    def set_params(self, params, stream=None):
        import torch
        flat = np.zeros(self.n_params, dtype=np.float32)
        for name, (off, shape) in self.layout.items():
            a = np.asarray(params[name], dtype=np.float32)
            assert a.shape == shape, (name, a.shape, shape)
            flat[off:off + a.size] = a.ravel()
        self.params.copy_(torch.from_numpy(flat))
        self.sync_params(stream)

    def sync_params(self, stream=None):
        _check(lib().pulse_tstage_sync_params(self.h, None if self.dry else _stream_handle(stream)))

    def zero_grads(self):
        self.grads.zero_()

    def grads_dict(self):
        g = self.grads.cpu().numpy()
        return {n: g[o:o + int(np.prod(s))].reshape(s).copy() for n, (o, s) in self.layout.items()}

    def act(self, device="cuda"):
        import torch
        return torch.empty((self.B, self.L, self.C), dtype=torch.bfloat16, device=device)

    def to_dev(self, a, device="cuda"):
        import torch
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(
            device=device, dtype=torch.bfloat16)

    def forward(self, half, mb, inp, out=None, stream=None):
        if self.dry:
            _check(lib().pulse_tstage_forward(self.h, half, mb, None, None, None))
            return None
        out = self.act() if out is None else out
        _check(lib().pulse_tstage_forward(self.h, half, mb, _ptr(inp), _ptr(out),
                                          _stream_handle(stream)))
        return out

    def backward(self, half, mb, dout, din=None, stream=None):
        if self.dry:
            _check(lib().pulse_tstage_backward(self.h, half, mb, None, None, None))
            return None
        din = self.act() if din is None else din
        _check(lib().pulse_tstage_backward(self.h, half, mb, _ptr(dout), _ptr(din),
                                           _stream_handle(stream)))
        return din

    def skip_grad(self, mb, slot, stream=None):
        import torch
        dst = torch.empty((self.B, self.L, self.C), dtype=torch.float32, device="cuda")
        _check(lib().pulse_tstage_skip_grad(self.h, mb, slot, _ptr(dst), _stream_handle(stream)))
        return dst

    def release(self, mb):
        _check(lib().pulse_tstage_release(self.h, mb))

    def reset(self):
        _check(lib().pulse_tstage_reset(self.h))

    def inflight(self):
        return lib().pulse_tstage_inflight(self.h)

    def flops(self):
        return lib().pulse_tstage_flops(self.h)

    def overlap_bwd(self, enable):
        _check(lib().pulse_tstage_overlap_bwd(self.h, 1 if enable else 0))

    def flush(self, stream=None):
        _check(lib().pulse_tstage_flush(self.h, None if self.dry else _stream_handle(stream)))

    def timing(self, enable):
        _check(lib().pulse_tstage_timing(self.h, 1 if enable else 0))

    def timing_read(self):
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        fl = ctypes.c_double()
        by = ctypes.c_double()
        _check(lib().pulse_tstage_timing_read(self.h, ctypes.byref(n), ctypes.byref(ms),
                                              ctypes.byref(fl), ctypes.byref(by)))
        return n.value, ms.value, fl.value, by.value


def tsched_run_device(stage, D, d, M, table, io=None, t0=0, t1=None, stream=None):
    """Run steps [t0, t1) of device d's row of the schedule on a transformer
    stage.  ``io``: M dicts of device tensors (x, u, g_enc, g_dec in; y_enc,
    y_dec, dx, du out); None for a dry-run stage."""
    L = lib()
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
    _check(L.pulse_tsched_run_device(stage.h, D, d, M, buf, T, t0, t1, arr, s))
