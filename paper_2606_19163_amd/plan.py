"""Python binding of the planning calls (include/pulse_plan.h): argument
marshalling only; the partitioner runs in the library."""

from __future__ import annotations

import ctypes
import math

from . import stage as _S

_d = ctypes.c_double
_i32 = ctypes.c_int32
_dp = ctypes.POINTER(_d)
_ip = ctypes.POINTER(_i32)


class PartProblem(ctypes.Structure):
    _fields_ = [("n_ops", _i32), ("t_f", _dp), ("m_a", _dp), ("n_skips", _i32),
                ("skips", _ip), ("lam", _d), ("t_lat", _d), ("b_inter", _d)]


_bound = False


def _lib():
    global _bound
    L = _S.lib()
    if not _bound:
        L.pulse_partition.argtypes = [ctypes.POINTER(PartProblem), _i32, _ip, _dp]
        L.pulse_partition.restype = ctypes.c_int
        L.pulse_partition_cost.argtypes = [ctypes.POINTER(PartProblem), _i32, _ip, _dp, _ip,
                                           _dp]
        L.pulse_partition_cost.restype = ctypes.c_int
        _bound = True
    return L


def _problem(t_f, m_a, skips, lam, t_lat, b_inter):
    n = len(t_f)
    tf = (_d * n)(*t_f)
    ma = (_d * n)(*m_a)
    flat = [int(v) for pair in skips for v in pair]
    sk = (_i32 * max(1, len(flat)))(*flat)
    pb = PartProblem(n, tf, ma, len(skips), sk, lam, t_lat, b_inter)
    return pb, (tf, ma, sk)


def partition(t_f, m_a, skips, p, lam=0.0, t_lat=0.0, b_inter=1.0):
    """(cuts, cost): the skip-aware balanced partition into p stages; cuts[k]
    is the last op of stage k; cost is +inf (and cuts all -1) when no
    partition satisfies the skip constraints."""
    pb, keep = _problem(t_f, m_a, skips, lam, t_lat, b_inter)
    cuts = (_i32 * max(1, p - 1))()
    cost = _d()
    _S._check(_lib().pulse_partition(ctypes.byref(pb), p, cuts, ctypes.byref(cost)))
    return [cuts[k] for k in range(p - 1)], cost.value


def comm_volume(m_a, skips, n_stages, cuts, collocated):
    """Forward point-to-point bytes of one sample (pulse_comm_volume)."""
    n = len(m_a)
    pb, keep = _problem([0.0] * n, m_a, skips, 0.0, 0.0, 1.0)
    L = _lib()
    if not getattr(L, "_cv_bound", False):
        L.pulse_comm_volume.argtypes = [ctypes.POINTER(PartProblem), _i32, _ip, _i32, _dp]
        L.pulse_comm_volume.restype = ctypes.c_int
        L._cv_bound = True
    c = (_i32 * max(1, n_stages - 1))(*cuts)
    v = _d()
    _S._check(L.pulse_comm_volume(ctypes.byref(pb), n_stages, c, 1 if collocated else 0,
                                  ctypes.byref(v)))
    return v.value


def partition_cost(t_f, m_a, skips, p, cuts, lam=0.0, t_lat=0.0, b_inter=1.0):
    """(cost, valid, stage costs) of a given partition."""
    pb, keep = _problem(t_f, m_a, skips, lam, t_lat, b_inter)
    c = (_i32 * max(1, p - 1))(*cuts)
    cost = _d()
    valid = _i32()
    sc = (_d * p)()
    _S._check(_lib().pulse_partition_cost(ctypes.byref(pb), p, c, ctypes.byref(cost),
                                          ctypes.byref(valid), sc))
    return cost.value, bool(valid.value), [sc[k] for k in range(p)]


INF = math.inf


class TuneProblem(ctypes.Structure):
    _fields_ = [("n_ops", _i32), ("n_b", _i32), ("b", _ip), ("t_f", _dp), ("m_theta", _dp),
                ("m_a", _dp), ("m_o", _dp), ("n_skips", _i32), ("skips", _ip), ("lam", _d),
                ("t_lat", _d), ("b_inter", _d), ("b_intra", _d), ("m_limit", _d)]


class TuneRow(ctypes.Structure):
    _fields_ = [("P", _i32), ("G", _i32), ("b", _i32), ("feasible", _i32), ("t_sample", _d),
                ("t_sched", _d), ("m_peak", _d), ("t_ar", _d)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_tbound = False


def _tlib():
    global _tbound
    L = _lib()
    if not _tbound:
        L.pulse_tune.argtypes = [ctypes.POINTER(TuneProblem), _i32, ctypes.POINTER(TuneRow),
                                 _ip, ctypes.POINTER(TuneRow), _i32, _ip]
        L.pulse_tune.restype = ctypes.c_int
        L.pulse_tune_eval.argtypes = [ctypes.POINTER(TuneProblem), _i32, _i32, _i32, _ip,
                                      ctypes.POINTER(TuneRow)]
        L.pulse_tune_eval.restype = ctypes.c_int
        _tbound = True
    return L


def _tproblem(bs, t_f, m_theta, m_a, m_o, skips, lam, t_lat, b_inter, b_intra, m_limit):
    n = len(m_theta)
    bb = (_i32 * len(bs))(*bs)
    tf = (_d * (len(bs) * n))(*[v for row in t_f for v in row])
    mt = (_d * n)(*m_theta)
    ma = (_d * n)(*m_a)
    mo = (_d * n)(*m_o)
    flat = [int(v) for pair in skips for v in pair]
    sk = (_i32 * max(1, len(flat)))(*flat)
    tp = TuneProblem(n, len(bs), bb, tf, mt, ma, mo, len(skips), sk, lam, t_lat, b_inter,
                     b_intra, m_limit)
    return tp, (bb, tf, mt, ma, mo, sk)


def tune(N, bs, t_f, m_theta, m_a, m_o, skips, lam=0.0, t_lat=0.0, b_inter=1.0,
         b_intra=1.0, m_limit=float("inf")):
    """(best row dict or None, rows): the hybrid configuration for N devices
    (pulse_tune).  t_f[k] holds the op forward times at microbatch bs[k]."""
    tp, keep = _tproblem(bs, t_f, m_theta, m_a, m_o, skips, lam, t_lat, b_inter, b_intra,
                         m_limit)
    best = TuneRow()
    found = _i32()
    n_rows = _i32()
    _S._check(_tlib().pulse_tune(ctypes.byref(tp), N, ctypes.byref(best), ctypes.byref(found),
                                 None, 0, ctypes.byref(n_rows)))
    rows = (TuneRow * max(1, n_rows.value))()
    _S._check(_tlib().pulse_tune(ctypes.byref(tp), N, ctypes.byref(best), ctypes.byref(found),
                                 rows, n_rows.value, ctypes.byref(n_rows)))
    return (best.as_dict() if found.value else None), [rows[k].as_dict()
                                                        for k in range(n_rows.value)]


def tune_eval(P, G, b_index, cuts, bs, t_f, m_theta, m_a, m_o, skips, lam=0.0, t_lat=0.0,
              b_inter=1.0, b_intra=1.0, m_limit=float("inf")):
    """The Sec. VI models of one configuration with the given stage cuts."""
    tp, keep = _tproblem(bs, t_f, m_theta, m_a, m_o, skips, lam, t_lat, b_inter, b_intra,
                         m_limit)
    c = (_i32 * max(1, len(cuts)))(*cuts)
    row = TuneRow()
    _S._check(_tlib().pulse_tune_eval(ctypes.byref(tp), P, G, b_index, c, ctypes.byref(row)))
    return row.as_dict()
