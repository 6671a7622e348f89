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
