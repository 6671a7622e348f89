"""CPU oracle for the skip-aware balanced partition (plain Python, exhaustive).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` may import this module; the
library's partitioner (C++, ``pulse_partition``) shares no code with it.

What is modelled (Sec. IV-B)
----------------------------
A model is an ordered sequence of n operations with forward times t_f[l]
and output activation sizes m_a[l] (bytes of the tensor op l hands to op
l+1).  Skip connections are pairs (c1, c2), c1 < c2, of operation indices.
A partition cuts the sequence into p contiguous, non-empty stages
S_1 .. S_p (p even: the stages pair up as q and p-q+1).  It is valid when
every skip pair with c2 - c1 > 1 has op c1 in some stage q and op c2 in
stage p-q+1 (adjacent operations need no collocation).  Its cost is the
largest stage cost, and the partition sought minimises it (the DP target
of Sec. IV-B):

    cost(S_m) = sum of t_f over S_m + lam * (t_lat + a_m / b_inter)

where a_m is the boundary tensor the stage pays for: the output of its last
operation for the first p/2 stages, the output of the operation just before
its first one for the last p/2 stages (the two cost terms L and R of the
recurrence).

Readings (the paper leaves them open, or its formulas disagree): the
objective's communication term carries the static latency t_lat as the L and
R terms do; each stage pays exactly one boundary tensor as above; a model
with no valid partition has cost +inf.  Operation indices here are 0-based.
"""

from __future__ import annotations

import itertools
import math


def stages_of(n, cuts):
    """[(first, last)] of each stage; cuts[k] is the last op of stage k."""
    bounds = [-1] + list(cuts) + [n - 1]
    return [(bounds[k] + 1, bounds[k + 1]) for k in range(len(bounds) - 1)]


def is_valid(n, p, cuts, skips):
    st = stages_of(n, cuts)
    if any(a > b for a, b in st):
        return False
    part = [0] * n
    for q, (a, b) in enumerate(st):
        for l in range(a, b + 1):
            part[l] = q  # 0-based stage index
    for c1, c2 in skips:
        c1, c2 = min(c1, c2), max(c1, c2)
        if c2 - c1 <= 1:
            continue
        if part[c2] != p - 1 - part[c1]:
            return False
    return True


def stage_costs(n, p, cuts, t_f, m_a, lam, t_lat, b_inter):
    out = []
    for q, (a, b) in enumerate(stages_of(n, cuts)):
        work = sum(t_f[a:b + 1])
        if q < p // 2:
            boundary = m_a[b]
        else:
            boundary = m_a[a - 1]
        out.append(work + lam * (t_lat + boundary / b_inter))
    return out


def cost(n, p, cuts, t_f, m_a, skips, lam=0.0, t_lat=0.0, b_inter=1.0):
    """Largest stage cost of the partition, +inf when it is not valid."""
    if not is_valid(n, p, cuts, skips):
        return math.inf
    return max(stage_costs(n, p, cuts, t_f, m_a, lam, t_lat, b_inter))


def optimum(n, p, t_f, m_a, skips, lam=0.0, t_lat=0.0, b_inter=1.0):
    """(minimum cost, cut lists reaching it) over every way to place p-1
    cuts between n operations."""
    best, arg = math.inf, []
    for cuts in itertools.combinations(range(n - 1), p - 1):
        c = cost(n, p, cuts, t_f, m_a, skips, lam, t_lat, b_inter)
        if c < best:
            best, arg = c, [cuts]
        elif c == best and c < math.inf:
            arg.append(cuts)
    return best, arg


def comm_volume(n, m_a, skips, n_stages, cuts, collocated):
    """Forward point-to-point bytes of one sample: stage boundaries between
    devices, plus every skip that crosses devices, forwarded stage by stage
    from its source device to its destination device (the traffic model of
    Sec. II-C counts a skip between adjacent ops apart from the boundary).
    Collocated placement puts stage s on device min(s, n_stages - 1 - s)."""
    def dev_of_stage(st):
        return min(st, n_stages - 1 - st) if collocated else st
    dev = [0] * n
    for st, (a, b) in enumerate(stages_of(n, cuts)):
        for l in range(a, b + 1):
            dev[l] = dev_of_stage(st)
    v = 0.0
    for st in range(n_stages - 1):
        if dev_of_stage(st) != dev_of_stage(st + 1):
            v += m_a[cuts[st]]
    for c1, c2 in skips:
        c1, c2 = min(c1, c2), max(c1, c2)
        if dev[c1] == dev[c2]:
            continue
        # a valid collocated partition keeps non-adjacent skips on one device
        assert not (collocated and c2 - c1 > 1), "a skip crosses devices"
        v += m_a[c1] * abs(dev[c2] - dev[c1])
    return v

