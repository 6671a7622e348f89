"""CPU oracle for the hybrid-parallelism tuner (plain Python enumeration).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` may import this module; the
library's tuner (C++, ``pulse_tune``) shares no code with it.

What is modelled (Sec. VI)
--------------------------
N devices run G data-parallel replicas of a pipeline of P devices (N = P*G)
holding 2P collocated stages, fed microbatches of b samples.  Per stage s
(1-based, s = 1 .. 2P), from the ops the skip-aware partition puts in it:
T_f^s(b) the forward time at microbatch size b, M_theta^s the parameter
bytes, M_a^s the activation bytes kept per sample, M_o^s the output bytes
per sample of its last op.  The models of Sec. VI:

    M_peak  = 7 (M_theta^P + M_theta^(P+1)) + P (M_a^P + M_a^(P+1)) b
              + P M_o^(P-1)
    T_sched = (10P - 4) T_f(b) + (10P - 12) (t_lat + b M_o / B_inter) + T_AR
    T_f(b)  = max_s T_f^s(b),   M_o = max_s M_o^s
    T_AR    = t_lat + 2 (G - 1) M_theta^max / (G B_intra),
              M_theta^max = max_s M_theta^s
    T_sample = T_sched / (b P G)

For every factorisation N = P G (with 2P <= number of ops) the largest b of
the candidate list with M_peak < M_limit is kept, and the configuration with
the smallest T_sample wins.

Readings (the paper leaves them open or its formulas break down): the
partition for (P, b) is the skip-aware optimum of the op forward times at b
with boundary bytes b * (op output bytes per sample); for P = 1 the
transfer term's factor 10P - 12 is negative and is taken as 0 (one device
sends nothing), and the stage P-1 of M_peak does not exist (its term is 0);
M_o^(P-1) enters M_peak as printed, without a factor b; T_AR is charged
for G = 1 as printed (its latency term remains); ties go to the smaller P,
then the smaller G.
"""

from __future__ import annotations

import math

from oracle import partition_oracle as po


def stage_sums(cuts, n, per_op):
    return [sum(per_op[a:b + 1]) for a, b in po.stages_of(n, cuts)]


def stage_last(cuts, n, per_op):
    return [per_op[b] for a, b in po.stages_of(n, cuts)]


def evaluate(P, G, b, cuts, n, t_f_b, m_theta, m_a, m_o, t_lat, b_inter, b_intra):
    """(T_sample, T_sched, M_peak, T_AR) of one configuration whose 2P
    stages are given by `cuts` (0-based cut list)."""
    Tf = stage_sums(cuts, n, t_f_b)
    Mth = stage_sums(cuts, n, m_theta)
    Ma = stage_sums(cuts, n, m_a)
    Mo = stage_last(cuts, n, m_o)
    # stage s (1-based) is index s-1 here
    m_peak = 7 * (Mth[P - 1] + Mth[P]) + P * (Ma[P - 1] + Ma[P]) * b
    if P >= 2:
        m_peak += P * Mo[P - 2]
    t_ar = t_lat + 2 * (G - 1) * max(Mth) / (G * b_intra)
    comm_steps = max(0, 10 * P - 12)
    t_sched = (10 * P - 4) * max(Tf) + comm_steps * (t_lat + b * max(Mo) / b_inter) + t_ar
    return t_sched / (b * P * G), t_sched, m_peak, t_ar


def tune(N, bs, t_f, m_theta, m_a, m_o, skips, lam, t_lat, b_inter, b_intra, m_limit):
    """Best configuration as a dict (None when nothing fits), and every
    (P, G, b) row evaluated.  t_f[k] is the per-op forward time at bs[k]."""
    n = len(m_theta)
    rows = []
    best = None
    for P in range(1, N + 1):
        if N % P or 2 * P > n:
            continue
        G = N // P
        chosen = None
        for k, b in enumerate(bs):
            c, args = po.optimum(n, 2 * P, t_f[k], [b * v for v in m_o], skips,
                                 lam, t_lat, b_inter)
            if c == math.inf:
                continue
            cuts = args[0]
            ts, tsch, mp, tar = evaluate(P, G, b, cuts, n, t_f[k], m_theta, m_a, m_o,
                                         t_lat, b_inter, b_intra)
            row = dict(P=P, G=G, b=b, t_sample=ts, t_sched=tsch, m_peak=mp, t_ar=tar,
                       feasible=mp < m_limit, cuts=cuts)
            rows.append(row)
            if row["feasible"]:
                chosen = row  # candidates ascend: the last feasible is the largest b
        if chosen is not None and (best is None or chosen["t_sample"] < best["t_sample"]):
            best = chosen
    return best, rows
