"""Pins of the tuner oracle (oracle/tuner_oracle.py): a worked example whose
numbers were computed by hand from the models of Sec. VI, at four memory
limits that move the choice between pipeline and data parallelism and
between microbatch sizes, the one-device case, and monotonicity in the
link bandwidths."""

import random

import pytest

from oracle import tuner_oracle as to

# 4 unit ops with one long skip (op 0 -> op 3), 2 devices, b in {1, 2}
EX = dict(bs=[1, 2], t_f=[[1.0] * 4, [2.0] * 4], m_theta=[10.0] * 4, m_a=[1.0] * 4,
          m_o=[4.0] * 4, skips=[(0, 3)], lam=0.0, t_lat=0.5, b_inter=2.0, b_intra=4.0)

# By hand.  P = 1, G = 2: stages {0,1} | {2,3}; M_peak = 7*40 + 4b = 280 + 4b;
# T_AR = 0.5 + 2*1*20/(2*4) = 5.5; T_sched = 6 T_f(b) + 5.5 with T_f = 2b
# (the transfer term's factor 10P-12 = -2 counts as 0), so b = 1: 17.5 ->
# T_sample 17.5/2 = 8.75; b = 2: 29.5 -> 29.5/4 = 7.375.
# P = 2, G = 1: one op per stage; M_peak = 7*20 + 2*2*b + 2*4 = 148 + 4b;
# T_AR = 0.5; T_sched = 16 T_f(b) + 8 (0.5 + 4b/2) + 0.5 with T_f = b, so
# b = 1: 36.5 -> 18.25; b = 2: 68.5 -> 17.125.
CASES = [
    (300.0, (1, 2, 2, 7.375)),
    (285.0, (1, 2, 1, 8.75)),
    (155.0, (2, 1, 1, 18.25)),
    (150.0, None),
]


@pytest.mark.parametrize("m_limit,want", CASES)
def test_worked_example(m_limit, want):
    best, rows = to.tune(2, m_limit=m_limit, **EX)
    if want is None:
        assert best is None
        return
    P, G, b, ts = want
    assert (best["P"], best["G"], best["b"]) == (P, G, b)
    assert best["t_sample"] == pytest.approx(ts, rel=1e-12)
    by = {(r["P"], r["b"]): r for r in rows}
    assert by[(1, 1)]["m_peak"] == 284.0 and by[(1, 2)]["m_peak"] == 288.0
    assert by[(2, 1)]["m_peak"] == 152.0 and by[(2, 2)]["m_peak"] == 156.0
    assert by[(1, 2)]["t_ar"] == 5.5 and by[(2, 2)]["t_ar"] == 0.5
    assert by[(2, 2)]["t_sched"] == 68.5 and by[(1, 1)]["t_sched"] == 17.5


def test_one_device():
    best, rows = to.tune(1, m_limit=1e9, **EX)
    assert (best["P"], best["G"], best["b"]) == (1, 1, 2)
    # no replicas: the all-reduce is its latency alone
    assert best["t_ar"] == 0.5
    assert best["t_sched"] == pytest.approx(6 * 4.0 + 0.5)


def _random_problem(rng, n):
    bs = [1, 2, 4]
    base = [rng.uniform(0.5, 2.0) for _ in range(n)]
    t_f = [[v * b * rng.uniform(0.9, 1.0) for v in base] for b in bs]
    return dict(bs=bs, t_f=t_f, m_theta=[rng.uniform(1, 5) for _ in range(n)],
                m_a=[rng.uniform(0.5, 2) for _ in range(n)],
                m_o=[rng.uniform(0.5, 2) for _ in range(n)],
                skips=[(i, n - 1 - i) for i in range(n // 2) if rng.random() < 0.5],
                lam=0.0, t_lat=0.1, b_inter=3.0, b_intra=5.0)


def test_monotone_in_bandwidth():
    rng = random.Random(4)
    for _ in range(10):
        pr = _random_problem(rng, 8)
        best, _ = to.tune(4, m_limit=60.0, **pr)
        if best is None:
            continue
        faster = dict(pr, b_intra=2 * pr["b_intra"], b_inter=2 * pr["b_inter"])
        # same partitions and feasibility, cheaper transfers and all-reduce
        assert to.tune(4, m_limit=60.0, **faster)[0]["t_sample"] <= best["t_sample"] + 1e-12
