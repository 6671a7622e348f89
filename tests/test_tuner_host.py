"""The library's hybrid tuner (pulse_tune, pulse_tune_eval; Sec. VI) against
the tuner oracle, on the host."""

import random

import pytest

from oracle import partition_oracle as po
from oracle import tuner_oracle as to
from paper_2606_19163_amd import plan
from paper_2606_19163_amd import stage as S

from test_oracle_tuner import CASES, EX, _random_problem


@pytest.fixture(scope="module", autouse=True)
def built():
    import os
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_19163_amd import build
        build.build()
    yield


KEYS = ("P", "G", "b", "t_sample", "t_sched", "m_peak", "t_ar")


def _same(a, b):
    for k in KEYS:
        assert a[k] == pytest.approx(b[k], rel=1e-12, abs=1e-15), k
    assert bool(a["feasible"]) == bool(b["feasible"])


@pytest.mark.parametrize("m_limit,want", CASES)
def test_worked_example(m_limit, want):
    best, rows = plan.tune(2, m_limit=m_limit, **EX)
    ref, ref_rows = to.tune(2, m_limit=m_limit, **EX)
    if want is None:
        assert best is None and ref is None
    else:
        _same(best, ref)
        assert (best["P"], best["G"], best["b"]) == want[:3]
    assert len(rows) == len(ref_rows)
    for a, b in zip(rows, ref_rows):
        _same(a, b)


def test_eval_matches_the_models():
    rng = random.Random(9)
    for _ in range(100):
        n = rng.randint(4, 12)
        pr = _random_problem(rng, n)
        P = rng.randint(1, n // 2)
        G = rng.randint(1, 4)
        k = rng.randrange(len(pr["bs"]))
        cuts = sorted(rng.sample(range(n - 1), 2 * P - 1))
        got = plan.tune_eval(P, G, k, cuts, m_limit=50.0, **pr)
        ts, tsch, mp, tar = to.evaluate(P, G, pr["bs"][k], cuts, n, pr["t_f"][k],
                                        pr["m_theta"], pr["m_a"], pr["m_o"], pr["t_lat"],
                                        pr["b_inter"], pr["b_intra"])
        _same(got, dict(P=P, G=G, b=pr["bs"][k], t_sample=ts, t_sched=tsch, m_peak=mp,
                        t_ar=tar, feasible=mp < 50.0))


def _unique_partitions(pr, N):
    n = len(pr["m_theta"])
    for P in range(1, N + 1):
        if N % P or 2 * P > n:
            continue
        for k, b in enumerate(pr["bs"]):
            c, args = po.optimum(n, 2 * P, pr["t_f"][k], [b * v for v in pr["m_o"]],
                                 pr["skips"], pr["lam"], pr["t_lat"], pr["b_inter"])
            if len(args) > 1:
                return False
    return True


def test_enumeration_matches_the_oracle():
    rng = random.Random(21)
    checked = 0
    for _ in range(60):
        n = rng.randint(4, 10)
        pr = _random_problem(rng, n)
        N = rng.choice([1, 2, 4, 6, 8])
        if not _unique_partitions(pr, N):
            continue  # the oracle and the library may break partition ties apart
        m_limit = rng.choice([20.0, 40.0, 80.0, 1e9])
        best, rows = plan.tune(N, m_limit=m_limit, **pr)
        ref, ref_rows = to.tune(N, m_limit=m_limit, **pr)
        assert (best is None) == (ref is None)
        if best is not None:
            _same(best, ref)
        assert len(rows) == len(ref_rows)
        for a, b in zip(rows, ref_rows):
            _same(a, b)
        checked += 1
    assert checked >= 20


def test_arguments():
    with pytest.raises(S.PulseError):
        plan.tune(0, **EX)
    with pytest.raises(S.PulseError):
        plan.tune(2, **dict(EX, bs=[2, 1]))
    with pytest.raises(S.PulseError):
        plan.tune(2, **dict(EX, b_intra=0.0))
    with pytest.raises(S.PulseError):
        plan.tune_eval(3, 1, 0, [0, 1, 2, 3, 4], **EX)  # 2P > n_ops
