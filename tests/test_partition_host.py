"""The library's skip-aware partitioner (pulse_partition, the dynamic
program of Sec. IV-B) against the exhaustive oracle, on the host."""

import math
import random
import time

import pytest

from oracle import partition_oracle as po
from paper_2606_19163_amd import plan
from paper_2606_19163_amd import stage as S


@pytest.fixture(scope="module", autouse=True)
def built():
    import os
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_19163_amd import build
        build.build()
    yield


def _random_case(rng, n_max=10):
    n = rng.randint(2, n_max)
    p = rng.choice([p for p in (2, 4, 6, 8) if p <= n])
    t = [rng.choice([0.5, 1.0, 2.0, 3.0, 5.0]) for _ in range(n)]
    m = [rng.choice([0.0, 1.0, 4.0]) for _ in range(n)]
    if rng.random() < 0.5:
        skips = [(i, n - 1 - i) for i in range(n // 2) if rng.random() < 0.6]
    else:
        skips = []
        for _ in range(rng.randint(0, 3)):
            a, b = rng.randrange(n), rng.randrange(n)
            if a != b:
                skips.append((a, b))
    lam = rng.choice([0.0, 0.0, 0.5])
    return n, p, t, m, skips, lam, rng.choice([0.0, 1.0]), rng.choice([1.0, 2.0])


def test_matches_exhaustive_search():
    rng = random.Random(11)
    seen_inf = seen_fin = 0
    for _ in range(300):
        n, p, t, m, skips, lam, tl, bi = _random_case(rng)
        ref, args = po.optimum(n, p, t, m, skips, lam, tl, bi)
        cuts, c = plan.partition(t, m, skips, p, lam, tl, bi)
        if ref == math.inf:
            seen_inf += 1
            assert c == math.inf and cuts == [-1] * (p - 1)
            continue
        seen_fin += 1
        assert c == pytest.approx(ref, rel=1e-12, abs=1e-12)
        assert po.is_valid(n, p, cuts, skips)
        assert po.cost(n, p, cuts, t, m, skips, lam, tl, bi) == pytest.approx(ref, rel=1e-12)
    assert seen_inf > 10 and seen_fin > 100


def test_cost_call_matches_the_oracle():
    rng = random.Random(5)
    for _ in range(200):
        n, p, t, m, skips, lam, tl, bi = _random_case(rng)
        cuts = sorted(rng.sample(range(n - 1), p - 1))
        c, valid, sc = plan.partition_cost(t, m, skips, p, cuts, lam, tl, bi)
        assert valid == po.is_valid(n, p, cuts, skips)
        assert sc == pytest.approx(po.stage_costs(n, p, cuts, t, m, lam, tl, bi))
        assert c == (max(sc) if valid else math.inf)


def test_hand_cases():
    assert plan.partition([1.0] * 8, [0.0] * 8, [(0, 3)], 4) == ([0, 1, 2], 5.0)
    assert plan.partition([1.0] * 4, [0.0] * 4, [(0, 2)], 4)[1] == math.inf
    assert plan.partition([0.0] * 4, [5.0, 1.0, 7.0, 0.0], [], 2, lam=1.0) == ([1], 1.0)


def test_large_mirrored_model_is_fast_and_balanced():
    # 256 ops in mirrored pairs, 16 stages: the DP stays well under a second
    rng = random.Random(2)
    n, p = 256, 16
    t = [rng.uniform(0.5, 2.0) for _ in range(n)]
    skips = [(i, n - 1 - i) for i in range(0, n // 2, 3)]
    t0 = time.perf_counter()
    cuts, c = plan.partition(t, [1.0] * n, skips, p, lam=0.1)
    assert time.perf_counter() - t0 < 5.0
    c2, valid, sc = plan.partition_cost(t, [1.0] * n, skips, p, cuts, lam=0.1)
    assert valid and c2 == pytest.approx(c)
    assert c <= 1.5 * sum(t) / p


def test_arguments():
    with pytest.raises(S.PulseError):
        plan.partition([1.0] * 4, [0.0] * 4, [], 3)       # odd p
    with pytest.raises(S.PulseError):
        plan.partition([1.0] * 4, [0.0] * 4, [], 6)       # p > n
    with pytest.raises(S.PulseError):
        plan.partition([1.0] * 4, [0.0] * 4, [(0, 9)], 2)  # skip out of range
    with pytest.raises(S.PulseError):
        plan.partition([-1.0] * 4, [0.0] * 4, [], 2)      # negative time
    with pytest.raises(S.PulseError):
        plan.partition([1.0] * 4, [0.0] * 4, [], 2, b_inter=0.0)
    with pytest.raises(S.PulseError):
        plan.partition_cost([1.0] * 4, [0.0] * 4, [], 2, [3])  # cut at the last op


def test_comm_volume_matches_the_oracle():
    rng = random.Random(13)
    for _ in range(200):
        n = rng.randint(2, 12)
        m = [rng.choice([0.0, 1.0, 4.0, 9.0]) for _ in range(n)]
        skips = [(i, n - 1 - i) for i in range(n // 2) if rng.random() < 0.6]
        p = rng.randint(1, n)
        cuts = sorted(rng.sample(range(n - 1), p - 1))
        assert plan.comm_volume(m, skips, p, cuts, False) == \
            pytest.approx(po.comm_volume(n, m, skips, p, cuts, False))
        if p % 2 == 0 and po.is_valid(n, p, cuts, skips):
            assert plan.comm_volume(m, skips, p, cuts, True) == \
                pytest.approx(po.comm_volume(n, m, skips, p, cuts, True))
    # a collocated placement whose skip crosses devices is rejected
    with pytest.raises(S.PulseError):
        plan.comm_volume([1.0] * 8, [(0, 3)], 4, [1, 3, 5], True)
