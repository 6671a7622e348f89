"""Pins of the partition oracle (oracle/partition_oracle.py): without skips
it equals the classical linear partition found by an independent method
(bisection on the answer with a greedy feasibility test); uniform mirrored
models split evenly; hand-worked cases fix the forced imbalance of a skip,
infeasibility, and which boundary tensor each stage pays for."""

import itertools
import math
import random

import pytest

from oracle import partition_oracle as po


def _linear_partition(t, p):
    """Smallest achievable largest-stage sum over p contiguous non-empty
    stages, by bisection over the candidate sums with a greedy test."""
    cands = sorted({sum(t[a:b]) for a in range(len(t)) for b in range(a + 1, len(t) + 1)})

    def fits(x):
        groups, cur = 1, 0.0
        for v in t:
            if v > x:
                return False
            if cur + v > x:
                groups, cur = groups + 1, v
            else:
                cur += v
        return groups <= p  # fewer groups can always be split further

    lo, hi = 0, len(cands) - 1
    while lo < hi:
        mid = (lo + hi) // 2
        if fits(cands[mid]):
            hi = mid
        else:
            lo = mid + 1
    return cands[lo]


def test_no_skips_is_the_linear_partition():
    rng = random.Random(3)
    for _ in range(60):
        n = rng.randint(2, 10)
        p = rng.choice([2, 4, 6])
        if p > n:
            continue
        t = [rng.choice([1, 2, 3, 5, 8]) for _ in range(n)]
        best, _ = po.optimum(n, p, t, [0.0] * n, [])
        assert best == _linear_partition(t, p)


@pytest.mark.parametrize("k,p", [(1, 2), (2, 2), (3, 2), (1, 4), (2, 4), (2, 6), (1, 8)])
def test_uniform_mirrored_model_splits_evenly(k, p):
    n = k * p
    skips = [(i, n - 1 - i) for i in range(n // 2)]
    best, args = po.optimum(n, p, [1.0] * n, [0.0] * n, skips)
    assert best == k
    assert tuple(range(k - 1, n - 1, k)) in args
    # a communication term adds the same lam * (t_lat + a / b) to every stage
    best2, _ = po.optimum(n, p, [1.0] * n, [6.0] * n, skips, lam=0.5, t_lat=1.0, b_inter=3.0)
    assert best2 == pytest.approx(k + 0.5 * (1.0 + 6.0 / 3.0))


def test_a_skip_forces_imbalance():
    # 8 unit ops, 4 stages: without skips 2 ops per stage; a skip from op 0
    # (always in stage 0) to op 3 puts op 3 into stage 3, so stages 0-2 hold
    # one op each and stage 3 holds ops 3..7
    best, args = po.optimum(8, 4, [1.0] * 8, [0.0] * 8, [])
    assert best == 2
    best, args = po.optimum(8, 4, [1.0] * 8, [0.0] * 8, [(0, 3)])
    assert best == 5 and args == [(0, 1, 2)]


def test_adjacent_skip_is_free_and_infeasible_case():
    # adjacent ops need no collocation
    assert po.optimum(4, 4, [1.0] * 4, [0.0] * 4, [(1, 2)])[0] == 1
    # op 2 would have to sit in stage 3, leaving only op 1 for stages 1 and 2
    best, args = po.optimum(4, 4, [1.0] * 4, [0.0] * 4, [(0, 2)])
    assert best == math.inf and args == []


def test_boundary_tensor_of_each_half():
    # zero work: the cost is the boundary each stage pays.  A cut after op k
    # makes stage 0 pay the output of op k and stage 1 pay the output of the
    # op before its first op, which is op k again.
    m_a = [5.0, 1.0, 7.0, 0.0]
    for k, want in ((0, 5.0), (1, 1.0), (2, 7.0)):
        assert po.cost(4, 2, (k,), [0.0] * 4, m_a, [], lam=1.0) == want
        assert po.stage_costs(4, 2, (k,), [0.0] * 4, m_a, 1.0, 0.0, 1.0) == [want, want]
    best, args = po.optimum(4, 2, [0.0] * 4, m_a, [], lam=1.0)
    assert best == 1.0 and args == [(1,)]
    # four stages: stages 0 and 1 pay their own outputs, stages 2 and 3 their inputs
    sc = po.stage_costs(6, 4, (0, 2, 3), [0.0] * 6, [1.0, 2.0, 3.0, 4.0, 5.0, 6.0],
                        1.0, 0.0, 1.0)
    assert sc == [1.0, 3.0, 3.0, 4.0]


def test_invariants():
    rng = random.Random(7)
    for _ in range(40):
        n = rng.randint(4, 9)
        p = rng.choice([2, 4])
        t = [rng.choice([1.0, 2.0, 4.0]) for _ in range(n)]
        skips = [(i, n - 1 - i) for i in range(n // 2) if rng.random() < 0.5]
        best, _ = po.optimum(n, p, t, [0.0] * n, skips)
        if best == math.inf:
            continue
        assert best >= max(t) and best >= sum(t) / p - 1e-12
        # more constraints never help
        extra = skips + [(0, n - 1)]
        assert po.optimum(n, p, t, [0.0] * n, extra)[0] >= best
        # scaling the times scales the optimum
        assert po.optimum(n, p, [2 * v for v in t], [0.0] * n, skips)[0] == 2 * best
        # every reported argmin is valid and reaches the optimum
        for cuts in po.optimum(n, p, t, [0.0] * n, skips)[1]:
            assert po.is_valid(n, p, cuts, skips)
            assert po.cost(n, p, cuts, t, [0.0] * n, skips) == best


@pytest.mark.parametrize("K,D", [(8, 4), (8, 2), (16, 4), (16, 8), (24, 4), (12, 2), (32, 8)])
def test_sequential_skip_volume_closed_form(K, D):
    """K blocks (K/2 encoder, K/2 decoder, block i's skip feeding block
    K-1-i), each producing `a` bytes, cut sequentially into D stages of K/D
    blocks: forward traffic ((K+4)D/4 - 1) a (Sec. II-C); the collocated
    placement of the same model over 2D stages on D devices sends only its
    2(D-1) boundaries (Sec. V-B)."""
    a = 3.0
    m_a = [a] * K
    skips = [(i, K - 1 - i) for i in range(K // 2)]
    seq = [K // D * (s + 1) - 1 for s in range(D - 1)]
    want = ((K + 4) * D / 4 - 1) * a
    assert po.comm_volume(K, m_a, skips, D, seq, collocated=False) == pytest.approx(want)
    if K % (2 * D) == 0:
        col = [K // (2 * D) * (s + 1) - 1 for s in range(2 * D - 1)]
        assert po.is_valid(K, 2 * D, col, skips)
        assert po.comm_volume(K, m_a, skips, 2 * D, col, collocated=True) == 2 * (D - 1) * a
