"""Pins of the schedule oracle (oracle/schedule_oracle.py): closed forms of
the minimum makespan, the symmetric placement's optimality among all
placements the constraints allow, and the checker flagging each constraint
of the scheduling formulation (Sec. V-A) on schedules with one planted
mistake."""

import copy

import pytest

from oracle import schedule_oracle as so


@pytest.mark.parametrize("M", [1, 2, 3, 5])
def test_one_device_runs_everything_serially(M):
    # D = 1: all 4 stages of every microbatch on device 0, one per step
    assert so.optimal_makespan(1, M) == 4 * M


@pytest.mark.parametrize("D", [1, 2, 3])
def test_one_microbatch_is_its_chain(D):
    # M = 1: the 4D stages of the chain run back to back
    assert so.optimal_makespan(D, 1) == 4 * D


@pytest.mark.parametrize("D,M", [(2, 2), (2, 3), (2, 4), (3, 2), (3, 3)])
def test_bounds(D, M):
    t = so.optimal_makespan(D, M)
    # every device holds 4 stages x M microbatches; the chain needs 4D steps
    assert t >= max(4 * M, 4 * D)
    # one microbatch after another is always feasible
    assert t <= 4 * D * M


def test_forward_turnaround_bound():
    """Device D-1 runs the forwards of partitions D-1 and D (stages D-1 and
    D).  Before stage D of the last microbatch it has run stage D-1 for all M
    microbatches and stage D for the M-1 before it (constraints (5), (6)),
    starting no earlier than step D-1; 3D-1 stages follow.  So every schedule
    takes at least 4D + 2M - 2 steps."""
    for D, M in [(1, 1), (1, 4), (2, 1), (2, 2), (2, 3), (2, 4), (3, 1), (3, 2), (3, 3)]:
        assert so.optimal_makespan(D, M) >= 4 * D + 2 * M - 2


@pytest.mark.parametrize("D,M", [(1, 2), (1, 4), (2, 1), (2, 2), (2, 3), (2, 4), (2, 5),
                                 (3, 1), (3, 2), (3, 3), (4, 2)])
def test_optimum_follows_the_wave_pattern(D, M):
    """The exhaustive optimum equals max(4D + 2M - 2, 4M + 2D - 2): the
    turnaround bound above while M <= D, and four steps per added
    microbatch, i.e. full devices in steady state, beyond it."""
    assert so.optimal_makespan(D, M) == max(4 * D + 2 * M - 2, 4 * M + 2 * D - 2)


def _greedy(D, M, dev=None):
    """A schedule built step by step (deepest runnable stage first) on the
    stage-to-device map `dev` (default: the symmetric placement)."""
    S = 4 * D
    dev = dev or so.symmetric_mapping(D)
    k = [0] * S
    done = {}
    table = [[] for _ in range(D)]
    t = 0
    while any(x < M for x in k):
        pick = {}
        for s in range(S - 1, -1, -1):
            if k[s] >= M:
                continue
            if s > 0 and not (k[s - 1] > k[s] and done[(s - 1, k[s])] <= t - 1):
                continue
            pick.setdefault(dev[s], s)
        for d in range(D):
            if d in pick:
                s = pick[d]
                table[d].append((s, k[s]))
                done[(s, k[s])] = t
            else:
                table[d].append(None)
        for s in pick.values():
            k[s] += 1
        t += 1
    return table


def _cells(table):
    return [(d, t) for d, row in enumerate(table) for t, c in enumerate(row) if c is not None]


def test_checker_accepts_a_valid_schedule():
    for D, M in [(1, 3), (2, 3), (3, 2)]:
        assert so.check(D, M, _greedy(D, M)) == []


def test_checker_flags_each_planted_mistake():
    D, M = 2, 3
    base = _greedy(D, M)
    assert so.check(D, M, base) == []
    # (1) a task dropped
    t = copy.deepcopy(base)
    d, i = _cells(t)[0]
    t[d][i] = None
    assert 1 in so.check(D, M, t)
    # (1) a task scheduled twice
    t = copy.deepcopy(base)
    d, i = _cells(t)[-1]
    t[d].append(t[d][i])
    assert 1 in so.check(D, M, t)
    # (3) one microbatch of a stage moved to the other device
    t = copy.deepcopy(base)
    (s, m) = t[0][0]
    t[0][0] = None
    t[1].append((s, m))
    for row in t:
        row += [None] * (max(len(r) for r in t) - len(row))
    assert 3 in so.check(D, M, t)
    # (4) a whole stage (all microbatches) moved away from its pair's device:
    # stage 3 (forward of partition 3, partner of partition 0) onto device 1
    dev = so.symmetric_mapping(D)
    dev[3] = 1
    t = _greedy(D, M, dev)
    assert so.check(D, M, t) == [4]
    # (5) stage 1 of microbatch 0 moved into the step that runs its stage 0
    # (device 1 is idle in step 0 of the base schedule)
    t = copy.deepcopy(base)
    assert t[0][0] == (0, 0) and t[1][0] is None
    d1, i1 = next((d, i) for d, row in enumerate(t) for i, c in enumerate(row) if c == (1, 0))
    t[d1][i1] = None
    t[1][0] = (1, 0)
    assert so.check(D, M, t) == [5]
    # (6) two microbatches of one stage in reverse order
    t = copy.deepcopy(base)
    cells = {c: (d, i) for d, row in enumerate(t) for i, c in enumerate(row) if c is not None}
    s = 4 * D - 1
    da, ia = cells[(s, 0)]
    db, ib = cells[(s, 1)]
    t[da][ia], t[db][ib] = (s, 1), (s, 0)
    assert 6 in so.check(D, M, t)
    # anchor: everything mirrored to the other device
    t = [base[1], base[0]]
    assert 0 in so.check(D, M, t)


def test_symmetric_placement_is_optimal():
    """The exhaustive optimum over every placement the constraints allow is
    reached with pair q on device q."""
    from collections import deque
    for D, M in [(2, 2), (2, 3), (3, 2)]:
        best_any = so.optimal_makespan(D, M)
        # restrict the oracle's search to the symmetric mapping
        S = 4 * D
        dev = so.symmetric_mapping(D)
        start, goal = tuple([0] * S), tuple([M] * S)
        seen, q = {start}, deque([(start, 0)])
        while q:
            k, depth = q.popleft()
            if k == goal:
                break
            run = {}
            for s in range(S):
                if k[s] < M and (s == 0 or k[s - 1] > k[s]):
                    run.setdefault(dev[s], []).append(s)
            from itertools import product
            for pick in product(*[[None] + v for v in run.values()]):
                if all(x is None for x in pick):
                    continue
                nk = list(k)
                for s in pick:
                    if s is not None:
                        nk[s] += 1
                nk = tuple(nk)
                if nk not in seen:
                    seen.add(nk)
                    q.append((nk, depth + 1))
        assert depth == best_any
