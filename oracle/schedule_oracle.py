"""CPU oracle for the collocated pipeline schedule (plain Python, exhaustive).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` may import this module; the
library's scheduler (C++, ``pulse_sched_*``) shares no code with it.

What is modelled (Sec. V-A)
---------------------------
A model cut into P = 2D partitions runs on D devices.  Partition p and its
skip partner P-1-p are collocated (Sec. IV-B), and every partition's forward
and backward run where its weights live.  The schedule assigns unit-time
stages of M microbatches to (device, step) cells.  One microbatch is the
chain of S = 2P stages

    s = 0 .. P-1      : forward of partition s
    s = P .. 2P-1     : backward of partition 2P-1-s

(forward through the partitions, then backward in reverse).  The six
constraints of the scheduling formulation are checked as written there:

    (1) every (stage, microbatch) is scheduled exactly once;
    (2) a device runs at most one stage per step;
    (3) every stage stays on one device for all microbatches;
    (4) collocated stages share a device -- here the forward and backward of
        a partition and of its skip partner;
    (5) stage s+1 of a microbatch runs at least one step after stage s;
    (6) a stage processes microbatch m+1 no earlier than microbatch m;

plus the anchor of the first stage on device 0.  The objective is the last
occupied step T_max (makespan T_max + 1).

Readings (the paper leaves them open): the formulation's S stages, which
cover forward and backward passes, are the 2P forward/backward stages above; a
partition's forward and backward are collocated (its weights and saved
activations live on one device); stages take one step each.
"""

from __future__ import annotations

from collections import deque
from itertools import product


def stages(D):
    """[(kind, partition)] for s = 0 .. 4D-1."""
    P = 2 * D
    return [("F", s) if s < P else ("B", 2 * P - 1 - s) for s in range(2 * P)]


def partition_of(D, s):
    return stages(D)[s][1]


def pair_of(D, p):
    """Index of the collocated pair {p, 2D-1-p}."""
    return min(p, 2 * D - 1 - p)


def check(D, M, table):
    """Violated constraints of a schedule, as a sorted list of numbers
    (1-6, and 0 for the anchor); empty when the schedule is valid.

    table[d][t] is (s, m) or None."""
    S = 4 * D
    where = {}
    bad = set()
    for d, row in enumerate(table):
        for t, cell in enumerate(row):
            if cell is None:
                continue
            s, m = cell
            if not (0 <= s < S and 0 <= m < M):
                bad.add(1)
                continue
            if (s, m) in where:
                bad.add(1)
            where[(s, m)] = (d, t)
    if len(where) != S * M:
        bad.add(1)
    # (2) holds by construction: one cell per (device, step)
    dev = {}
    for (s, m), (d, t) in where.items():
        dev.setdefault(s, set()).add(d)
    for s, ds in dev.items():
        if len(ds) > 1:
            bad.add(3)
    if 3 not in bad:
        one = {s: next(iter(ds)) for s, ds in dev.items()}
        for s in range(S):
            for s2 in range(S):
                if s in one and s2 in one and \
                        pair_of(D, partition_of(D, s)) == pair_of(D, partition_of(D, s2)) and \
                        one[s] != one[s2]:
                    bad.add(4)
        if 0 in one and one[0] != 0:
            bad.add(0)
    for m in range(M):
        for s in range(S - 1):
            if (s, m) in where and (s + 1, m) in where and \
                    where[(s + 1, m)][1] < where[(s, m)][1] + 1:
                bad.add(5)
    for s in range(S):
        for m in range(M - 1):
            if (s, m) in where and (s, m + 1) in where and \
                    where[(s, m + 1)][1] < where[(s, m)][1]:
                bad.add(6)
    return sorted(bad)


def makespan(table):
    last = -1
    for row in table:
        for t, cell in enumerate(row):
            if cell is not None:
                last = max(last, t)
    return last + 1


def optimal_makespan(D, M):
    """Exact minimum makespan over every device mapping allowed by (3), (4)
    and the anchor, by breadth-first search over the schedule's progress.

    With (6) a stage finishes its microbatches in order, so after any step
    the progress is the vector k[s] of microbatches stage s has finished;
    (5) makes (s, k[s]) runnable when k[s-1] > k[s].  A step advances any set
    of runnable stages on distinct devices by one.  The BFS depth at which
    k = (M, .., M) is first reached is the minimum makespan for that
    mapping."""
    S = 4 * D
    P = 2 * D
    best = None
    for mapping in product(range(D), repeat=D):  # device of each pair
        if mapping[0] != 0:  # the anchor: stage 0 (pair 0) on device 0
            continue
        dev = [mapping[pair_of(D, partition_of(D, s))] for s in range(S)]
        start = tuple([0] * S)
        goal = tuple([M] * S)
        seen = {start}
        frontier = deque([(start, 0)])
        found = None
        while frontier:
            k, depth = frontier.popleft()
            if k == goal:
                found = depth
                break
            runnable = [s for s in range(S)
                        if k[s] < M and (s == 0 or k[s - 1] > k[s])]
            by_dev = {}
            for s in runnable:
                by_dev.setdefault(dev[s], []).append(s)
            choices = [[None] + ss for ss in by_dev.values()]
            for pick in product(*choices):
                if all(x is None for x in pick):
                    continue
                nk = list(k)
                for s in pick:
                    if s is not None:
                        nk[s] += 1
                nk = tuple(nk)
                if nk not in seen:
                    seen.add(nk)
                    frontier.append((nk, depth + 1))
        if found is not None and (best is None or found < best):
            best = found
    return best


def symmetric_mapping(D):
    """Device of each stage under the symmetric placement: pair q on
    device q."""
    return [pair_of(D, partition_of(D, s)) for s in range(4 * D)]
