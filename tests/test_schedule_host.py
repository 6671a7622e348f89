"""The library's schedule (pulse_sched_build / _check / _run_device) against
the schedule oracle, on the host: exact schedules reach the oracle's minimum
makespan, every built schedule passes the oracle's constraint check, the
library's checker agrees with the oracle's on valid and mutated tables, and
a device's row drives a dry-run stage through a legal microbatch order."""

import copy

import pytest

from oracle import schedule_oracle as so
from paper_2606_19163_amd import configs
from paper_2606_19163_amd import stage as S


@pytest.fixture(scope="module", autouse=True)
def built():
    import os
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_19163_amd import build
        build.build()
    yield


def _to_cells(table, M):
    return [[None if v < 0 else (v // M, v % M) for v in row] for row in table]


def _to_ints(cells, M):
    return [[-1 if c is None else c[0] * M + c[1] for c in row] for row in cells]


def _mask(bad):
    return sum(1 << k for k in bad)


EXACT = [(1, 1), (1, 3), (2, 1), (2, 2), (2, 3), (2, 4), (3, 1), (3, 2), (3, 3), (4, 2), (4, 3)]


@pytest.mark.parametrize("D,M", EXACT)
def test_exact_schedule_reaches_the_optimum(D, M):
    table, exact = S.sched_build(D, M)
    assert exact
    cells = _to_cells(table, M)
    assert so.check(D, M, cells) == []
    assert so.makespan(cells) == len(table[0]) == so.optimal_makespan(D, M)


@pytest.mark.parametrize("D,M", [(2, 16), (3, 12), (4, 4), (4, 16), (8, 32), (16, 8)])
def test_large_schedules_are_valid(D, M):
    table, exact = S.sched_build(D, M)
    cells = _to_cells(table, M)
    assert so.check(D, M, cells) == []
    T = len(table[0])
    assert max(4 * M, 4 * D) <= T <= 4 * D * M
    assert S.sched_check(D, M, table) == 0


def _wave_steps(D, M):
    return max(4 * D + 2 * M - 2, 4 * M + 2 * D - 2)


def test_large_schedules_reach_the_wave_pattern():
    """Beyond the exhaustive search the builder still reaches the step count
    of the exact optimum's pattern, max(4D + 2M - 2, 4M + 2D - 2), whose
    first term is a lower bound for every schedule."""
    for D in range(1, 9):
        for M in (1, 2, 3, 5, 7, 8, 12, 13, 16, 31, 32):
            table, _ = S.sched_build(D, M)
            assert len(table[0]) == _wave_steps(D, M), (D, M)
    for D, M in [(16, 64), (32, 96)]:
        table, _ = S.sched_build(D, M)
        assert len(table[0]) == _wave_steps(D, M)
        assert S.sched_check(D, M, table) == 0


def _peak(D, M, cells):
    """Microbatches between device d's encoder forward (stage d) and encoder
    backward (stage 4D-1-d), at most, from the oracle-format table."""
    out = []
    for d, row in enumerate(cells):
        cur = peak = 0
        for c in row:
            if c is None:
                continue
            if c[0] == d:
                cur += 1
                peak = max(peak, cur)
            if c[0] == 4 * D - 1 - d:
                cur -= 1
        out.append(peak)
    return out


@pytest.mark.parametrize("D,M", [(1, 3), (2, 3), (2, 8), (3, 4), (4, 4), (4, 16), (8, 32)])
def test_inflight(D, M):
    table, _ = S.sched_build(D, M)
    peak = S.sched_inflight(D, M, table)
    assert peak == _peak(D, M, _to_cells(table, M))
    if M % D == 0 and M > D:
        # backward-first order: device d holds 2D-1-d microbatches at most
        assert peak == [min(M, 2 * D - 1 - d) for d in range(D)]


def _mutations(D, M, cells):
    """(name, table) pairs, each with one change of the valid `cells`."""
    out = []
    flat = [(d, t) for d, row in enumerate(cells) for t, c in enumerate(row) if c is not None]
    t = copy.deepcopy(cells)
    d, i = flat[0]
    t[d][i] = None
    out.append(("drop", t))
    t = copy.deepcopy(cells)
    d, i = flat[-1]
    t[d].append(t[d][i])
    for r in t:
        r += [None] * (len(t[d]) - len(r))
    out.append(("duplicate", t))
    for d in range(len(cells)):
        for i in range(len(cells[d])):
            for j in range(i + 1, min(i + 4, len(cells[d]))):
                t = copy.deepcopy(cells)
                t[d][i], t[d][j] = t[d][j], t[d][i]
                out.append((f"swap {d} {i} {j}", t))
    if len(cells) > 1:
        out.append(("mirror", cells[::-1]))
        for d, i in flat[::3]:
            t = copy.deepcopy(cells)
            c = t[d][i]
            t[d][i] = None
            t[(d + 1) % len(cells)].append(c)
            w = max(len(r) for r in t)
            for r in t:
                r += [None] * (w - len(r))
            out.append((f"move {c}", t))
    return out


@pytest.mark.parametrize("D,M", [(1, 3), (2, 3), (3, 2)])
def test_checker_agrees_with_the_oracle(D, M):
    table, _ = S.sched_build(D, M)
    cells = _to_cells(table, M)
    assert S.sched_check(D, M, table) == 0
    muts = _mutations(D, M, cells)
    flagged = 0
    for name, t in muts:
        want = _mask(so.check(D, M, t))
        got = S.sched_check(D, M, _to_ints(t, M))
        assert got == want, (name, got, want)
        flagged += want != 0
    assert flagged > len(muts) // 2


def test_build_arguments():
    with pytest.raises(S.PulseError):
        S.sched_build(0, 4)
    with pytest.raises(S.PulseError):
        S.sched_build(2, 0)


@pytest.mark.parametrize("D,M", [(1, 3), (2, 3), (3, 4), (4, 6)])
def test_rows_drive_a_dry_stage(D, M):
    """Each device's row is a legal order for its stage: the stage's own
    microbatch state machine (encoder forward, decoder forward, decoder
    backward, encoder backward per microbatch, skips cached in between)
    accepts every call, and no microbatch is left in flight."""
    table, _ = S.sched_build(D, M)
    for d in range(D):
        desc = configs.l64()
        desc["max_inflight"] = M
        st = S.Stage(desc, dry_run=True)
        T = len(table[0])
        # one step at a time, as a runtime that exchanges between steps does
        for t in range(T):
            S.sched_run_device(st, D, d, M, table, t0=t, t1=t + 1)
        assert st.inflight() == 0
        st2 = S.Stage(desc, dry_run=True)
        S.sched_run_device(st2, D, d, M, table)
        assert st2.inflight() == 0


def test_run_device_rejects_foreign_cells_and_ranges():
    D, M = 2, 2
    table, _ = S.sched_build(D, M)
    desc = configs.l64()
    desc["max_inflight"] = M
    st = S.Stage(desc, dry_run=True)
    swapped = [table[1], table[0]]
    with pytest.raises(S.PulseError) as e:
        S.sched_run_device(st, D, 0, M, swapped)
    assert e.value.status == S.E_INVALID_ARG
    assert st.inflight() == 0  # nothing ran
    T = len(table[0])
    for t0, t1 in [(-1, 2), (3, 2), (0, T + 1)]:
        with pytest.raises(S.PulseError):
            S.sched_run_device(st, D, 0, M, table, t0=t0, t1=t1)
    with pytest.raises(S.PulseError):
        S.sched_run_device(st, D, 2, M, table)


def test_too_small_a_cache_is_reported():
    D, M = 2, 4
    table, _ = S.sched_build(D, M)
    st = S.Stage(configs.l64(), dry_run=True)  # max_inflight 1
    with pytest.raises(S.PulseError) as e:
        S.sched_run_device(st, D, 0, M, table)
    assert e.value.status == S.E_CACHE_FULL
