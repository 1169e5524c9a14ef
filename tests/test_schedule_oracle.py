"""Pins for the decode-loop scheduling oracle (oracle/schedule.py), CPU only.

The loop is greedy list scheduling of samples (jobs of o_i decode steps) on BS
batch slots (identical machines), so textbook facts about LPT fix its results
independently of the code: Graham's worst-case family (LPT makespan 4m - 1
against an optimum of 3m), the (4/3 - 1/(3m)) bound against brute-force optima
of small instances, and the trivial lower bounds. A hand-traced FIFO run pins
admission, refill order and the page stack.
"""
import itertools

import numpy as np
import pytest

from oracle import schedule as S


def graham_instance(m: int):
    """2m + 1 jobs: two each of 2m-1, 2m-2, ..., m+1 and three of m (Graham 1969)."""
    jobs = []
    for k in range(2 * m - 1, m, -1):
        jobs += [k, k]
    return jobs + [m, m, m]


def brute_force_opt(jobs, m):
    best = sum(jobs)
    for assign in itertools.product(range(m), repeat=len(jobs)):
        loads = [0] * m
        for j, a in zip(jobs, assign):
            loads[a] += j
        best = min(best, max(loads))
    return best


def run(jobs, m, order="lpt", est=None, prompt=None, S=S):
    n = len(jobs)
    prompt = prompt if prompt is not None else [0] * n
    blocks = max(-(-(p + o) // 16) for p, o in zip(prompt, jobs)) + 1
    return S.simulate(prompt, jobs, est if est is not None else jobs, m, m * blocks + 4, blocks, order)


# ----------------------------------------------------------------- pins
# Each pin takes the scheduling module, so test_schedule_mutants.py can run
# the same pins against deliberately broken copies.

def pin_graham_worst_case(S):
    for m in (2, 3, 4, 5, 6):
        jobs = graham_instance(m)
        assert run(jobs, m, S=S).makespan == 4 * m - 1, m
    for m in (2, 3):
        assert brute_force_opt(graham_instance(m), m) == 3 * m


def pin_lpt_bound_against_brute_force(S):
    rng = np.random.default_rng(1)
    worst = 0.0
    for _ in range(60):
        m = int(rng.integers(2, 4))
        jobs = [int(x) for x in rng.integers(1, 30, int(rng.integers(m + 1, 8)))]
        opt = brute_force_opt(jobs, m)
        lpt = run(jobs, m, S=S).makespan
        assert lpt <= (4 / 3 - 1 / (3 * m)) * opt + 1e-9, (jobs, m, lpt, opt)
        assert lpt >= opt
        worst = max(worst, lpt / opt)
    assert worst > 1.0   # some instance is not solved optimally, so the bound is exercised


def pin_lower_bounds_and_list_scheduling_form(S):
    rng = np.random.default_rng(2)
    for order in ("lpt", "fifo"):
        for _ in range(40):
            m = int(rng.integers(1, 9))
            jobs = [int(x) for x in np.exp(rng.uniform(0, 6, int(rng.integers(1, 40))))]
            sch = run(jobs, m, order, S=S)
            assert sch.makespan >= max(-(-sum(jobs) // m), max(jobs))
            assert sch.makespan == S.makespan_of_list_schedule(jobs, m, S.admission_order(jobs, order))
            for i, o in enumerate(jobs):
                assert sch.finish_step[i] - sch.admit_step[i] + 1 == o
            for b in range(m):
                spans = sorted((sch.admit_step[i], sch.finish_step[i]) for i in range(len(jobs)) if sch.slot[i] == b)
                assert all(x[1] < y[0] for x, y in zip(spans, spans[1:]))


def pin_estimates_order_true_lengths_time(S):
    jobs = [5, 1, 9, 2]
    est = [1, 9, 2, 5]                    # order by estimate: 1, 3, 2, 0
    sch = run(jobs, 1, "lpt", est=est, S=S)
    assert sch.admit_step == [1 + 2 + 9, 0, 1 + 2, 1]
    assert sch.makespan == sum(jobs)
    # equal estimates keep index order: true lengths 1, 5, 9 run in that order
    sch = run([1, 5, 9], 1, "lpt", est=[4, 4, 4], S=S)
    assert sch.admit_step == [0, 1, 6]


def pin_fifo_hand_trace(S):
    sch = S.simulate([0, 16, 5], [3, 1, 2], [3, 1, 2], 2, 8, 4, "fifo", checkpoints=(0, 1, 2))
    assert sch.makespan == 3
    assert sch.slot == [0, 1, 1]
    assert sch.admit_step == [0, 0, 1]
    assert sch.finish_step == [2, 0, 2]
    lens0, tab0 = sch.checkpoints[0]
    assert lens0 == [1, 17] and tab0[0][0] == 1 and tab0[1][:2] == [0, 2]
    lens1, tab1 = sch.checkpoints[1]
    assert lens1 == [2, 6] and tab1[0][0] == 1 and tab1[1][0] == 0
    lens2, _ = sch.checkpoints[2]
    assert lens2 == [3, 7]


def pin_pages_never_shared(S):
    rng = np.random.default_rng(3)
    M, BS = 50, 6
    prompt = [int(x) for x in rng.integers(0, 70, M)]
    out = [int(x) for x in rng.integers(1, 90, M)]
    blocks = max(-(-(p + o) // 16) for p, o in zip(prompt, out))
    N = BS * blocks
    sch = S.simulate(prompt, out, out, BS, N, blocks, "lpt", checkpoints=list(range(0, 2000, 7)))
    for st, (lens, table) in sch.checkpoints.items():
        used = [table[b][k] for b in range(BS) for k in range(-(-lens[b] // 16))]
        assert len(used) == len(set(used)), f"page shared at step {st}"
        assert all(0 <= p < N for p in used)


ALL_PINS = [pin_graham_worst_case, pin_lpt_bound_against_brute_force, pin_lower_bounds_and_list_scheduling_form,
            pin_estimates_order_true_lengths_time, pin_fifo_hand_trace, pin_pages_never_shared]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(S)



