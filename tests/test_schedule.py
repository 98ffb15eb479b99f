"""Host logic of the profiler and the one-GPU stream packing (no GPU needed).

  * LPT list scheduling: every task on exactly one lane, lane loads are the
    sums of their tasks' costs, tasks are taken longest first, and on small
    random instances the makespan is within Graham's bound (4/3 - 1/(3L)) of
    the optimum found by brute force over all assignments;
  * plan(): the chosen lane count minimises max(load) * slowdown, lane counts
    whose largest tasks do not fit the memory budget are skipped, and an
    impossible budget is an error;
  * the epoch extrapolation is the mean step time times the steps per epoch;
  * sat_profile rejects a wrong struct_size and bad step counts before it
    touches the GPU.
"""

import ctypes as C
import itertools

import numpy as np
import pytest

from paper_2309_01226_amd import schedule


def _brute_opt(costs, L):
    best = float("inf")
    for a in itertools.product(range(L), repeat=len(costs)):
        loads = [0.0] * L
        for c, j in zip(costs, a):
            loads[j] += c
        best = min(best, max(loads))
    return best


def test_lpt_assignment_properties():
    costs = [5, 3, 3, 2, 2, 2, 1]
    lanes, loads = schedule.lpt_lanes(costs, 3)
    assert sorted(i for l in lanes for i in l) == list(range(len(costs)))
    for l, ld in zip(lanes, loads):
        assert ld == sum(costs[i] for i in l)
        assert [costs[i] for i in l] == sorted((costs[i] for i in l), reverse=True)
    assert lanes == [[0, 5], [1, 3, 6], [2, 4]]
    with pytest.raises(ValueError):
        schedule.lpt_lanes(costs, 0)


def test_lpt_within_graham_bound():
    rng = np.random.default_rng(0)
    for _ in range(40):
        n = int(rng.integers(1, 8))
        L = int(rng.integers(1, 4))
        costs = list(rng.uniform(0.1, 10.0, size=n))
        _, loads = schedule.lpt_lanes(costs, L)
        opt = _brute_opt(costs, L)
        assert max(loads) <= (4 / 3 - 1 / (3 * L)) * opt + 1e-9, (costs, L)
        assert max(loads) >= opt - 1e-9


def test_plan_chooses_minimum_and_respects_memory():
    costs = [4.0, 4.0, 4.0, 4.0]
    mem = [10, 10, 10, 10]
    # perfect overlap up to 2 lanes, none beyond
    p = schedule.plan(costs, mem, {1: 1.0, 2: 1.0, 4: 4.0})
    assert p["n_lanes"] == 2 and p["est_makespan"] == 8.0
    assert p["estimates"] == {1: 16.0, 2: 8.0, 4: 16.0}
    # two lanes no longer fit
    p = schedule.plan(costs, mem, {1: 1.0, 2: 1.0}, mem_budget=15)
    assert p["n_lanes"] == 1
    with pytest.raises(ValueError):
        schedule.plan(costs, mem, {2: 1.0}, mem_budget=15)


def test_epoch_extrapolation():
    assert schedule.estimate_epoch_ms({"step_ms_mean": 2.5}, 1000, 8) == 2.5 * 125
    assert schedule.estimate_epoch_ms({"step_ms_mean": 2.0}, 1001, 8) == 2.0 * 126


def test_sat_profile_rejects_bad_arguments():
    from paper_2309_01226_amd import _lib
    from paper_2309_01226_amd.model import make_config
    cfg = make_config("gpt2", 2, 64, 4, 256, 512, seq_len=32, batch=2)
    r = _lib.sat_profile_result()
    r.struct_size = 3
    st = _lib.lib().sat_profile(C.byref(cfg), None, 1, 2, 0, C.byref(r))
    assert st == _lib.SAT_EINVAL
    r.struct_size = C.sizeof(_lib.sat_profile_result)
    assert _lib.lib().sat_profile(C.byref(cfg), None, 1, 0, 0, C.byref(r)) == _lib.SAT_EINVAL
    assert _lib.lib().sat_profile(C.byref(cfg), None, -1, 2, 0, C.byref(r)) == _lib.SAT_EINVAL
    cfg.d_model = 65  # d % heads != 0
    assert _lib.lib().sat_profile(C.byref(cfg), None, 1, 2, 0, C.byref(r)) == _lib.SAT_EINVAL
