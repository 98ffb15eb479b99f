"""The profiler (sat_profile) and a stream-packed execution plan on the GPU.

  * a profile of the tiny decoder: consistent step statistics, the epoch time
    equal to the mean step time times ceil(samples / batch), the arena size
    and step FLOPs the model reports, a finite loss after the timed steps;
  * running three tasks packed onto two streams (LPT lanes) leaves every
    task's parameters and loss bitwise equal to running it alone;
  * the measured concurrency slowdown of two copies is a positive number.
"""

import math

import numpy as np
import pytest

from tests.gpu_util import flush

pytestmark = pytest.mark.gpu

TINY = dict(arch="gpt2", n_layers=2, d_model=64, n_heads=4, d_mlp=256, vocab=512, seq_len=32,
            batch=2, lr=1e-3)


def test_profile_tiny():
    from paper_2309_01226_amd import schedule
    from paper_2309_01226_amd.model import Model, arena_bytes, make_config
    r = schedule.profile(TINY, warmup=2, steps=6, samples_per_epoch=1001)
    flush(r)
    assert r["steps"] == 6
    assert 0 < r["step_ms_min"] <= r["step_ms_mean"] <= r["step_ms_max"]
    assert r["steps_per_epoch"] == math.ceil(1001 / TINY["batch"])
    assert r["epoch_ms"] == pytest.approx(r["step_ms_mean"] * r["steps_per_epoch"], rel=1e-12)
    assert r["arena_bytes"] == arena_bytes(make_config(**TINY))
    m = Model(TINY)
    assert r["step_tflop"] == pytest.approx(m.stats()[2] / 1e12, rel=1e-12)
    m.close()
    assert r["tokens_per_s"] == pytest.approx(TINY["batch"] * TINY["seq_len"] / (r["step_ms_mean"] * 1e-3))
    assert math.isfinite(r["final_loss"]) and r["final_loss"] < math.log(TINY["vocab"]) + 1.0
    r0 = schedule.profile(TINY, warmup=0, steps=1)
    assert r0["steps_per_epoch"] == 0 and r0["epoch_ms"] == 0.0


def test_packed_plan_equals_solo_runs():
    from paper_2309_01226_amd import schedule
    tasks = [(dict(TINY, lr=1e-3), 3), (dict(TINY, lr=3e-4, batch=4), 2),
             (dict(TINY, lr=1e-3, frozen_layers=1, n_layers=3), 4)]
    lanes, _ = schedule.lpt_lanes([n for _, n in tasks], 2)
    packed = schedule.run_plan(tasks, lanes, seed=3)
    solo = schedule.run_plan(tasks, [[0, 1, 2]], seed=3)
    for i in range(len(tasks)):
        assert packed[i][0] == solo[i][0], i
        for n in solo[i][1]:
            assert np.array_equal(packed[i][1][n], solo[i][1][n]), (i, n)


def test_slowdown_positive():
    from paper_2309_01226_amd import schedule
    s = schedule.measure_slowdown(TINY, [1, 2], steps=3)
    flush(s)
    assert s[1] > 0 and s[2] > 0
