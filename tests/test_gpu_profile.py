"""The profiler (sat_profile) and a stream-packed execution plan on the GPU.

  * a profile of the tiny decoder: consistent step statistics, the epoch time
    equal to the mean step time times ceil(samples / batch), the arena size
    and step FLOPs the model reports, a finite loss after the timed steps;
  * running three tasks packed onto two streams (LPT lanes) leaves every
    task's parameters and loss bitwise equal to running it alone;
  * the measured concurrency slowdown of two copies is a positive number;
  * against the float64 oracle: the profiling batch has the task's shape and
    ranges with next-token labels, the loss sat_profile reports after its
    steps is the oracle's after the same steps, and every task of a packed
    plan ends with the oracle's parameters and loss.
"""

import math


import numpy as np
import pytest
import torch

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


# ---------------------------------------------------------------- against the oracle

def _oracle_cfg(kw):
    from tests.test_gpu_step import oracle_cfg
    return oracle_cfg(kw)


def _oracle_run(kw, P0, batches):
    """The float64 oracle trained on the given host batches from P0."""
    import oracle
    ocfg = _oracle_cfg(kw)
    P = {n: v.astype(np.float64) for n, v in P0.items()}
    state = {}
    for xh, yh in batches:
        _, _, P, state, _ = oracle.train_step(ocfg, P, state, xh, yh)
    return ocfg, P


def _zero_init(n):
    return n.endswith(".b")


def _check_params(kw, got, ref, P0):
    import oracle
    from tests.gpu_util import rel
    train = oracle.trainable_mask(_oracle_cfg(kw))
    num = den = 0.0
    for n, p in got.items():
        if not train[n]:
            assert np.array_equal(p, P0[n]), ("frozen param changed", n)
            continue
        num += float(np.sum((p - ref[n]) ** 2))
        den += float(np.sum(ref[n] ** 2))
        if not _zero_init(n):
            assert rel(p, ref[n]) < 1e-2, ("param", n, rel(p, ref[n]))
    assert np.sqrt(num / den) < 1e-2, ("global param error", np.sqrt(num / den))


PROFILE_CASES = {
    "tiny_gpt2": TINY,
    "small_gptj_k1": dict(arch="gptj", n_layers=2, d_model=128, n_heads=2, d_mlp=256, vocab=97,
                          seq_len=40, batch=2, rotary_dim=16, lr=1e-3, frozen_layers=1),
    "small_vit": dict(arch="vit", n_layers=2, d_model=160, n_heads=2, d_mlp=320, vocab=10,
                      img_size=28, patch=14, channels=3, batch=4, lr=1e-3),
}


@pytest.mark.parametrize("name", list(PROFILE_CASES))
def test_profile_batch_and_final_loss_match_oracle(name):
    """The batch sat_profile trains on has the task's shape and value ranges
    (decoders: tokens in [0, V) with next-token labels), and the loss it
    reports after warmup + steps train steps on that batch is the oracle's
    loss after the same steps from the same initial parameters."""
    import oracle
    from paper_2309_01226_amd import schedule
    from paper_2309_01226_amd.model import Model
    kw = PROFILE_CASES[name]
    flush(f"profile batch + final loss vs oracle: {name}")
    x, y = schedule.profile_batch(kw)
    xh, yh = x.cpu().numpy(), y.cpu().numpy()
    V = kw["vocab"]
    assert yh.min() >= 0 and yh.max() < V
    if kw["arch"] == "vit":
        assert xh.shape == (kw["batch"], 3, kw["img_size"], kw["img_size"])
        assert xh.min() >= -1.0 and xh.max() < 1.0 and abs(float(xh.mean())) < 0.05
    else:
        assert xh.shape == yh.shape == (kw["batch"], kw["seq_len"])
        assert xh.min() >= 0 and xh.max() < V
        assert np.array_equal(yh[:, :-1], xh[:, 1:])          # labels are the next token
        assert len(np.unique(xh)) > min(V, xh.size) // 4       # not a constant stream
    x2, y2 = schedule.profile_batch(kw)
    assert torch.equal(x, x2) and torch.equal(y, y2)            # a function of the seed
    m = Model(kw)
    P0 = m.params()
    m.close()
    warm, steps = 2, 3
    r = schedule.profile(kw, warmup=warm, steps=steps)
    ocfg, P = _oracle_run(kw, P0, [(xh, yh)] * (warm + steps))
    ref = oracle.eval_loss(ocfg, P, xh, yh)
    flush(f"profile final loss {r['final_loss']:.6f} oracle {ref:.6f}")
    assert abs(r["final_loss"] - ref) / ref < 2e-2


def test_planned_tasks_match_oracle():
    """Every task of a two-lane packed plan (three tasks, one with a frozen
    block) ends where the oracle ends after the same steps on the same
    batch sequence: final parameters within the step tolerances and the
    final evaluation loss within 2e-2."""
    import oracle
    from paper_2309_01226_amd import schedule
    from paper_2309_01226_amd.inputs import batch_for
    from paper_2309_01226_amd.model import Model
    tasks = [(dict(TINY, lr=1e-3), 3), (dict(TINY, lr=3e-4, batch=4), 2),
             (dict(TINY, lr=1e-3, frozen_layers=1, n_layers=3), 4)]
    lanes, _ = schedule.lpt_lanes([n for _, n in tasks], 2)
    assert len(lanes) == 2 and all(lanes)
    out = schedule.run_plan(tasks, lanes, seed=3)
    for i, (kw, n) in enumerate(tasks):
        m = Model(kw)
        P0 = m.params()
        m.close()
        ocfg, P = _oracle_run(kw, P0, [batch_for(kw, seed=3, step=t) for t in range(n)])
        xh, yh = batch_for(kw, seed=3, step=0)
        ref = oracle.eval_loss(ocfg, P, xh, yh)
        loss, params = out[i]
        flush(f"task {i}: final loss {loss:.6f} oracle {ref:.6f}")
        assert abs(loss - ref) / ref < 2e-2
        _check_params(kw, params, P, P0)
