"""Runtime estimates and one-GPU stream packing for a set of fine-tuning tasks.

The paper's Trial Runner (Sec. 3.2) profiles every task for a few minibatches
and extrapolates its runtime; its optimizer then decides how tasks share the
hardware so that the whole set finishes soonest (Sec. 4).  On one GPU the
sharing decision is how many tasks run at once, each on its own HIP stream,
and which tasks follow each other on a stream.  This module holds that host
logic:

  profile(kw)              sat_profile: mean step time of a task (and its epoch
                           time extrapolated from it), measured by the library
  profile_batch(kw)        the synthetic batch sat_profile trains on
  measure_slowdown(kw, L)  step time of one task when L copies of it run at
                           once on L streams, relative to running alone
  lpt_lanes(costs, L)      longest-processing-time-first list scheduling of
                           tasks onto L lanes (a textbook makespan heuristic:
                           within 4/3 of optimal for identical lanes)
  plan(...)                the lane count and assignment with the smallest
                           estimated makespan that fits the memory budget
  run_plan(...)            executes a plan: every lane on its own stream, its
                           tasks back to back, lanes advanced round-robin

Every step runs in libsaturn.so; this module only orders work.
"""

import ctypes as C
import math

from . import _lib
from .inputs import batch_for
from .model import Model, make_config


def profile(cfg_kwargs, warmup=2, steps=5, samples_per_epoch=0, stream=None):
    """Trial-Runner estimate of one task (sat_profile), as a dict."""
    import torch
    cfg = make_config(**cfg_kwargs)
    r = _lib.sat_profile_result()
    r.struct_size = C.sizeof(_lib.sat_profile_result)
    st = stream if stream is not None else torch.cuda.current_stream()
    _lib.call("sat_profile", C.byref(cfg), C.c_void_p(st.cuda_stream), int(warmup), int(steps),
              int(samples_per_epoch), C.byref(r))
    return {k: getattr(r, k) for k, _ in r._fields_ if k != "struct_size"}


def profile_batch(cfg_kwargs, stream=None):
    """The synthetic batch sat_profile trains on (sat_profile_batch), as
    device tensors (inputs, labels)."""
    import torch
    cfg = make_config(**cfg_kwargs)
    B = cfg_kwargs["batch"]
    if cfg_kwargs["arch"] == "vit":
        c, i = cfg_kwargs.get("channels", 3), cfg_kwargs["img_size"]
        x = torch.empty(B, c, i, i, device="cuda", dtype=torch.float32)
        y = torch.empty(B, device="cuda", dtype=torch.int32)
    else:
        x = torch.empty(B, cfg_kwargs["seq_len"], device="cuda", dtype=torch.int32)
        y = torch.empty_like(x)
    st = stream if stream is not None else torch.cuda.current_stream()
    _lib.call("sat_profile_batch", C.byref(cfg), C.c_void_p(x.data_ptr()), C.c_void_p(y.data_ptr()),
              C.c_void_p(st.cuda_stream))
    st.synchronize()
    return x, y


def measure_slowdown(cfg_kwargs, n_lanes, steps=5, warmup=2, seed=0):
    """Mean step time of L concurrent copies of a task (one stream each), over
    its step time alone: 1 means the copies overlap perfectly, L that they
    serialise."""
    import torch

    def run(L):
        streams = [torch.cuda.Stream() for _ in range(L)]
        models = [Model(cfg_kwargs, stream=s) for s in streams]
        x, y = batch_for(cfg_kwargs, seed=seed, step=0)
        xd, yd = torch.as_tensor(x).cuda(), torch.as_tensor(y).cuda()
        torch.cuda.synchronize()
        for _ in range(warmup):
            for m in models:
                m.train_step(xd, yd, sync=False)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for s in streams:
            s.wait_event(e0)
        for _ in range(steps):
            for m in models:
                m.train_step(xd, yd, sync=False)
        for s in streams:
            ev = torch.cuda.Event()
            ev.record(s)
            torch.cuda.current_stream().wait_event(ev)
        e1.record()
        torch.cuda.synchronize()
        for m in models:
            m.close()
        return e0.elapsed_time(e1) / steps  # ms per round of L steps

    solo = run(1)
    return {L: run(L) / solo for L in n_lanes}


def lpt_lanes(costs, n_lanes):
    """Assign tasks (costs[i] = its total run time) to n_lanes lanes, longest
    first, each to the currently least-loaded lane (lowest index on ties).
    Returns (lanes, loads): lanes[j] = task indices in execution order."""
    if n_lanes < 1:
        raise ValueError("n_lanes must be >= 1")
    lanes = [[] for _ in range(n_lanes)]
    loads = [0.0] * n_lanes
    for i in sorted(range(len(costs)), key=lambda i: (-costs[i], i)):
        j = min(range(n_lanes), key=lambda j: (loads[j], j))
        lanes[j].append(i)
        loads[j] += costs[i]
    return lanes, loads


def plan(costs, arena_bytes, slowdown, mem_budget=None):
    """Choose the lane count L (a key of `slowdown`) and an LPT assignment
    minimising the estimated makespan max(lane load) * slowdown[L], where
    every task's cost is its solo run time and running L lanes at once
    stretches each step by slowdown[L].  Plans whose L largest tasks would not
    fit in mem_budget bytes at once are skipped.  Returns a dict with
    n_lanes, lanes, est_makespan and the estimate of every candidate."""
    best = None
    est = {}
    order = sorted(arena_bytes, reverse=True)
    for L in sorted(slowdown):
        if L > max(len(costs), 1):
            continue
        if mem_budget is not None and sum(order[:L]) > mem_budget:
            continue
        lanes, loads = lpt_lanes(costs, L)
        est[L] = max(loads) * slowdown[L]
        if best is None or est[L] < best["est_makespan"] - 1e-12:
            best = {"n_lanes": L, "lanes": lanes, "est_makespan": est[L]}
    if best is None:
        raise ValueError("no lane count fits the memory budget")
    best["estimates"] = est
    return best


def run_plan(tasks, lanes, seed=0, keep_params=True):
    """Execute a plan.  tasks[i] = (cfg_kwargs, n_steps); lanes from plan() /
    lpt_lanes().  Every lane has its own stream and at most one model alive;
    task i's step t trains on batch_for(cfg, seed, t).  Returns
    {task index: (final loss, parameters or None)}."""
    import torch
    streams = [torch.cuda.Stream() for _ in lanes]
    pos = [0] * len(lanes)          # next task of each lane
    cur = [None] * len(lanes)       # (task index, model, steps done)
    out = {}

    def start(j):
        while pos[j] < len(lanes[j]):
            i = lanes[j][pos[j]]
            pos[j] += 1
            if tasks[i][1] > 0:
                cur[j] = (i, Model(tasks[i][0], stream=streams[j]), 0)
                return
            m = Model(tasks[i][0], stream=streams[j])
            out[i] = (float("nan"), m.params() if keep_params else None)
            m.close()
        cur[j] = None

    def finish(j):
        i, m, _ = cur[j]
        x, y = batch_for(tasks[i][0], seed=seed, step=0)
        loss = m.eval_loss(torch.as_tensor(x).cuda(), torch.as_tensor(y).cuda())
        out[i] = (loss, m.params() if keep_params else None)
        m.close()
        start(j)

    for j in range(len(lanes)):
        start(j)
    while any(c is not None for c in cur):
        for j, c in enumerate(cur):
            if c is None:
                continue
            i, m, t = c
            x, y = batch_for(tasks[i][0], seed=seed, step=t)
            with torch.cuda.stream(streams[j]):
                xd, yd = torch.as_tensor(x).cuda(non_blocking=False), torch.as_tensor(y).cuda()
            m.train_step(xd, yd, sync=False)
            cur[j] = (i, m, t + 1)
            if t + 1 == tasks[i][1]:
                streams[j].synchronize()
                finish(j)
    torch.cuda.synchronize()
    return out


def estimate_epoch_ms(profile_result, samples_per_epoch, batch):
    """Epoch time from a profile's mean step time (the Trial Runner's
    extrapolation), for a dataset size other than the one profiled."""
    return profile_result["step_ms_mean"] * math.ceil(samples_per_epoch / batch)
