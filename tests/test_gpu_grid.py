"""A model-selection grid advanced concurrently on one GPU, one HIP stream per
model (the paper's set of tasks trained together: grid search over learning
rate x batch size, each member freezing its own bottom-k blocks).

A scaled-down grid of four GPT-2-style decoders shares one initial model (one
seed) and one stream of synthetic batches: every step draws rows for the
largest batch and the smaller-batch members use the leading rows.  All four
steps are enqueued before any is waited on, so the members' kernels interleave
on the device.  Checked per member against the float64 oracle on the same
inputs, and bitwise against the same member run alone on the default stream
(the kernels are deterministic and the members share no device state).
"""

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import flush, rel

pytestmark = pytest.mark.gpu

BASE = dict(arch="gpt2", n_layers=4, d_model=64, n_heads=4, d_mlp=256, vocab=512, seq_len=32)
LRS = (1e-3, 3e-3)
BATCHES = (2, 4)
STEPS = 2


def members():
    out = []
    for i, lr in enumerate(LRS):
        for j, b in enumerate(BATCHES):
            out.append(dict(BASE, lr=lr, batch=b, frozen_layers=2 if (i + j) % 2 else 0))
    return out


def oracle_cfg(kw):
    keys = ("arch", "n_layers", "d_model", "n_heads", "d_mlp", "vocab", "seq_len", "batch",
            "frozen_layers", "lr")
    return oracle.Config(**{k: kw[k] for k in keys})


def grid_batch(kw, step, seed=7):
    from paper_2309_01226_amd.inputs import decoder_batch
    return decoder_batch(kw["batch"], kw["seq_len"], kw["vocab"], seed=seed, step=step,
                         rows=max(BATCHES))


def run_members(kws, streams):
    """Advance every member STEPS steps; each step is enqueued for all members
    before any is synchronised.  Returns per member: losses after each step,
    grads of the last step, final params, initial params, and the params the
    last step started from."""
    from paper_2309_01226_amd.model import Model
    models = [Model(kw, stream=s) for kw, s in zip(kws, streams)]
    init = [m.params() for m in models]
    losses = [[] for _ in kws]
    before_last = None
    for step in range(STEPS):
        if step == STEPS - 1:
            before_last = [m.params() for m in models]
        batches = []
        for kw, s in zip(kws, streams):
            x, y = grid_batch(kw, step)
            with torch.cuda.stream(s):
                batches.append((torch.as_tensor(x).cuda(), torch.as_tensor(y).cuda()))
        torch.cuda.synchronize()
        for m, (x, y) in zip(models, batches):
            m.train_step(x, y, sync=False)
        for i, m in enumerate(models):
            losses[i].append(m.eval_loss(*batches[i]))
    torch.cuda.synchronize()
    out = [(losses[i], models[i].grads(), models[i].params(), init[i], before_last[i])
           for i in range(len(kws))]
    for m in models:
        m.close()
    return out


def test_grid_members_on_streams_match_oracle():
    kws = members()
    flush("grid: 4 members on 4 streams", [(k["lr"], k["batch"], k["frozen_layers"]) for k in kws])
    streams = [torch.cuda.Stream() for _ in kws]
    res = run_members(kws, streams)
    # one base model: every member starts from the same parameters
    for _, _, _, p0, _ in res[1:]:
        for n, v in p0.items():
            assert np.array_equal(v, res[0][3][n]), n
    for kw, (losses, G, P_gpu, P0, P_bl) in zip(kws, res):
        ocfg = oracle_cfg(kw)
        train = oracle.trainable_mask(ocfg)
        P = {n: v.astype(np.float64) for n, v in P0.items()}
        state = {}
        for step in range(STEPS):
            x, y = grid_batch(kw, step)
            _, og, P, state, _ = oracle.train_step(ocfg, P, state, x, y)
            # the loss after the step, on the same batch, from the updated parameters
            ol, _ = oracle.forward(ocfg, P, x, y)
            flush(f"member lr={kw['lr']} b={kw['batch']} k={kw['frozen_layers']} step {step}: "
                  f"gpu {losses[step]:.6f} oracle {ol:.6f}")
            assert abs(losses[step] - ol) / abs(ol) < 2e-2
        # last step's gradients against the oracle's at the same starting
        # parameters (the member's own, read back before that step), so that
        # the check measures one step's arithmetic, not trajectory drift
        x, y = grid_batch(kw, STEPS - 1)
        _, cache = oracle.forward(ocfg, {n: v.astype(np.float64) for n, v in P_bl.items()}, x, y)
        og = oracle.backward(ocfg, {n: v.astype(np.float64) for n, v in P_bl.items()}, cache)
        num = den = 0.0
        for n, g in G.items():
            if not train[n]:
                assert not g.any(), ("frozen grad written", n)
                assert np.array_equal(P_gpu[n], P0[n]), ("frozen param changed", n)
                continue
            assert rel(g, og[n]) < 3e-2, ("grad", n, rel(g, og[n]))
            num += float(np.sum((P_gpu[n] - P[n]) ** 2))
            den += float(np.sum(P[n] ** 2))
        assert np.sqrt(num / den) < 1e-2, ("global param error", np.sqrt(num / den))


def test_grid_streams_bitwise_equal_serial_runs():
    kws = members()
    flush("grid: concurrent vs one-at-a-time")
    conc = run_members(kws, [torch.cuda.Stream() for _ in kws])
    for i, kw in enumerate(kws):
        alone = run_members([kw], [torch.cuda.current_stream()])[0]
        assert alone[0] == conc[i][0], ("losses", i)
        for n in alone[1]:
            assert np.array_equal(alone[1][n], conc[i][1][n]), ("grad", i, n)
            assert np.array_equal(alone[2][n], conc[i][2][n]), ("param", i, n)
