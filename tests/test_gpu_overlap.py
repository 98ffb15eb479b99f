"""The blocks' weight-gradient products on the library's second stream
(SAT_OPT_OVERLAP_WGRAD, the default) give bitwise the results of running
every launch on the model's stream: same kernels on the same operands, only
the order in which independent launches run differs.  Checked over several
steps on every architecture, with a frozen prefix, with activation
checkpointing, with split-K weight-gradient products (their own workspace on
the second stream), with the AdamW step fused into the products (the GPT-J
layer at full width: every block weight fused) and with it in the separate
pass, and with two models stepping on their own streams at once.  Step
parity against the oracle runs with the overlap on (tests/test_gpu_step.py
and the others use the default)."""

import numpy as np
import pytest
import torch

from tests.gpu_util import flush

pytestmark = pytest.mark.gpu

CASES = {
    "gpt2": dict(arch="gpt2", n_layers=3, d_model=64, n_heads=4, d_mlp=256, vocab=512,
                 seq_len=32, batch=2, lr=1e-3),
    "gptj": dict(arch="gptj", n_layers=3, d_model=128, n_heads=2, d_mlp=256, vocab=97,
                 seq_len=40, batch=2, rotary_dim=16, lr=1e-3),
    "vit": dict(arch="vit", n_layers=3, d_model=160, n_heads=2, d_mlp=320, vocab=10,
                img_size=28, patch=14, channels=3, batch=4, lr=1e-3),
    "gpt2_k1": dict(arch="gpt2", n_layers=4, d_model=64, n_heads=4, d_mlp=256, vocab=512,
                    seq_len=32, batch=2, lr=1e-3, frozen_layers=1),
    "gptj_ckpt": dict(arch="gptj", n_layers=3, d_model=128, n_heads=2, d_mlp=256, vocab=97,
                      seq_len=40, batch=2, rotary_dim=16, lr=1e-3, checkpoint=1),
    "gpt2_splitk": dict(arch="gpt2", n_layers=2, d_model=256, n_heads=4, d_mlp=1024, vocab=512,
                        seq_len=1024, batch=2, lr=1e-3),
    # every block weight's AdamW step fused into its weight-gradient product
    "gptj_fused": dict(arch="gptj", n_layers=2, d_model=2048, n_heads=8, d_mlp=8192, vocab=8200,
                       seq_len=2048, batch=2, rotary_dim=64, lr=1e-3),
}


def _pair(kw, extra=None):
    from paper_2309_01226_amd.model import Model
    a, b = Model(kw), Model(kw)
    a.set_option("overlap_wgrad", 1)
    b.set_option("overlap_wgrad", 0)
    for k, v in (extra or {}).items():
        a.set_option(k, v)
        b.set_option(k, v)
    return a, b


def _same(a, b, what):
    pa, pb = a.params(), b.params()
    for n in pa:
        assert np.array_equal(pa[n], pb[n]), (what, "param", n)
    sa, ta = a.state()
    sb, tb = b.state()
    assert ta == tb
    for n in sa:
        assert np.array_equal(sa[n][0], sb[n][0]) and np.array_equal(sa[n][1], sb[n][1]), (what, "state", n)


@pytest.mark.parametrize("name", list(CASES))
def test_overlap_bitwise_equal(name):
    from paper_2309_01226_amd.model import device_batch
    kw = CASES[name]
    flush(f"overlap vs serial: {name}")
    a, b = _pair(kw)
    for step in range(3):
        x, y = device_batch(kw, seed=5, step=step)
        la, lb = a.train_step(x, y), b.train_step(x, y)
        assert la == lb, (name, step, la, lb)
    _same(a, b, name)
    a.close()
    b.close()


@pytest.mark.parametrize("name", ["gptj", "gpt2_splitk"])
def test_overlap_gradients_and_separate_adamw(name):
    """Kept gradients (fused step) and the separate AdamW pass: gradients and
    parameters bitwise equal with and without the second stream."""
    from paper_2309_01226_amd.model import device_batch
    kw = CASES[name]
    for extra in ({"keep_grads": 1}, {"fused_adamw": 0}):
        flush(f"overlap vs serial: {name} {extra}")
        a, b = _pair(kw, extra)
        for step in range(2):
            x, y = device_batch(kw, seed=8, step=step)
            assert a.train_step(x, y) == b.train_step(x, y)
        ga, gb = a.grads(), b.grads()
        for n in ga:
            assert np.array_equal(ga[n], gb[n]), (name, extra, "grad", n)
        _same(a, b, name)
        a.close()
        b.close()


def test_overlap_two_models_on_their_own_streams():
    """Two models with second streams stepping at once (as the grid runs
    them) match their serial twins."""
    from paper_2309_01226_amd.model import Model, device_batch
    kws = [CASES["gptj"], dict(CASES["gpt2"], lr=3e-4)]
    streams = [torch.cuda.Stream() for _ in kws]
    conc = [Model(kw, stream=s) for kw, s in zip(kws, streams)]
    ser = [Model(kw) for kw in kws]
    for m in ser:
        m.set_option("overlap_wgrad", 0)
    for step in range(3):
        batches = [device_batch(kw, seed=2, step=step) for kw in kws]
        torch.cuda.synchronize()
        for m, (x, y) in zip(conc, batches):
            m.train_step(x, y, sync=False)
        torch.cuda.synchronize()
        for m, (x, y) in zip(ser, batches):
            m.train_step(x, y)
    for c, s in zip(conc, ser):
        _same(c, s, "two models")
        c.close()
        s.close()
