"""Activation checkpointing (sat_config.checkpoint): the backward of each block
rebuilds the block's saved activations from its input with the same kernels
on the same values, so a checkpointed model must train bitwise like one that
kept every block's activations: equal losses, gradients, parameters and
optimizer state after every step, for each architecture and with frozen
layers; and its arena must be smaller by all but one block's activation set.
The checkpointed step is also held against the float64 oracle directly, with
the same three-step parity run as the step tests.
"""

import numpy as np
import pytest

from tests.gpu_util import flush

pytestmark = pytest.mark.gpu

CASES = {
    "gpt2": dict(arch="gpt2", n_layers=3, d_model=64, n_heads=4, d_mlp=256, vocab=512, seq_len=32,
                 batch=2, lr=1e-3),
    "gptj": dict(arch="gptj", n_layers=3, d_model=128, n_heads=2, d_mlp=256, vocab=97, seq_len=40,
                 batch=2, rotary_dim=16, lr=1e-3),
    "vit": dict(arch="vit", n_layers=2, d_model=160, n_heads=2, d_mlp=320, vocab=10, img_size=28,
                patch=14, channels=3, batch=4, lr=1e-3),
    "gptj_k1": dict(arch="gptj", n_layers=3, d_model=128, n_heads=2, d_mlp=256, vocab=97, seq_len=40,
                    batch=2, rotary_dim=16, lr=1e-3, frozen_layers=1),
    "gptj_1024": dict(arch="gptj", n_layers=2, d_model=1024, n_heads=4, d_mlp=4096, vocab=1024,
                      seq_len=256, batch=2, rotary_dim=64, lr=1e-4),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_checkpoint_bitwise(name):
    from paper_2309_01226_amd.model import Model, arena_bytes, device_batch, make_config
    kw = CASES[name]
    a, b = Model(kw), Model(dict(kw, checkpoint=1))
    for step in range(2):
        x, y = device_batch(kw, seed=5, step=step)
        la, lb = a.train_step(x, y), b.train_step(x, y)
        flush(f"{name} step {step}: {la!r} {lb!r}")
        assert la == lb
        Ga, Gb = a.grads(), b.grads()
        for n in Ga:
            assert np.array_equal(Ga[n], Gb[n]), ("grad", n)
    Pa, Pb = a.params(), b.params()
    Sa, _ = a.state()
    Sb, _ = b.state()
    for n in Pa:
        assert np.array_equal(Pa[n], Pb[n]), ("param", n)
        assert np.array_equal(Sa[n][0], Sb[n][0]) and np.array_equal(Sa[n][1], Sb[n][1]), ("state", n)
    k = kw.get("frozen_layers", 0)
    sets = kw["n_layers"] - k + (1 if k > 0 else 0)
    full, ck = arena_bytes(make_config(**kw)), arena_bytes(make_config(**dict(kw, checkpoint=1)))
    assert ck < full or sets == 1
    a.close()
    b.close()


ORACLE_CASES = ["tiny_gpt2", "small_gptj", "small_vit", "small_gptj_k1"]


@pytest.mark.parametrize("name", ORACLE_CASES)
def test_checkpoint_oracle_parity(name):
    """With checkpointing on, the three-step parity run against the float64
    oracle (loss, activations, logits, gradients, exact AdamW, parameters,
    frozen tensors) holds as it does without it."""
    from tests.test_gpu_step import CASES as STEP_CASES, run_parity
    flush(f"checkpointed step parity case {name}")
    run_parity(dict(STEP_CASES[name], checkpoint=1))
