"""Tiny oracle configurations and helpers shared by the oracle pin tests."""

import numpy as np

from oracle import Config, param_spec

TINY = {
    "gpt2": dict(arch="gpt2", n_layers=2, d_model=16, n_heads=2, d_mlp=32, vocab=23,
                 seq_len=5, batch=2),
    "gptj": dict(arch="gptj", n_layers=2, d_model=16, n_heads=2, d_mlp=32, vocab=19,
                 seq_len=7, batch=2, rotary_dim=4),
    "vit": dict(arch="vit", n_layers=2, d_model=16, n_heads=2, d_mlp=32, vocab=10,
                img_size=8, patch=4, channels=3, batch=2),
}


def make_cfg(arch, **over):
    c = dict(TINY[arch])
    c.update(over)
    return Config(**c)


def rough_params(cfg, rng, scale=0.3):
    """Non-degenerate parameters: every tensor random (LN gains around 1), so
    that no term of the computation is hidden behind a zero or a one."""
    out = {}
    for name, shape, _ in param_spec(cfg):
        x = rng.normal(0.0, scale, size=shape)
        if name.endswith(".g"):
            x = 1.0 + x
        out[name] = x
    return out


def batch(cfg, rng):
    if cfg.arch == "vit":
        img = rng.standard_normal((cfg.batch, cfg.channels, cfg.img_size, cfg.img_size))
        lab = rng.integers(0, cfg.vocab, size=(cfg.batch,))
        return img, lab
    tok = rng.integers(0, cfg.vocab, size=(cfg.batch, cfg.seq_len + 1))
    return tok[:, :-1], tok[:, 1:]
