"""Seeded synthetic inputs shared by the tests, the bench and the oracle checks.

Holds none of the method's arithmetic: it only draws token ids, labels and
images.  Batch t of a run with seed s comes from numpy's generator seeded with
(s, t).  Decoders draw tokens [B, S+1] uniform in [0, V) and use the first S as
inputs and the last S as next-token labels; ViT and the ResNet draw N(0, 1)
images and uniform class labels.  These stand in for WikiText-2 and ImageNet (the paper's
datasets), whose contents are not used.
"""

import numpy as np


def decoder_batch(batch, seq_len, vocab, seed=0, step=0, rows=None):
    rng = np.random.default_rng((seed, step))
    n = batch if rows is None else rows
    tok = rng.integers(0, vocab, size=(n, seq_len + 1), dtype=np.int64).astype(np.int32)
    tok = tok[:batch]
    return np.ascontiguousarray(tok[:, :seq_len]), np.ascontiguousarray(tok[:, 1:])


def vit_batch(batch, img_size, n_classes, channels=3, seed=0, step=0):
    rng = np.random.default_rng((seed, step))
    img = rng.standard_normal((batch, channels, img_size, img_size), dtype=np.float32)
    lab = rng.integers(0, n_classes, size=(batch,), dtype=np.int64).astype(np.int32)
    return img, lab


def batch_for(cfg, seed=0, step=0, rows=None):
    """cfg: a dict or an object with the config fields."""
    g = (lambda k: cfg[k]) if isinstance(cfg, dict) else (lambda k: getattr(cfg, k))
    if g("arch") in ("vit", "resnet"):
        return vit_batch(g("batch"), g("img_size"), g("vocab"), g("channels"), seed, step)
    return decoder_batch(g("batch"), g("seq_len"), g("vocab"), seed, step, rows)
