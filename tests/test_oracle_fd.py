"""Pin the oracle's hand-written backward to its forward by central finite
differences in float64 (brute force on tiny inputs)."""

import numpy as np
import pytest

from oracle import backward, forward, trainable_mask
from tests.oracle_cases import batch, make_cfg, rough_params


def _loss(cfg, P, x, y):
    return forward(cfg, P, x, y)[0]


@pytest.mark.parametrize("arch", ["gpt2", "gptj", "vit"])
@pytest.mark.parametrize("k", [0, 1])
def test_finite_differences(arch, k):
    cfg = make_cfg(arch, frozen_layers=k)
    rng = np.random.default_rng(1234 + k)
    P = rough_params(cfg, rng)
    x, y = batch(cfg, rng)
    if cfg.arch != "vit":
        y = y.copy()
        y[0, 1] = -1  # one ignored label exercises the valid-count divisor
    _, cache = forward(cfg, P, x, y)
    G = backward(cfg, P, cache)
    train = trainable_mask(cfg)
    assert set(G) == {n for n, t in train.items() if t}
    for name in G:
        flat = P[name].reshape(-1)
        idx = rng.choice(flat.size, size=min(16, flat.size), replace=False)
        fd = []
        for i in idx:
            old = flat[i]
            h = 1e-6 * max(1.0, abs(old))
            flat[i] = old + h
            lp = _loss(cfg, P, x, y)
            flat[i] = old - h
            lm = _loss(cfg, P, x, y)
            flat[i] = old
            fd.append((lp - lm) / (2 * h))
        fd = np.array(fd)
        an = G[name].reshape(-1)[idx]
        err = np.linalg.norm(an - fd) / max(np.linalg.norm(fd), 1e-8)
        assert err < 1e-6, (name, err)


@pytest.mark.parametrize("arch", ["gpt2", "gptj", "vit"])
def test_frozen_grads_match_full_backward(arch):
    """Grads of blocks >= k are the same numbers with k = 1 as with k = 0."""
    rng = np.random.default_rng(7)
    cfg0 = make_cfg(arch, frozen_layers=0)
    cfg1 = make_cfg(arch, frozen_layers=1)
    P = rough_params(cfg0, rng)
    x, y = batch(cfg0, rng)
    l0, c0 = forward(cfg0, P, x, y)
    l1, c1 = forward(cfg1, P, x, y)
    assert l0 == l1  # forward does not depend on k
    G0 = backward(cfg0, P, c0)
    G1 = backward(cfg1, P, c1)
    for n, g in G1.items():
        assert np.array_equal(g, G0[n]), n
    frozen = [n for n in G0 if n not in G1]
    assert any(n.startswith("h0.") for n in frozen)
    assert all(not n.startswith("h1.") for n in frozen)
