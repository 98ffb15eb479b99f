"""Pins of the float64 ResNet oracle (oracle/resnet.py) against things other
than itself:

  * structure: the parameter counts of the standard ResNet-50 and ResNet-152
    (25,557,032 and 60,192,808 with batch-norm gains and shifts and the
    classifier bias), golden values in tests/golden/resnet_params.txt;
  * torch's CPU float64 convolution, batch norm, max pool, linear layer and
    cross-entropy with autograd, on a small network with both kinds of
    shortcut: loss, logits and every gradient;
  * central finite differences of the whole loss on a tiny network, with and
    without a frozen prefix;
  * closed forms: a convolution of a one-pixel image reproduces the weights,
    batch norm gives zero-mean unit-variance channels, max pooling of a
    constant map is that constant and passes the gradient to the first
    position of each window.
"""

import math
import os

import numpy as np
import pytest

from oracle import resnet as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "resnet_params.txt")


def _golden():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, blocks, width, classes, n = line.split()
        out[name] = (tuple(int(b) for b in blocks.split(",")), int(width), int(classes), int(n))
    return out


def _count(cfg):
    return sum(int(np.prod(s)) for _, s, _ in R.param_spec(cfg))


@pytest.mark.parametrize("name", ["resnet50", "resnet152"])
def test_parameter_count_matches_published(name):
    blocks, width, classes, n = _golden()[name]
    assert _count(R.ResNetConfig(blocks=blocks, width=width, classes=classes)) == n


def test_workload_size_is_about_200m():
    n = _count(R.ResNetConfig())
    assert 180e6 < n < 260e6, n


def _small(**kw):
    base = dict(blocks=(2, 1, 1, 1), width=4, classes=7, img_size=32, channels=3, batch=3)
    base.update(kw)
    return R.ResNetConfig(**base)


def _batch(cfg, rng):
    x = rng.normal(size=(cfg.batch, cfg.channels, cfg.img_size, cfg.img_size))
    y = rng.integers(0, cfg.classes, size=cfg.batch)
    return x, y


def _rough(cfg, rng):
    """Parameters with gains and shifts away from 1 and 0 (exercises them)."""
    P = R.init_params(cfg, rng, std=0.3)
    for n in P:
        if n.endswith(".g"):
            P[n] = 1.0 + 0.3 * rng.normal(size=P[n].shape)
        elif n.endswith(".b"):
            P[n] = 0.3 * rng.normal(size=P[n].shape)
    return P


def test_against_torch_autograd():
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    cfg = _small()
    rng = np.random.default_rng(0)
    P = _rough(cfg, rng)
    x, y = _batch(cfg, rng)
    loss, cache = R.forward(cfg, P, x, y)
    G = R.backward(cfg, P, cache)

    T = {n: torch.tensor(v, dtype=torch.float64, requires_grad=True) for n, v in P.items()}

    def conv(h, name, k, stride, pad):
        w = T[name]
        w4 = w.reshape(w.shape[0], k, k, -1).permute(0, 3, 1, 2)
        return F.conv2d(h, w4, stride=stride, padding=pad)

    def bn(h, pre):
        return F.batch_norm(h, None, None, T[pre + ".g"], T[pre + ".b"], training=True, eps=cfg.ln_eps)

    h = torch.tensor(x)
    h = F.max_pool2d(F.relu(bn(conv(h, "stem.conv.w", 7, 2, 3), "stem.bn")), 3, 2, 1)
    for i, _, cin, mid, cout, stride, proj in R.block_specs(cfg):
        p = f"b{i}."
        o = F.relu(bn(conv(h, p + "conv1.w", 1, 1, 0), p + "bn1"))
        o = F.relu(bn(conv(o, p + "conv2.w", 3, stride, 1), p + "bn2"))
        o = bn(conv(o, p + "conv3.w", 1, 1, 0), p + "bn3")
        s = bn(conv(h, p + "down.w", 1, stride, 0), p + "down.bn") if proj else h
        h = F.relu(o + s)
    z = F.linear(h.mean(dim=(2, 3)), T["fc.w"], T["fc.b"])
    tl = F.cross_entropy(z, torch.tensor(y))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-12 * abs(loss)
    assert np.allclose(cache["logits"], z.detach().numpy(), rtol=1e-12, atol=1e-13)
    for n in P:
        ref = T[n].grad.numpy()
        assert np.linalg.norm(G[n] - ref) <= 1e-10 * max(np.linalg.norm(ref), 1e-300), n


@pytest.mark.parametrize("k", [0, 1])
def test_finite_differences(k):
    cfg = _small(blocks=(1, 1, 1, 1), width=2, img_size=16, batch=2, classes=5, frozen_layers=k)
    rng = np.random.default_rng(1 + k)
    P = _rough(cfg, rng)
    x, y = _batch(cfg, rng)
    loss, cache = R.forward(cfg, P, x, y)
    G = R.backward(cfg, P, cache)
    train = R.trainable_mask(cfg)
    for n, v in P.items():
        if not train[n]:
            assert n not in G
            continue
        idx = rng.choice(v.size, size=min(6, v.size), replace=False)
        for j in idx:
            h = 1e-6 * max(1.0, abs(v.flat[j]))
            Pp = dict(P)
            Pp[n] = v.copy()
            Pp[n].flat[j] += h
            lp = R.forward(cfg, Pp, x, y)[0]
            Pp[n].flat[j] -= 2 * h
            lm = R.forward(cfg, Pp, x, y)[0]
            fd = (lp - lm) / (2 * h)
            assert abs(fd - G[n].flat[j]) <= 1e-6 * max(1.0, abs(fd)) + 1e-9, (n, j, fd, G[n].flat[j])


def test_conv_of_one_pixel_is_the_kernel():
    rng = np.random.default_rng(2)
    k, C, Co = 3, 2, 4
    w = rng.normal(size=(Co, k * k * C))
    x = np.zeros((1, 5, 5, C))
    x[0, 2, 2, :] = [1.0, 0.0]
    out, _ = R.conv_fwd(x, w, k, 1, 1)
    w4 = w.reshape(Co, k, k, C)
    # out[i, j] = sum_{a, b} x[i + a - 1, j + b - 1] w[a, b]: the pixel at (2, 2)
    # is seen by output (i, j) through tap (a, b) = (3 - i, 3 - j)
    for i in range(1, 4):
        for j in range(1, 4):
            assert np.allclose(out[0, i, j], w4[:, 3 - i, 3 - j, 0])
    assert np.count_nonzero(np.abs(out).sum(axis=-1)) == 9
    # stride 2 keeps every other output position
    out2, _ = R.conv_fwd(x, w, k, 2, 1)
    assert out2.shape == (1, 3, 3, Co)
    assert np.allclose(out2, out[:, ::2, ::2])


def test_batchnorm_channel_statistics():
    rng = np.random.default_rng(3)
    x = rng.normal(3.0, 2.5, size=(4, 5, 6, 7))
    y, _ = R.bn_fwd(x, np.ones(7), np.zeros(7), 0.0)
    y2 = y.reshape(-1, 7)
    assert np.allclose(y2.mean(axis=0), 0, atol=1e-13)
    assert np.allclose((y2 ** 2).mean(axis=0), 1, atol=1e-12)
    dy = rng.normal(size=x.shape)
    dx, dg, db = R.bn_bwd(dy, R.bn_fwd(x, np.ones(7), np.zeros(7), 0.0)[1])
    xh = y.reshape(-1, 7)
    assert np.allclose(dx.reshape(-1, 7).sum(axis=0), 0, atol=1e-11)
    assert np.allclose((dx.reshape(-1, 7) * xh).sum(axis=0), 0, atol=1e-11)
    assert np.allclose(db, dy.reshape(-1, 7).sum(axis=0))


def test_maxpool_constant_and_first_position():
    x = np.full((1, 6, 6, 2), 1.5)
    out, cache = R.maxpool_fwd(x)
    assert out.shape == (1, 3, 3, 2) and np.all(out == 1.5)
    dx = R.maxpool_bwd(np.ones_like(out), cache)
    # window (i, j) covers rows 2i - 1 .. 2i + 1; its first in-bounds position
    # is (max(2i - 1, 0), max(2j - 1, 0))
    expect = np.zeros((6, 6))
    for i in range(3):
        for j in range(3):
            expect[max(2 * i - 1, 0), max(2 * j - 1, 0)] += 1.0
    assert np.array_equal(dx[0, :, :, 0], expect)
    # a strict maximum takes the whole gradient
    rng = np.random.default_rng(4)
    x = rng.normal(size=(2, 7, 7, 3))
    out, cache = R.maxpool_fwd(x)
    dx = R.maxpool_bwd(np.ones_like(out), cache)
    for n in range(2):
        for c in range(3):
            for i in range(out.shape[1]):
                for j in range(out.shape[2]):
                    r0, c0 = max(2 * i - 1, 0), max(2 * j - 1, 0)
                    win = x[n, r0:2 * i + 2, c0:2 * j + 2, c]
                    assert out[n, i, j, c] == win.max()
    assert math.isclose(dx.sum(), out.size)


def test_frozen_prefix_and_three_steps():
    cfg = _small(frozen_layers=2, batch=4)
    rng = np.random.default_rng(5)
    P = R.init_params(cfg, rng)
    x, y = _batch(cfg, rng)
    train = R.trainable_mask(cfg)
    assert not train["stem.conv.w"] and not train["b1.conv2.w"] and train["b2.conv2.w"] and train["fc.w"]
    P0 = {n: v.copy() for n, v in P.items()}
    state, losses = {}, []
    for _ in range(3):
        loss, G, P, state, _ = R.train_step(cfg, P, state, x, y)
        losses.append(loss)
        assert set(G) == {n for n, t in train.items() if t}
    for n, t in train.items():
        assert np.array_equal(P[n], P0[n]) != t, n
    assert losses[2] < losses[0]


def test_step_flops_counts():
    """ResNet-50 forward at 224 x 224: 4.09 G multiply-adds (the figure usually
    quoted for the stride-on-3x3 variant), within 1 %; a step with nothing
    frozen is three forwards less the stem's input gradient."""
    cfg = R.ResNetConfig(blocks=(3, 4, 6, 3), width=64, batch=1)
    macs = R.forward_flops(cfg) / 2.0
    assert abs(macs - 4.09e9) / 4.09e9 < 0.01, macs
    stem = 2.0 * 112 * 112 * 147 * 64
    assert abs(R.step_flops(cfg) - (3.0 * R.forward_flops(cfg) - stem)) < 1.0
    k2 = R.ResNetConfig(blocks=(3, 4, 6, 3), width=64, batch=1, frozen_layers=16)
    head = 2.0 * 2048 * 1000
    assert abs(R.step_flops(k2) - (R.forward_flops(k2) + 2.0 * head)) < 1.0


def test_bf16_rounding():
    """Round to nearest, ties to even, on hand values; and torch's own
    float32 -> bfloat16 conversion on random values of every magnitude."""
    assert R.bf16_round(np.array([1.0]))[0] == 1.0
    assert R.bf16_round(np.array([1.0 + 2.0 ** -8]))[0] == 1.0                 # tie -> even (1.0)
    assert R.bf16_round(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6  # tie -> even (odd lsb up)
    assert R.bf16_round(np.array([1.0 + 2.0 ** -8 + 2.0 ** -12]))[0] == 1.0 + 2.0 ** -7
    assert R.bf16_round(np.array([-3.0 - 2.0 ** -7]))[0] == -3.0
    assert R.bf16_round(np.array([0.0, -0.0, np.inf]))[2] == np.inf
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    x = rng.normal(size=4000) * np.exp(rng.uniform(-30, 30, size=4000))
    ref = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(R.bf16_round(x), ref)


def test_bf16_operands_mode():
    """With operands already bfloat16-exact (small dyadic values) the first
    convolution is unchanged by the rounding mode; with general operands the
    mode changes the result (every product sees rounded operands)."""
    cfg = _small(blocks=(1, 1, 1, 1), width=4, img_size=32, batch=2, classes=5)
    cfgb = _small(blocks=(1, 1, 1, 1), width=4, img_size=32, batch=2, classes=5, operands="bf16")
    rng = np.random.default_rng(8)
    P = {n: np.round(v * 64) / 64 for n, v in _rough(cfg, rng).items()}
    x = np.round(rng.normal(size=(2, 3, 32, 32)) * 8) / 8
    y = rng.integers(0, 5, size=2)
    l0, c0 = R.forward(cfg, P, x, y)
    l1, c1 = R.forward(cfgb, P, x, y)
    # the first convolution's operands are exact, so the stem activation agrees
    assert np.allclose(c0["acts"][0], c1["acts"][0], rtol=1e-12, atol=1e-12)
    assert abs(l0 - l1) < 0.05 * abs(l0)
    # general operands: every rounded product sees operands within 2^-8 relative
    P2 = _rough(cfg, rng)
    l2, _ = R.forward(cfg, P2, x, y)
    l3, _ = R.forward(cfgb, P2, x, y)
    assert l2 != l3 and np.isfinite(l3)
