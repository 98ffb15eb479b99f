"""Pins of the oracle's forward pieces against closed forms, invariants,
special cases and brute force written independently of the oracle."""

import math
import os

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import Config, adamw_update, forward, init_params, train_step, trainable_mask
from oracle import layers as L
from tests.oracle_cases import batch, make_cfg, rough_params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- loss at init

def _golden_loss_table():
    rows = {}
    with open(os.path.join(GOLDEN, "loss_at_init.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            name, V, d, lnv, l0 = line.split()
            rows[name] = (int(V), int(d), float(lnv), float(l0))
    return rows


def test_golden_table_is_the_closed_form():
    for name, (V, d, lnv, l0) in _golden_loss_table().items():
        assert abs(lnv - math.log(V)) < 1e-5 and abs(l0 - (math.log(V) + 2e-4 * d)) < 1e-5, name


def test_loss_at_init_tiny_decoder():
    """2-layer d=64 decoder, vocab 512, 0.02-std init: mean loss over seeds is
    within 3 % of ln V + 2e-4 d, and within 2 % of ln V."""
    V, d, lnv, l0 = _golden_loss_table()["tiny"]
    cfg = Config(arch="gpt2", n_layers=2, d_model=d, n_heads=4, d_mlp=256, vocab=V,
                 seq_len=32, batch=2)
    losses = []
    for s in range(4):
        rng = np.random.default_rng(s)
        P = init_params(cfg, rng)
        x, y = batch(cfg, rng)
        losses.append(forward(cfg, P, x, y)[0])
    mean = float(np.mean(losses))
    assert abs(mean - l0) / l0 < 0.03
    assert abs(mean - lnv) / lnv < 0.02


def test_loss_at_init_vit():
    """ViT with 1000 classes and d = 1280 over a 1-layer, 2-image model: the CLS
    row feeds the head, so the same closed form holds (ln 1000 + 0.256)."""
    V, d, lnv, l0 = _golden_loss_table()["vith"]
    cfg = Config(arch="vit", n_layers=1, d_model=d, n_heads=16, d_mlp=64, vocab=V,
                 img_size=28, patch=14, channels=3, batch=64)
    rng = np.random.default_rng(5)
    P = init_params(cfg, rng)
    x, y = batch(cfg, rng)
    loss = forward(cfg, P, x, y)[0]
    assert abs(loss - l0) / l0 < 0.03


# ---------------------------------------------------------------- cross-entropy

def test_cross_entropy_uniform_logits():
    V, N = 37, 6
    z = np.full((N, V), 2.5)
    lab = np.arange(N) % V
    loss, dz = L.cross_entropy(z, lab)
    assert abs(loss - math.log(V)) < 1e-14
    expect = np.full((N, V), 1.0 / V)
    expect[np.arange(N), lab] -= 1.0
    assert np.allclose(dz, expect / N, atol=1e-16)


def test_cross_entropy_library_and_ignore():
    rng = np.random.default_rng(0)
    z = rng.normal(0, 3, size=(9, 50))
    lab = rng.integers(0, 50, size=9)
    lab[[2, 5]] = -1
    loss, dz = L.cross_entropy(z, lab)
    keep = lab >= 0
    ref = np.mean(logsumexp(z[keep], axis=1) - z[keep, lab[keep]])
    assert abs(loss - ref) < 1e-13
    assert np.all(dz[~keep] == 0)
    assert np.allclose(dz.sum(axis=1), 0, atol=1e-16)


# ---------------------------------------------------------------- LayerNorm

def test_layernorm_constant_row_gives_shift():
    x = np.full((3, 8), 4.2)
    g = np.linspace(0.5, 2.0, 8)
    b = np.linspace(-1.0, 1.0, 8)
    y, _ = L.layernorm_fwd(x, g, b, 1e-5)
    assert np.allclose(y, b, atol=1e-12)


def test_layernorm_unit_stats_and_bwd_invariants():
    rng = np.random.default_rng(3)
    x = rng.normal(2.0, 3.0, size=(5, 32))
    y, cache = L.layernorm_fwd(x, np.ones(32), np.zeros(32), 0.0)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-13)
    assert np.allclose((y ** 2).mean(axis=1), 1, atol=1e-12)
    dy = rng.normal(size=(5, 32))
    dx, _, _ = L.layernorm_bwd(dy, cache)
    xhat = cache[0]
    assert np.allclose(dx.sum(axis=1), 0, atol=1e-12)
    assert np.allclose((dx * xhat).sum(axis=1), 0, atol=1e-12)


# ---------------------------------------------------------------- GELU

def test_gelu_erf_against_math_erf_and_tanh_form():
    xs = np.linspace(-6, 6, 241)
    ref = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in xs])
    assert np.allclose(L.gelu_erf(xs), ref, atol=1e-15, rtol=1e-14)
    assert np.max(np.abs(L.gelu_tanh(xs) - ref)) < 1e-3
    # derivatives against central differences
    h = 1e-6
    for f, df in ((L.gelu_tanh, L.gelu_tanh_grad), (L.gelu_erf, L.gelu_erf_grad)):
        fd = (f(xs + h) - f(xs - h)) / (2 * h)
        assert np.allclose(df(xs), fd, atol=1e-8)


# ---------------------------------------------------------------- rotary

def test_rope_invariants():
    rng = np.random.default_rng(4)
    S, dh, rd = 11, 12, 8
    q = rng.normal(size=(S, dh))
    k = rng.normal(size=(S, dh))
    rq = L.rope_apply(q, rd)
    assert np.allclose(np.linalg.norm(rq, axis=1), np.linalg.norm(q, axis=1))
    assert np.array_equal(rq[:, rd:], q[:, rd:])           # pass-through dims
    assert np.allclose(rq[0], q[0])                         # position 0 is identity
    assert np.allclose(L.rope_apply(rq, rd, inverse=True), q)
    assert np.array_equal(L.rope_apply(q, 0), q)
    # <R_m a, R_n b> depends only on m - n
    a, b = rng.normal(size=dh), rng.normal(size=dh)
    A = L.rope_apply(np.tile(a, (S, 1)), rd)
    Bm = L.rope_apply(np.tile(b, (S, 1)), rd)
    assert abs(A[7] @ Bm[4] - A[5] @ Bm[2]) < 1e-12
    assert abs(A[9] @ Bm[9] - a @ b) < 1e-12
    # one hand value: pair 0 at position 1 turns by exactly 1 radian
    e = np.zeros((2, dh))
    e[:, 0] = 1.0
    r = L.rope_apply(e, rd)
    assert np.allclose(r[1, :2], [math.cos(1.0), math.sin(1.0)])
    # pair 1 at position 1 turns by 10000^(-2/rd)
    e = np.zeros((2, dh))
    e[:, 2] = 1.0
    r = L.rope_apply(e, rd)
    th = 10000.0 ** (-2.0 / rd)
    assert np.allclose(r[1, 2:4], [math.cos(th), math.sin(th)])


# ---------------------------------------------------------------- attention

def _attn_bruteforce(q, k, v, causal):
    S, dh = q.shape
    out = np.zeros_like(v)
    for i in range(S):
        js = range(i + 1) if causal else range(S)
        s = [sum(q[i, t] * k[j, t] for t in range(dh)) / math.sqrt(dh) for j in js]
        mx = max(s)
        w = [math.exp(x - mx) for x in s]
        tot = sum(w)
        for jj, j in enumerate(js):
            out[i] += w[jj] / tot * v[j]
    return out


@pytest.mark.parametrize("causal", [True, False])
def test_attention_bruteforce(causal):
    rng = np.random.default_rng(8)
    q, k, v = (rng.normal(size=(6, 4)) for _ in range(3))
    o, P = L.attention_fwd(q, k, v, causal)
    assert np.allclose(o, _attn_bruteforce(q, k, v, causal), atol=1e-13)
    assert np.allclose(P.sum(axis=1), 1)


def test_attention_special_cases():
    rng = np.random.default_rng(9)
    q, k, v = (rng.normal(size=(5, 4)) for _ in range(3))
    o, _ = L.attention_fwd(q[:1], k[:1], v[:1], True)
    assert np.allclose(o[0], v[0])                         # S = 1
    o, _ = L.attention_fwd(np.zeros_like(q), k, v, True)   # zero queries
    for i in range(5):
        assert np.allclose(o[i], v[: i + 1].mean(axis=0))
    o, _ = L.attention_fwd(np.zeros_like(q), k, v, False)
    assert np.allclose(o, v.mean(axis=0))


@pytest.mark.parametrize("arch", ["gpt2", "gptj"])
def test_model_causality(arch):
    """Changing tokens after position s leaves the residual stream at positions
    <= s unchanged, bit for bit."""
    cfg = make_cfg(arch)
    rng = np.random.default_rng(10)
    P = rough_params(cfg, rng)
    x, y = batch(cfg, rng)
    _, c1 = forward(cfg, P, x, y)
    x2 = x.copy()
    s = 2
    x2[:, s + 1:] = (x2[:, s + 1:] + 3) % cfg.vocab
    _, c2 = forward(cfg, P, x2, y)
    for a1, a2 in zip(c1["acts"], c2["acts"]):
        assert np.array_equal(a1[:, : s + 1], a2[:, : s + 1])
        assert not np.array_equal(a1[:, s + 1:], a2[:, s + 1:])


def test_gptj_rotary_zero_is_plain_attention():
    """With rotary_dim = 0 the GPT-J block equals the same block without rotary,
    which for a single position is also position-free."""
    cfg = make_cfg("gptj", rotary_dim=0)
    cfg4 = make_cfg("gptj", rotary_dim=4)
    rng = np.random.default_rng(11)
    P = rough_params(cfg, rng)
    x, y = batch(cfg, rng)
    l0 = forward(cfg, P, x, y)[0]
    l4 = forward(cfg4, P, x, y)[0]
    assert l0 != l4
    # position 0 is rotated by angle 0, so the first row agrees
    a0 = forward(cfg, P, x, y)[1]["acts"][1][:, 0]
    a4 = forward(cfg4, P, x, y)[1]["acts"][1][:, 0]
    assert np.allclose(a0, a4, atol=1e-14)


# ---------------------------------------------------------------- AdamW

def test_adamw_first_step_closed_form():
    cfg = Config(arch="gpt2", n_layers=1, d_model=4, n_heads=1, d_mlp=4, vocab=4,
                 lr=1e-3, weight_decay=0.01)
    rng = np.random.default_rng(12)
    p0, g = rng.normal(size=100), rng.normal(size=100)
    g[:3] = [0.0, 1e-12, -1e-12]
    p1, m1, v1 = adamw_update(cfg, p0, g, np.zeros(100), np.zeros(100), 1)
    expect = p0 * (1 - cfg.lr * cfg.weight_decay) - cfg.lr * g / (np.abs(g) + cfg.eps)
    assert np.allclose(p1, expect, rtol=1e-12, atol=1e-15)
    assert np.allclose(m1, 0.1 * g) and np.allclose(v1, 0.001 * g * g)


def test_adamw_constant_gradient_steps():
    """A constant gradient keeps m_hat = g and v_hat = g^2 at every step, so each
    step moves by lr * g / (|g| + eps) after decay."""
    cfg = Config(arch="gpt2", n_layers=1, d_model=4, n_heads=1, d_mlp=4, vocab=4,
                 lr=1e-2, weight_decay=0.0)
    g = np.array([0.5, -2.0, 3e-3])
    p, m, v = np.zeros(3), np.zeros(3), np.zeros(3)
    for t in range(1, 6):
        p, m, v = adamw_update(cfg, p, g, m, v, t)
    assert np.allclose(p, -5 * cfg.lr * g / (np.abs(g) + cfg.eps), rtol=1e-12)


# ---------------------------------------------------------------- whole step

@pytest.mark.parametrize("arch", ["gpt2", "gptj", "vit"])
def test_frozen_tensors_untouched(arch):
    cfg = make_cfg(arch, frozen_layers=1)
    rng = np.random.default_rng(13)
    P = rough_params(cfg, rng)
    state = {}
    P0 = {n: a.copy() for n, a in P.items()}
    for _ in range(2):
        x, y = batch(cfg, rng)
        _, G, P, state, _ = train_step(cfg, P, state, x, y)
    for n, t in trainable_mask(cfg).items():
        if not t:
            assert np.array_equal(P[n], P0[n]) and not state["m"][n].any() and not state["v"][n].any()
            assert n not in G
        else:
            assert not np.array_equal(P[n], P0[n])


@pytest.mark.parametrize("arch", ["gpt2", "gptj", "vit"])
def test_batch_decomposition(arch):
    """With equal valid counts per row, the batch loss and gradient are the
    means of the per-row ones."""
    cfg = make_cfg(arch)
    cfg1 = make_cfg(arch, batch=1)
    rng = np.random.default_rng(14)
    P = rough_params(cfg, rng)
    x, y = batch(cfg, rng)
    from oracle import backward
    loss, c = forward(cfg, P, x, y)
    G = backward(cfg, P, c)
    parts = []
    for b in range(cfg.batch):
        lb, cb = forward(cfg1, P, x[b:b + 1], y[b:b + 1])
        parts.append((lb, backward(cfg1, P, cb)))
    assert abs(loss - np.mean([p[0] for p in parts])) < 1e-12
    for n in G:
        assert np.allclose(G[n], np.mean([p[1][n] for p in parts], axis=0), atol=1e-14)


def test_three_steps_lower_the_loss():
    cfg = Config(arch="gpt2", n_layers=2, d_model=64, n_heads=4, d_mlp=256, vocab=512,
                 seq_len=32, batch=2, lr=1e-3)
    rng = np.random.default_rng(15)
    P = init_params(cfg, rng)
    x, y = batch(cfg, rng)
    state, losses = {}, []
    for _ in range(4):
        loss, _, P, state, _ = train_step(cfg, P, state, x, y)
        losses.append(loss)
    assert all(b < a for a, b in zip(losses, losses[1:])), losses
