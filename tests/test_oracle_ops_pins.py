"""Pins of the op-level oracle outputs that the kernel tests compare against
(``oracle/ops.py``): the attention log-sum-exp, the per-row cross-entropy
loss and the LayerNorm mean / reciprocal standard deviation.

Each is tied to something other than the oracle's own formula: closed forms
of special inputs, brute-force loops with ``math.fsum``, and SciPy's
``logsumexp`` library routine."""

import math

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import ops


# ---------------------------------------------------------------- attention LSE

def _lse_bruteforce(q, k, causal):
    """Per-query log-sum-exp of the scaled (masked) scores, one score at a time."""
    S, dh = q.shape
    out = np.empty(S)
    for i in range(S):
        js = range(i + 1) if causal else range(S)
        s = [math.fsum(q[i, t] * k[j, t] for t in range(dh)) / math.sqrt(dh) for j in js]
        mx = max(s)
        out[i] = mx + math.log(math.fsum(math.exp(x - mx) for x in s))
    return out


@pytest.mark.parametrize("causal", [True, False])
def test_attention_lse_against_bruteforce_and_scipy(causal):
    rng = np.random.default_rng(21)
    B, H, S, dh = 2, 2, 7, 5
    q, k, v = (rng.normal(0, 1.5, size=(B, H, S, dh)) for _ in range(3))
    _, lse, P = ops.attention(q, k, v, causal)
    for b in range(B):
        for h in range(H):
            assert np.allclose(lse[b, h], _lse_bruteforce(q[b, h], k[b, h], causal), atol=1e-13)
            sc = q[b, h] @ k[b, h].T / math.sqrt(dh)
            if causal:
                sc = np.where(np.tril(np.ones((S, S), bool)), sc, -np.inf)
            assert np.allclose(lse[b, h], logsumexp(sc, axis=1), atol=1e-13)
            # the probabilities the oracle returns are exp(score - lse)
            assert np.allclose(P[b, h], np.exp(sc - lse[b, h][:, None]), atol=1e-14)


def test_attention_lse_closed_forms():
    rng = np.random.default_rng(22)
    dh = 6
    q, k, v = (rng.normal(size=(1, 1, 1, dh)) for _ in range(3))
    # S = 1: a single score, so lse = q . k / sqrt(dh)
    _, lse, _ = ops.attention(q, k, v, causal=True)
    assert abs(lse[0, 0, 0] - float(q[0, 0, 0] @ k[0, 0, 0]) / math.sqrt(dh)) < 1e-14
    # zero queries: every visible score is 0, so lse = ln(#visible keys)
    S = 9
    q0 = np.zeros((1, 1, S, dh))
    k, v = (rng.normal(size=(1, 1, S, dh)) for _ in range(2))
    _, lse, _ = ops.attention(q0, k, v, causal=True)
    assert np.allclose(lse[0, 0], np.log(np.arange(1, S + 1)), atol=1e-14)
    _, lse, _ = ops.attention(q0, k, v, causal=False)
    assert np.allclose(lse[0, 0], math.log(S), atol=1e-14)
    # a constant shift of every score by c (keys with a fixed component along q)
    # shifts the lse by exactly c
    q1 = np.zeros((1, 1, S, dh))
    q1[..., 0] = 2.0
    k1 = k.copy()
    k1[..., 0] = 0.75                    # every score = 2 * 0.75 / sqrt(dh)
    _, lse, _ = ops.attention(q1, k1, v, causal=True)
    c = 1.5 / math.sqrt(dh)
    assert np.allclose(lse[0, 0], c + np.log(np.arange(1, S + 1)), atol=1e-13)


# ---------------------------------------------------------------- cross-entropy rows

def test_cross_entropy_rows_uniform_logits():
    """Uniform logits: every valid row's loss is ln V exactly, ignored rows are 0."""
    V, N = 29, 7
    z = np.full((N, V), -3.25)
    lab = np.arange(N) % V
    lab[[1, 4]] = -1
    rows, dz, loss = ops.cross_entropy(z, lab)
    keep = lab >= 0
    assert np.allclose(rows[keep], math.log(V), atol=1e-14)
    assert np.all(rows[~keep] == 0.0)
    assert abs(loss - math.log(V)) < 1e-14


def test_cross_entropy_rows_against_scipy_and_bruteforce():
    rng = np.random.default_rng(23)
    N, V = 11, 40
    z = rng.normal(0, 4, size=(N, V))
    lab = rng.integers(0, V, size=N)
    lab[[0, 6, 10]] = -1
    rows, dz, loss = ops.cross_entropy(z, lab)
    for i in range(N):
        if lab[i] < 0:
            assert rows[i] == 0.0
            continue
        mx = max(z[i])
        brute = mx + math.log(math.fsum(math.exp(x - mx) for x in z[i])) - z[i, lab[i]]
        assert abs(rows[i] - brute) < 1e-13
        assert abs(rows[i] - (logsumexp(z[i]) - z[i, lab[i]])) < 1e-13
        assert rows[i] > 0.0
    keep = lab >= 0
    # the mean loss is the mean over valid rows of the per-row losses
    assert abs(loss - math.fsum(rows[keep]) / keep.sum()) < 1e-13
    # the per-row loss is the negative log of the softmax probability of the label,
    # and dz carries that probability minus one at the label (over N valid rows)
    for i in np.nonzero(keep)[0]:
        p = math.exp(-rows[i])
        assert abs(dz[i, lab[i]] - (p - 1.0) / keep.sum()) < 1e-14


def test_cross_entropy_rows_one_hot_dominant():
    """A label logit far above the rest gives a per-row loss of about
    (V - 1) exp(-gap): the first-order term of log(1 + sum exp(-gap))."""
    V, gap = 16, 30.0
    z = np.zeros((2, V))
    z[0, 3] = gap
    z[1, 7] = gap
    rows, _, _ = ops.cross_entropy(z, np.array([3, 7]))
    expect = math.log1p((V - 1) * math.exp(-gap))
    assert np.allclose(rows, expect, rtol=1e-12)


# ---------------------------------------------------------------- LayerNorm statistics

def test_layernorm_mean_and_rstd_bruteforce():
    rng = np.random.default_rng(24)
    R, D, eps = 6, 13, 1e-5
    x = rng.normal(1.5, 2.0, size=(R, D))
    _, mean, rstd = ops.layernorm_fwd(x, np.ones(D), np.zeros(D), eps)
    for r in range(R):
        mu = math.fsum(x[r]) / D
        var = math.fsum((t - mu) ** 2 for t in x[r]) / D       # biased variance
        assert abs(mean[r] - mu) < 1e-14
        assert abs(rstd[r] - 1.0 / math.sqrt(var + eps)) < 1e-12 * rstd[r]


def test_layernorm_stats_closed_forms():
    D, eps = 8, 1e-5
    # constant row c: mean c, variance 0, so rstd = 1/sqrt(eps)
    x = np.full((2, D), -7.5)
    _, mean, rstd = ops.layernorm_fwd(x, np.ones(D), np.zeros(D), eps)
    assert np.allclose(mean, -7.5, atol=1e-15)
    assert np.allclose(rstd, 1.0 / math.sqrt(eps), rtol=1e-12)
    # alternating +-a around m: mean m, variance a^2
    a, m = 3.0, 0.25
    x = m + a * np.tile([1.0, -1.0], (1, D // 2))
    _, mean, rstd = ops.layernorm_fwd(x, np.ones(D), np.zeros(D), eps)
    assert abs(mean[0] - m) < 1e-15
    assert abs(rstd[0] - 1.0 / math.sqrt(a * a + eps)) < 1e-14
    # shifting a row shifts its mean and leaves rstd unchanged
    rng = np.random.default_rng(25)
    x = rng.normal(size=(3, D))
    _, m0, r0 = ops.layernorm_fwd(x, np.ones(D), np.zeros(D), eps)
    _, m1, r1 = ops.layernorm_fwd(x + 4.0, np.ones(D), np.zeros(D), eps)
    assert np.allclose(m1, m0 + 4.0, atol=1e-14)
    assert np.allclose(r1, r0, rtol=1e-12)


# ---------------------------------------------------------------- embedding backward

def test_embed_bwd_bruteforce_duplicates():
    """Scatter-add by token id, summing duplicate tokens, checked row by row."""
    rng = np.random.default_rng(26)
    V, T, D = 9, 20, 4
    tok = rng.integers(0, V, size=T)
    tok[:5] = 3                                # force duplicates
    dh = rng.normal(size=(T, D))
    out = ops.embed_bwd(tok, dh, V)
    for r in range(V):
        for c in range(D):
            assert abs(out[r, c] - math.fsum(dh[i, c] for i in range(T) if tok[i] == r)) < 1e-13
