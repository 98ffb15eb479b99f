"""Building blocks of the oracle, each as a forward and a hand-written VJP.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

All arithmetic is numpy float64.  Each function is the plain textbook
definition; no blocking, fusion or reordering.  The paper (Saturn, arXiv
2309.01226) names the models whose fine-tuning step this is (GPT-2, GPT-J,
ViT; Sec. 1 case study, Table 3) but fixes none of their layer formulas, so
the formulas below are the standard published definitions of those layers.
"""

import math

import numpy as np
from scipy.special import erf as _erf

F64 = np.float64


# ----------------------------------------------------------------------------
# LayerNorm: y = (x - mean) / sqrt(var + eps) * g + b, biased variance.
# ----------------------------------------------------------------------------

def layernorm_fwd(x, g, b, eps):
    """Row-wise LayerNorm over the last axis; returns (y, cache)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    y = xhat * g + b
    return y, (xhat, rstd, g)


def layernorm_bwd(dy, cache):
    """VJP of ``layernorm_fwd``: returns (dx, dg, db).

    With g_ = dy * gamma:  dx = rstd * (g_ - mean(g_) - xhat * mean(g_ * xhat)).
    """
    xhat, rstd, g = cache
    gy = dy * g
    mean_gy = gy.mean(axis=-1, keepdims=True)
    mean_gyx = (gy * xhat).mean(axis=-1, keepdims=True)
    dx = rstd * (gy - mean_gy - xhat * mean_gyx)
    red = tuple(range(dy.ndim - 1))
    dg = (dy * xhat).sum(axis=red)
    db = dy.sum(axis=red)
    return dx, dg, db


# ----------------------------------------------------------------------------
# GELU, tanh approximation (GPT-2, GPT-J) and exact erf form (ViT).
# ----------------------------------------------------------------------------

_C = math.sqrt(2.0 / math.pi)
_A = 0.044715


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(_C * (x + _A * x ** 3)))


def gelu_tanh_grad(x):
    t = np.tanh(_C * (x + _A * x ** 3))
    return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * _C * (1.0 + 3.0 * _A * x * x)


def gelu_erf(x):
    return 0.5 * x * (1.0 + _erf(x / math.sqrt(2.0)))


def gelu_erf_grad(x):
    cdf = 0.5 * (1.0 + _erf(x / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
    return cdf + x * pdf


def gelu(x, kind):
    return gelu_tanh(x) if kind == "tanh" else gelu_erf(x)


def gelu_grad(x, kind):
    return gelu_tanh_grad(x) if kind == "tanh" else gelu_erf_grad(x)


# ----------------------------------------------------------------------------
# Rotary position embedding on interleaved pairs (GPT-J convention).
# Pair i (dims 2i, 2i+1), i < rotary_dim/2, is rotated by the angle
# pos * 10000^(-2i/rotary_dim); dims >= rotary_dim pass through.
# ----------------------------------------------------------------------------

def rope_angles(seq_len, rotary_dim):
    i = np.arange(rotary_dim // 2, dtype=F64)
    theta = 10000.0 ** (-2.0 * i / rotary_dim)
    pos = np.arange(seq_len, dtype=F64)
    return np.outer(pos, theta)  # [S, rotary_dim/2]


def rope_apply(x, rotary_dim, inverse=False):
    """Rotate x[..., S, dh] in place-free fashion; inverse=True applies R^T."""
    if rotary_dim == 0:
        return x.copy()
    S = x.shape[-2]
    ang = rope_angles(S, rotary_dim)
    c, s = np.cos(ang), np.sin(ang)
    if inverse:
        s = -s
    out = x.copy()
    x0 = x[..., 0:rotary_dim:2]
    x1 = x[..., 1:rotary_dim:2]
    out[..., 0:rotary_dim:2] = x0 * c - x1 * s
    out[..., 1:rotary_dim:2] = x0 * s + x1 * c
    return out


# ----------------------------------------------------------------------------
# Scaled dot-product attention for one (batch, head): P = softmax(q k^T /
# sqrt(dh) + mask), o = P v.  Causal mask keeps key j <= query i.
# ----------------------------------------------------------------------------

def attention_fwd(q, k, v, causal):
    """q, k, v: [S, dh] float64.  Returns (o, P)."""
    S, dh = q.shape
    scores = (q @ k.T) / math.sqrt(dh)
    if causal:
        mask = np.triu(np.ones((S, S), dtype=bool), k=1)
        scores = np.where(mask, -np.inf, scores)
    m = scores.max(axis=-1, keepdims=True)
    e = np.exp(scores - m)
    P = e / e.sum(axis=-1, keepdims=True)
    return P @ v, P


def attention_bwd(do, q, k, v, P):
    """VJP of ``attention_fwd`` given the saved probabilities P."""
    dh = q.shape[1]
    dv = P.T @ do
    dP = do @ v.T
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True))
    dq = dS @ k / math.sqrt(dh)
    dk = dS.T @ q / math.sqrt(dh)
    return dq, dk, dv


# ----------------------------------------------------------------------------
# Softmax cross-entropy, mean over rows whose label is not -1.
# ----------------------------------------------------------------------------

def cross_entropy(z, labels):
    """z: [N, V] float64, labels: [N] ints (-1 = ignore).  Returns (loss, dz)."""
    valid = labels >= 0
    n_valid = int(valid.sum())
    m = z.max(axis=-1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[:, 0]
    rows = np.nonzero(valid)[0]
    nll = lse[rows] - z[rows, labels[rows]]
    loss = nll.sum() / max(n_valid, 1)
    p = np.exp(z - lse[:, None])
    dz = p.copy()
    dz[rows, labels[rows]] -= 1.0
    dz[~valid] = 0.0
    dz /= max(n_valid, 1)
    return loss, dz
