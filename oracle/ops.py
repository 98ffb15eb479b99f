"""Op-level references for the kernel tests: each is the plain definition in
float64, built from the oracle's layer functions or a library primitive.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).
"""

import numpy as np

from . import layers as L


def gemm(A, B):
    """C = A @ B^T for A [M, K], B [N, K] (float64 library matmul)."""
    return np.asarray(A, np.float64) @ np.asarray(B, np.float64).T


def gelu(x, erf_form):
    return L.gelu(np.asarray(x, np.float64), "erf" if erf_form else "tanh")


def gelu_grad(x, erf_form):
    return L.gelu_grad(np.asarray(x, np.float64), "erf" if erf_form else "tanh")


def layernorm_fwd(x, g, b, eps):
    y, (xhat, rstd, _) = L.layernorm_fwd(np.asarray(x, np.float64), g, b, eps)
    mean = np.asarray(x, np.float64).mean(axis=-1)
    return y, mean, rstd[..., 0]


def layernorm_bwd(dy, x, g, eps):
    _, cache = L.layernorm_fwd(np.asarray(x, np.float64), g, np.zeros_like(g), eps)
    return L.layernorm_bwd(np.asarray(dy, np.float64), cache)


def attention(q, k, v, causal):
    """q, k, v: [B, H, S, dh].  Returns o [B, H, S, dh], lse [B, H, S], probs."""
    B, H, S, dh = q.shape
    o = np.empty((B, H, S, dh))
    lse = np.empty((B, H, S))
    probs = np.empty((B, H, S, S))
    for b in range(B):
        for h in range(H):
            o[b, h], probs[b, h] = L.attention_fwd(q[b, h], k[b, h], v[b, h], causal)
            sc = q[b, h] @ k[b, h].T / np.sqrt(dh)
            if causal:
                sc = np.where(np.triu(np.ones((S, S), bool), 1), -np.inf, sc)
            mx = sc.max(axis=-1)
            lse[b, h] = mx + np.log(np.exp(sc - mx[:, None]).sum(axis=-1))
    return o, lse, probs


def attention_bwd(do, q, k, v, probs):
    B, H = q.shape[:2]
    dq, dk, dv = np.empty_like(q), np.empty_like(k), np.empty_like(v)
    for b in range(B):
        for h in range(H):
            dq[b, h], dk[b, h], dv[b, h] = L.attention_bwd(do[b, h], q[b, h], k[b, h], v[b, h], probs[b, h])
    return dq, dk, dv


def rope(x, rd, inverse=False):
    """x: [B, H, S, dh]."""
    return L.rope_apply(np.asarray(x, np.float64), rd, inverse)


def cross_entropy(z, labels):
    """Returns (per-row nll (0 for ignored), dz, mean loss)."""
    z = np.asarray(z, np.float64)
    loss, dz = L.cross_entropy(z, labels)
    m = z.max(axis=-1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[:, 0]
    rows = np.where(labels >= 0, lse - z[np.arange(len(labels)), np.maximum(labels, 0)], 0.0)
    return rows, dz, loss


def adamw(p, g, m, v, t, lr, beta1, beta2, eps, wd):
    from .model import Config, adamw_update
    cfg = Config(arch="gpt2", n_layers=1, d_model=1, n_heads=1, d_mlp=1, vocab=1, lr=lr,
                 beta1=beta1, beta2=beta2, eps=eps, weight_decay=wd)
    return adamw_update(cfg, np.asarray(p, np.float64), np.asarray(g, np.float64),
                        np.asarray(m, np.float64), np.asarray(v, np.float64), t)


def embed_bwd(tok, dh, V):
    out = np.zeros((V, dh.shape[-1]))
    np.add.at(out, np.asarray(tok).reshape(-1), np.asarray(dh, np.float64).reshape(-1, dh.shape[-1]))
    return out
