"""Pin the oracle to independent library routines: the same models assembled
from torch's CPU float64 operators (F.embedding, F.layer_norm, F.linear,
F.scaled_dot_product_attention, F.gelu, F.unfold, F.cross_entropy), gradients
from torch autograd, and the update from torch.optim.AdamW.  Rotary is written
as a multiplication of complex numbers, not as the oracle's cos/sin pairs."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import param_spec, train_step, trainable_mask
from tests.oracle_cases import batch, make_cfg, rough_params


def _rope_complex(x, rd):
    if rd == 0:
        return x
    S = x.shape[-2]
    i = torch.arange(rd // 2, dtype=torch.float64)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * (10000.0 ** (-2.0 * i / rd))[None]
    rot = torch.polar(torch.ones_like(ang), ang)
    xc = torch.view_as_complex(x[..., :rd].reshape(*x.shape[:-1], rd // 2, 2).contiguous())
    xr = torch.view_as_real(xc * rot).reshape(*x.shape[:-1], rd)
    return torch.cat([xr, x[..., rd:]], dim=-1)


def torch_loss(cfg, T, x, y):
    d, H = cfg.d_model, cfg.n_heads
    dh = d // H
    B = cfg.batch
    if cfg.arch == "vit":
        img = torch.as_tensor(x, dtype=torch.float64)
        pt = F.unfold(img, kernel_size=cfg.patch, stride=cfg.patch).transpose(1, 2)
        z = F.linear(pt, T["patch.w"], T["patch.b"])
        h = torch.cat([T["cls"].expand(B, 1, d), z], dim=1) + T["pos"]
    else:
        tok = torch.as_tensor(x, dtype=torch.long)
        h = F.embedding(tok, T["wte"])
        if cfg.arch == "gpt2":
            h = h + T["wpe"][: tok.shape[1]]
    S = h.shape[1]
    approx = "none" if cfg.arch == "vit" else "tanh"
    for l in range(cfg.n_layers):
        p = f"h{l}."
        a = F.layer_norm(h, (d,), T[p + "ln1.g"], T[p + "ln1.b"], cfg.ln_eps)
        qkv = F.linear(a, T[p + "attn.qkv.w"], T.get(p + "attn.qkv.b"))
        q, k, v = (t.reshape(B, S, H, dh).transpose(1, 2) for t in qkv.split(d, dim=-1))
        if cfg.arch == "gptj":
            q, k = _rope_complex(q, cfg.rotary_dim), _rope_complex(k, cfg.rotary_dim)
        o = F.scaled_dot_product_attention(q, k, v, is_causal=cfg.arch != "vit")
        o = o.transpose(1, 2).reshape(B, S, d)
        if cfg.arch == "gptj":
            mlp = F.linear(F.gelu(F.linear(a, T[p + "mlp.fc1.w"], T[p + "mlp.fc1.b"]), approximate=approx),
                           T[p + "mlp.fc2.w"], T[p + "mlp.fc2.b"])
            h = h + F.linear(o, T[p + "attn.proj.w"]) + mlp
        else:
            h = h + F.linear(o, T[p + "attn.proj.w"], T[p + "attn.proj.b"])
            c = F.layer_norm(h, (d,), T[p + "ln2.g"], T[p + "ln2.b"], cfg.ln_eps)
            h = h + F.linear(F.gelu(F.linear(c, T[p + "mlp.fc1.w"], T[p + "mlp.fc1.b"]), approximate=approx),
                             T[p + "mlp.fc2.w"], T[p + "mlp.fc2.b"])
    if cfg.arch == "vit":
        h = h[:, 0]
    f = F.layer_norm(h, (d,), T["lnf.g"], T["lnf.b"], cfg.ln_eps)
    logits = F.linear(f, T["head.w"], T.get("head.b"))
    lab = torch.as_tensor(np.asarray(y), dtype=torch.long).reshape(-1)
    return F.cross_entropy(logits.reshape(lab.shape[0], -1), lab, ignore_index=-1)


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)


@pytest.mark.parametrize("arch", ["gpt2", "gptj", "vit"])
@pytest.mark.parametrize("k", [0, 1])
def test_oracle_matches_torch_three_steps(arch, k):
    cfg = make_cfg(arch, frozen_layers=k, lr=3e-2, weight_decay=0.1)
    rng = np.random.default_rng(99 + k)
    P = rough_params(cfg, rng)
    train = trainable_mask(cfg)
    T = {n: torch.tensor(a, dtype=torch.float64, requires_grad=train[n]) for n, a in P.items()}
    opt = torch.optim.AdamW([T[n] for n, _, _ in param_spec(cfg) if train[n]], lr=cfg.lr,
                            betas=(cfg.beta1, cfg.beta2), eps=cfg.eps, weight_decay=cfg.weight_decay)
    state = {}
    for step in range(3):
        x, y = batch(cfg, rng)
        if cfg.arch != "vit":
            y = y.copy()
            y[1, 0] = -1
        loss, G, P, state, _ = train_step(cfg, P, state, x, y)
        opt.zero_grad()
        tl = torch_loss(cfg, T, x, y)
        tl.backward()
        assert abs(loss - tl.item()) <= 1e-12 * abs(loss), (step, loss, tl.item())
        for n, t in T.items():
            if train[n]:
                assert _rel(G[n], t.grad.numpy()) < 1e-10, (step, n)
            else:
                assert t.grad is None and n not in G
        opt.step()
        # The key bias has an exactly-zero true gradient (softmax is invariant
        # to a per-query constant), so both sides hold rounding noise of ~1e-17
        # there and AdamW's g / (|g| + eps) turns it into differences of up to
        # lr * 1e-9: hence 1e-9 rather than machine precision.
        for n, t in T.items():
            assert _rel(P[n], t.detach().numpy()) < 1e-9, (step, n)
