"""One fine-tuning step of a GPT-2-, GPT-J- or ViT-style transformer, fp64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Scope.  The Saturn paper (arXiv 2309.01226) schedules a set of model-training
tasks, each with its own hyper-parameters (Sec. 3.1 "Workload Specification";
Sec. 2 "Model selection"), over the fine-tuning of pre-trained GPT-2, GPT-J and
ViT models (Sec. 1 case study; Table 3), including model selection over which
layers are fine-tuned (Abstract).  The step below is that unit of work:
forward, exact gradient, and one AdamW update, with the bottom k blocks frozen.

Readings of points the paper leaves open (it fixes no layer formula):
  * pre-LN blocks; GPT-2 and ViT: bias on every linear; GPT-J: one LN per
    block feeding attention and MLP in parallel, no q/k/v/out bias, bias on
    fc1/fc2 and on the LM head;
  * LN eps from the config (1e-5), biased variance;
  * GELU tanh form for GPT-2/GPT-J, erf form for ViT;
  * GPT-J rotary on interleaved pairs of the first ``rotary_dim`` dims of every
    q/k head, base 10000, position = token index;
  * attention scale 1/sqrt(dh); causal mask keeps key <= query for decoders,
    no mask for ViT;
  * untied LM head, no LM-head bias for GPT-2;
  * freezing k > 0 freezes the embeddings and blocks [0, k); final LN and head
    always train; backward stops at the input of block k;
  * AdamW with decoupled decay applied to every trainable tensor, constant lr,
    bias correction, t starting at 1, no clipping, no dropout;
  * ViT patches flattened in (channel, row, col) order, patch grid row-major,
    CLS token at position 0, head on the CLS row after the final LN.

Parameter names and shapes are the interface shared with the GPU library's
parameter table; linear weights are stored [out, in], so y = x W^T + b.
"""

from dataclasses import dataclass

import numpy as np

from . import layers as Lr

F64 = np.float64


@dataclass
class Config:
    arch: str                  # "gpt2" | "gptj" | "vit"
    n_layers: int
    d_model: int
    n_heads: int
    d_mlp: int
    vocab: int                 # decoders: vocabulary size; ViT: classes
    seq_len: int = 0           # decoders: S; ViT: derived from image/patch
    batch: int = 1
    frozen_layers: int = 0
    rotary_dim: int = 0
    img_size: int = 0
    patch: int = 0
    channels: int = 3
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    ln_eps: float = 1e-5

    @property
    def head_dim(self):
        return self.d_model // self.n_heads

    @property
    def n_patches(self):
        return (self.img_size // self.patch) ** 2 if self.arch == "vit" else 0

    @property
    def seq(self):
        return self.n_patches + 1 if self.arch == "vit" else self.seq_len

    @property
    def causal(self):
        return self.arch != "vit"

    @property
    def gelu_kind(self):
        return "erf" if self.arch == "vit" else "tanh"


def param_spec(cfg):
    """Ordered list of (name, shape, group); group is "embed", a block index or "head".

    The order runs bottom to top so that the frozen tensors form a prefix.
    """
    d, m, V, S = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.seq
    spec = []
    if cfg.arch == "vit":
        pd = cfg.channels * cfg.patch * cfg.patch
        spec += [("patch.w", (d, pd), "embed"), ("patch.b", (d,), "embed"),
                 ("cls", (d,), "embed"), ("pos", (S, d), "embed")]
    else:
        spec += [("wte", (V, d), "embed")]
        if cfg.arch == "gpt2":
            spec += [("wpe", (S, d), "embed")]
    for l in range(cfg.n_layers):
        p = f"h{l}."
        if cfg.arch == "gptj":
            spec += [(p + "ln1.g", (d,), l), (p + "ln1.b", (d,), l),
                     (p + "attn.qkv.w", (3 * d, d), l),
                     (p + "mlp.fc1.w", (m, d), l), (p + "mlp.fc1.b", (m,), l),
                     (p + "attn.proj.w", (d, d), l),
                     (p + "mlp.fc2.w", (d, m), l), (p + "mlp.fc2.b", (d,), l)]
        else:
            spec += [(p + "ln1.g", (d,), l), (p + "ln1.b", (d,), l),
                     (p + "attn.qkv.w", (3 * d, d), l), (p + "attn.qkv.b", (3 * d,), l),
                     (p + "attn.proj.w", (d, d), l), (p + "attn.proj.b", (d,), l),
                     (p + "ln2.g", (d,), l), (p + "ln2.b", (d,), l),
                     (p + "mlp.fc1.w", (m, d), l), (p + "mlp.fc1.b", (m,), l),
                     (p + "mlp.fc2.w", (d, m), l), (p + "mlp.fc2.b", (d,), l)]
    spec += [("lnf.g", (d,), "head"), ("lnf.b", (d,), "head"), ("head.w", (V, d), "head")]
    if cfg.arch in ("gptj", "vit"):
        spec += [("head.b", (V,), "head")]
    return spec


def trainable_mask(cfg):
    """name -> bool: embeddings train only when k == 0, block l iff l >= k."""
    out = {}
    for name, _, grp in param_spec(cfg):
        if grp == "embed":
            out[name] = cfg.frozen_layers == 0
        elif grp == "head":
            out[name] = True
        else:
            out[name] = grp >= cfg.frozen_layers
    return out


def init_params(cfg, rng, std=0.02):
    """Reference initialisation for oracle-only tests: matrices, embeddings, CLS
    and position tables ~ N(0, std^2); biases 0; LN gain 1, LN shift 0."""
    out = {}
    for name, shape, _ in param_spec(cfg):
        if name.endswith(".g"):
            out[name] = np.ones(shape, F64)
        elif name.endswith(".b") or name == "patch.b":
            out[name] = np.zeros(shape, F64)
        else:
            out[name] = rng.normal(0.0, std, size=shape).astype(F64)
    return out


# ----------------------------------------------------------------------------
# forward
# ----------------------------------------------------------------------------

def _patches(cfg, images):
    """images [B, C, H, W] -> [B, n_patches, C*p*p], (c, kh, kw) flattening."""
    B, C, H, W = images.shape
    p = cfg.patch
    g = H // p
    x = images.reshape(B, C, g, p, g, p)           # b c r kh col kw
    x = x.transpose(0, 2, 4, 1, 3, 5)              # b r col c kh kw
    return x.reshape(B, g * g, C * p * p)


def _split_heads(x, H):
    """[B, S, H*dh] -> [B, H, S, dh]"""
    B, S, D = x.shape
    return x.reshape(B, S, H, D // H).transpose(0, 2, 1, 3)


def _merge_heads(x):
    B, H, S, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, S, H * dh)


def forward(cfg, P, inputs, labels):
    """Returns (loss, cache).  ``inputs``: int tokens [B, S] or images [B, C, H, W];
    ``labels``: ints [B, S] (decoders) or [B] (ViT), -1 = ignore."""
    B, d, H = cfg.batch, cfg.d_model, cfg.n_heads
    S = cfg.seq
    cache = {"blocks": []}
    if cfg.arch == "vit":
        pt = _patches(cfg, np.asarray(inputs, F64))
        z = pt @ P["patch.w"].T + P["patch.b"]
        cls = np.broadcast_to(P["cls"], (B, 1, d))
        h = np.concatenate([cls, z], axis=1) + P["pos"][None]
        cache["patches"] = pt
    else:
        tok = np.asarray(inputs)
        h = P["wte"][tok]
        if cfg.arch == "gpt2":
            h = h + P["wpe"][None, :S]
        cache["tokens"] = tok
    acts = [h.copy()]
    for l in range(cfg.n_layers):
        p = f"h{l}."
        c = {"h_in": h}
        a, c["ln1"] = Lr.layernorm_fwd(h, P[p + "ln1.g"], P[p + "ln1.b"], cfg.ln_eps)
        c["a"] = a
        qkv = a @ P[p + "attn.qkv.w"].T
        if cfg.arch != "gptj":
            qkv = qkv + P[p + "attn.qkv.b"]
        q = _split_heads(qkv[..., 0:d], H)
        k = _split_heads(qkv[..., d:2 * d], H)
        v = _split_heads(qkv[..., 2 * d:3 * d], H)
        if cfg.arch == "gptj":
            q = Lr.rope_apply(q, cfg.rotary_dim)
            k = Lr.rope_apply(k, cfg.rotary_dim)
        o = np.empty_like(q)
        probs = np.empty((B, H, S, S), F64)
        for b in range(B):
            for j in range(H):
                o[b, j], probs[b, j] = Lr.attention_fwd(q[b, j], k[b, j], v[b, j], cfg.causal)
        c.update(q=q, k=k, v=v, probs=probs)
        o = _merge_heads(o)
        c["o"] = o
        attn_out = o @ P[p + "attn.proj.w"].T
        if cfg.arch == "gptj":
            u = a @ P[p + "mlp.fc1.w"].T + P[p + "mlp.fc1.b"]
            g = Lr.gelu(u, cfg.gelu_kind)
            mlp_out = g @ P[p + "mlp.fc2.w"].T + P[p + "mlp.fc2.b"]
            h = h + attn_out + mlp_out
        else:
            h_mid = h + attn_out + P[p + "attn.proj.b"]
            c["h_mid"] = h_mid
            cc, c["ln2"] = Lr.layernorm_fwd(h_mid, P[p + "ln2.g"], P[p + "ln2.b"], cfg.ln_eps)
            c["c"] = cc
            u = cc @ P[p + "mlp.fc1.w"].T + P[p + "mlp.fc1.b"]
            g = Lr.gelu(u, cfg.gelu_kind)
            h = h_mid + g @ P[p + "mlp.fc2.w"].T + P[p + "mlp.fc2.b"]
        c.update(u=u, g=g)
        cache["blocks"].append(c)
        acts.append(h.copy())
    hf = h[:, 0] if cfg.arch == "vit" else h
    f, cache["lnf"] = Lr.layernorm_fwd(hf, P["lnf.g"], P["lnf.b"], cfg.ln_eps)
    f2 = f.reshape(-1, d)
    logits = f2 @ P["head.w"].T
    if "head.b" in P:
        logits = logits + P["head.b"]
    lab = np.asarray(labels).reshape(-1)
    loss, dz = Lr.cross_entropy(logits, lab)
    cache.update(f=f, logits=logits, dz=dz, acts=acts)
    return loss, cache


# ----------------------------------------------------------------------------
# backward
# ----------------------------------------------------------------------------

def backward(cfg, P, cache):
    """Exact gradient of the mean loss w.r.t. every trainable tensor.

    Frozen tensors get no entry.  The pass stops at the input of block k.
    """
    B, d, H, S = cfg.batch, cfg.d_model, cfg.n_heads, cfg.seq
    k_frz = cfg.frozen_layers
    G = {}
    dz = cache["dz"]
    f2 = cache["f"].reshape(-1, d)
    G["head.w"] = dz.T @ f2
    if "head.b" in P:
        G["head.b"] = dz.sum(axis=0)
    df = (dz @ P["head.w"]).reshape(cache["f"].shape)
    dhf, G["lnf.g"], G["lnf.b"] = Lr.layernorm_bwd(df, cache["lnf"])
    if cfg.arch == "vit":
        dh = np.zeros((B, S, d), F64)
        dh[:, 0] = dhf
    else:
        dh = dhf
    for l in range(cfg.n_layers - 1, k_frz - 1, -1):
        p = f"h{l}."
        c = cache["blocks"][l]
        if cfg.arch == "gptj":
            G[p + "mlp.fc2.w"] = _wgrad(dh, c["g"])
            G[p + "mlp.fc2.b"] = dh.sum(axis=(0, 1))
            dg = dh @ P[p + "mlp.fc2.w"]
            du = dg * Lr.gelu_grad(c["u"], cfg.gelu_kind)
            G[p + "mlp.fc1.w"] = _wgrad(du, c["a"])
            G[p + "mlp.fc1.b"] = du.sum(axis=(0, 1))
            G[p + "attn.proj.w"] = _wgrad(dh, c["o"])
            do = dh @ P[p + "attn.proj.w"]
            dqkv = _attn_bwd(cfg, do, c)
            G[p + "attn.qkv.w"] = _wgrad(dqkv, c["a"])
            da = dqkv @ P[p + "attn.qkv.w"] + du @ P[p + "mlp.fc1.w"]
            dx, G[p + "ln1.g"], G[p + "ln1.b"] = Lr.layernorm_bwd(da, c["ln1"])
            dh = dh + dx
        else:
            G[p + "mlp.fc2.w"] = _wgrad(dh, c["g"])
            G[p + "mlp.fc2.b"] = dh.sum(axis=(0, 1))
            dg = dh @ P[p + "mlp.fc2.w"]
            du = dg * Lr.gelu_grad(c["u"], cfg.gelu_kind)
            G[p + "mlp.fc1.w"] = _wgrad(du, c["c"])
            G[p + "mlp.fc1.b"] = du.sum(axis=(0, 1))
            dc = du @ P[p + "mlp.fc1.w"]
            dx, G[p + "ln2.g"], G[p + "ln2.b"] = Lr.layernorm_bwd(dc, c["ln2"])
            dh_mid = dh + dx
            G[p + "attn.proj.w"] = _wgrad(dh_mid, c["o"])
            G[p + "attn.proj.b"] = dh_mid.sum(axis=(0, 1))
            do = dh_mid @ P[p + "attn.proj.w"]
            dqkv = _attn_bwd(cfg, do, c)
            G[p + "attn.qkv.w"] = _wgrad(dqkv, c["a"])
            G[p + "attn.qkv.b"] = dqkv.sum(axis=(0, 1))
            da = dqkv @ P[p + "attn.qkv.w"]
            dx, G[p + "ln1.g"], G[p + "ln1.b"] = Lr.layernorm_bwd(da, c["ln1"])
            dh = dh_mid + dx
    if k_frz == 0:
        if cfg.arch == "vit":
            G["pos"] = dh.sum(axis=0)
            G["cls"] = dh[:, 0].sum(axis=0)
            dzp = dh[:, 1:]
            G["patch.w"] = _wgrad(dzp, cache["patches"])
            G["patch.b"] = dzp.sum(axis=(0, 1))
        else:
            tok = cache["tokens"].reshape(-1)
            dwte = np.zeros_like(P["wte"])
            np.add.at(dwte, tok, dh.reshape(-1, d))
            G["wte"] = dwte
            if cfg.arch == "gpt2":
                dwpe = np.zeros_like(P["wpe"])
                dwpe[:S] = dh.sum(axis=0)
                G["wpe"] = dwpe
    cache["dh_bottom"] = dh
    return G


def _wgrad(dy, x):
    """dW[out, in] = sum over all leading positions of dy[..., out] x[..., in]."""
    return dy.reshape(-1, dy.shape[-1]).T @ x.reshape(-1, x.shape[-1])


def _attn_bwd(cfg, do_merged, c):
    H = cfg.n_heads
    do = _split_heads(do_merged, H)
    q, k, v, probs = c["q"], c["k"], c["v"], c["probs"]
    dq = np.empty_like(q)
    dk = np.empty_like(k)
    dv = np.empty_like(v)
    for b in range(q.shape[0]):
        for j in range(H):
            dq[b, j], dk[b, j], dv[b, j] = Lr.attention_bwd(do[b, j], q[b, j], k[b, j], v[b, j], probs[b, j])
    if cfg.arch == "gptj":
        dq = Lr.rope_apply(dq, cfg.rotary_dim, inverse=True)
        dk = Lr.rope_apply(dk, cfg.rotary_dim, inverse=True)
    return np.concatenate([_merge_heads(dq), _merge_heads(dk), _merge_heads(dv)], axis=-1)


# ----------------------------------------------------------------------------
# AdamW (decoupled weight decay, bias-corrected moments)
# ----------------------------------------------------------------------------

def adamw_update(cfg, p, g, m, v, t):
    """One AdamW update at step number t (t >= 1).  Returns new (p, m, v).

    p <- p (1 - lr wd);  m <- b1 m + (1-b1) g;  v <- b2 v + (1-b2) g^2;
    p <- p - lr * (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
    """
    lr, b1, b2, eps, wd = cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay
    p = p * (1.0 - lr * wd)
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** t)
    vhat = v / (1.0 - b2 ** t)
    p = p - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v


def train_step(cfg, P, state, inputs, labels):
    """Forward + backward + AdamW on the trainable tensors.

    ``state`` = {"t": int, "m": {name: arr}, "v": {name: arr}} (created when
    empty).  Returns (loss, grads, new_params, new_state, cache).
    """
    loss, cache = forward(cfg, P, inputs, labels)
    grads = backward(cfg, P, cache)
    t = state.get("t", 0) + 1
    newP, newM, newV = {}, {}, {}
    train = trainable_mask(cfg)
    for name, arr in P.items():
        m0 = state.get("m", {}).get(name, np.zeros_like(arr))
        v0 = state.get("v", {}).get(name, np.zeros_like(arr))
        if train[name]:
            newP[name], newM[name], newV[name] = adamw_update(cfg, arr, grads[name], m0, v0, t)
        else:
            newP[name], newM[name], newV[name] = arr, m0, v0
    return loss, grads, newP, {"t": t, "m": newM, "v": newV}, cache


def eval_loss(cfg, P, inputs, labels):
    return forward(cfg, P, inputs, labels)[0]
