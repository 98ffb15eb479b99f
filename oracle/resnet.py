"""Plain float64 oracle of one fine-tuning step of a bottleneck ResNet, the
paper's second image model (Table 3 and Sec. 5 "Workloads": a ResNet of about
200 M parameters fine-tuned on ImageNet-shaped images).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper names the model and its size only.  The readings (also listed in
the repository's design notes):

  * Architecture: the standard bottleneck ResNet.  Stem: 7 x 7 convolution
    with stride 2 and padding 3, batch norm, ReLU, 3 x 3 max pool with
    stride 2 and padding 1.  Four stages of blocks; stage s has mid width
    width * 2^s and output width 4 * width * 2^s; a block is
    1 x 1 conv -> BN -> ReLU -> 3 x 3 conv (stride 2 in the first block of
    stages 1..3, padding 1) -> BN -> ReLU -> 1 x 1 conv -> BN, added to the
    shortcut, then ReLU.  The first block of every stage has a projection
    shortcut (1 x 1 conv with the block's stride, then BN); the others add
    their input.  Head: global average pool, then a linear layer with bias.
    No convolution has a bias.  The 200 M-parameter workload is the
    ResNet-152 depth (3, 8, 36, 3) at twice the standard width (stem 128).
  * Batch norm in training mode: statistics of the current batch over
    (N, H, W), biased variance, eps = ln_eps; no running statistics are kept,
    so evaluation uses the batch statistics too.
  * Initialisation: convolution and linear weights ~ N(0, 0.02^2), biases 0,
    BN gains 1 and shifts 0 (the GPU's values are read back, so the oracle
    needs no RNG parity).
  * Freezing k: k > 0 freezes the stem and blocks [0, k); the head always
    trains.
  * Loss: mean softmax cross-entropy over the batch; AdamW as for the
    transformers (decoupled decay on every trainable tensor).

Layouts: activations NHWC; a convolution weight is stored [Cout, KH, KW, Cin]
(exposed as the matrix [Cout, KH * KW * Cin]); input images NCHW.
Every function is the textbook definition in numpy float64 with a hand-written
vector-Jacobian product.
"""

from dataclasses import dataclass, field

import numpy as np

from . import layers as L
from .model import adamw_update  # noqa: F401  (same optimizer arithmetic)


@dataclass
class ResNetConfig:
    blocks: tuple = (3, 8, 36, 3)
    width: int = 128
    classes: int = 1000
    img_size: int = 224
    channels: int = 3
    batch: int = 64
    frozen_layers: int = 0
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    ln_eps: float = 1e-5
    arch: str = field(default="resnet")
    # "fp64": every product exact.  "bf16": the operands of every convolution
    # and head product rounded to bfloat16 first (round to nearest, ties to
    # even), the products themselves still exact: the arithmetic the GPU path
    # declares (bf16 operands, wide accumulation), written out.
    operands: str = "fp64"

    @property
    def n_blocks(self):
        return int(sum(self.blocks))


# ----------------------------------------------------------------------------
# Architecture description
# ----------------------------------------------------------------------------

def block_specs(cfg):
    """(index, stage, in channels, mid, out, stride, projection) of every block."""
    out = []
    cin = cfg.width
    i = 0
    for s, n in enumerate(cfg.blocks):
        mid = cfg.width * 2 ** s
        for j in range(n):
            stride = 2 if (j == 0 and s > 0) else 1
            out.append((i, s, cin, mid, 4 * mid, stride, j == 0))
            cin = 4 * mid
            i += 1
    return out


def param_spec(cfg):
    """(name, shape, group): group -1 = stem, i = block i, n_blocks = head."""
    w, C = cfg.width, cfg.channels
    spec = [("stem.conv.w", (w, 7 * 7 * C), -1), ("stem.bn.g", (w,), -1), ("stem.bn.b", (w,), -1)]
    for i, _, cin, mid, cout, _, proj in block_specs(cfg):
        p = f"b{i}."
        spec += [(p + "conv1.w", (mid, cin), i), (p + "bn1.g", (mid,), i), (p + "bn1.b", (mid,), i),
                 (p + "conv2.w", (mid, 9 * mid), i), (p + "bn2.g", (mid,), i), (p + "bn2.b", (mid,), i),
                 (p + "conv3.w", (cout, mid), i), (p + "bn3.g", (cout,), i), (p + "bn3.b", (cout,), i)]
        if proj:
            spec += [(p + "down.w", (cout, cin), i), (p + "down.bn.g", (cout,), i),
                     (p + "down.bn.b", (cout,), i)]
    feat = 4 * cfg.width * 2 ** (len(cfg.blocks) - 1)
    spec += [("fc.w", (cfg.classes, feat), cfg.n_blocks), ("fc.b", (cfg.classes,), cfg.n_blocks)]
    return spec


def trainable_mask(cfg):
    k = cfg.frozen_layers
    return {n: (g >= k if g >= 0 else k == 0) for n, _, g in param_spec(cfg)}


def init_params(cfg, rng, std=0.02):
    P = {}
    for n, shape, _ in param_spec(cfg):
        if n.endswith(".g"):
            P[n] = np.ones(shape)
        elif n.endswith(".b"):
            P[n] = np.zeros(shape)
        else:
            P[n] = rng.normal(0.0, std, size=shape)
    return P


# ----------------------------------------------------------------------------
# Operand precision
# ----------------------------------------------------------------------------

def bf16_round(x):
    """Round to the nearest bfloat16 value (ties to even), as float64: the
    value goes to float32 first, then the low 16 bits of its IEEE pattern are
    rounded away (add 0x7FFF plus the lowest kept bit, then truncate)."""
    f = np.ascontiguousarray(np.asarray(x, np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out).reshape(np.shape(x))


def _rounder(cfg):
    return bf16_round if getattr(cfg, "operands", "fp64") == "bf16" else (lambda a: a)


# ----------------------------------------------------------------------------
# Layers (NHWC)
# ----------------------------------------------------------------------------

def conv_fwd(x, w, k, stride, pad, rnd=None):
    """x [N, H, W, Cin]; w [Cout, k * k * Cin] (as [Cout, k, k, Cin]).
    out[n, i, j, o] = sum_{a, b, c} xpad[n, i s + a, j s + b, c] w[o, a, b, c].
    rnd: optional rounding of both operands before the product."""
    if rnd is not None:
        x, w = rnd(x), rnd(w)
    N, H, W, C = x.shape
    Cout = w.shape[0]
    w4 = w.reshape(Cout, k, k, C)
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C))
    xp[:, pad:pad + H, pad:pad + W] = x
    out = np.zeros((N, Ho, Wo, Cout))
    for a in range(k):
        for b in range(k):
            patch = xp[:, a:a + stride * (Ho - 1) + 1:stride, b:b + stride * (Wo - 1) + 1:stride]
            out += patch @ w4[:, a, b, :].T
    return out, (x.shape, xp, w4, k, stride, pad, rnd)


def conv_bwd(dy, cache):
    """VJP of conv_fwd: returns (dx, dw).  With a rounding the forward used,
    dy is rounded too (the operands of both backward products)."""
    (N, H, W, C), xp, w4, k, stride, pad, rnd = cache
    if rnd is not None:
        dy = rnd(dy)
    _, Ho, Wo, Cout = dy.shape
    dxp = np.zeros_like(xp)
    dw4 = np.zeros_like(w4)
    d2 = dy.reshape(-1, Cout)
    for a in range(k):
        for b in range(k):
            sl = (slice(None), slice(a, a + stride * (Ho - 1) + 1, stride),
                  slice(b, b + stride * (Wo - 1) + 1, stride))
            dw4[:, a, b, :] = d2.T @ xp[sl].reshape(-1, C)
            dxp[sl] += dy @ w4[:, a, b, :]
    return dxp[:, pad:pad + H, pad:pad + W], dw4.reshape(Cout, -1)


def bn_fwd(x, g, b, eps):
    """Training-mode batch norm over (N, H, W) per channel, biased variance."""
    C = x.shape[-1]
    x2 = x.reshape(-1, C)
    mu = x2.mean(axis=0)
    var = ((x2 - mu) ** 2).mean(axis=0)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x2 - mu) * rstd
    y = xhat * g + b
    return y.reshape(x.shape), (xhat, rstd, g, x.shape)


def bn_bwd(dy, cache):
    """VJP of bn_fwd: the per-channel LayerNorm formula with the roles of rows
    and columns exchanged (statistics over the N * H * W rows)."""
    xhat, rstd, g, shape = cache
    d2 = dy.reshape(-1, shape[-1])
    gy = d2 * g
    dx = rstd * (gy - gy.mean(axis=0) - xhat * (gy * xhat).mean(axis=0))
    return dx.reshape(shape), (d2 * xhat).sum(axis=0), d2.sum(axis=0)


def maxpool_fwd(x, k=3, stride=2, pad=1):
    """Max over k x k windows (padding never wins); ties go to the first
    position in row-major window order."""
    N, H, W, C = x.shape
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    xp = np.full((N, H + 2 * pad, W + 2 * pad, C), -np.inf)
    xp[:, pad:pad + H, pad:pad + W] = x
    out = np.full((N, Ho, Wo, C), -np.inf)
    arg = np.zeros((N, Ho, Wo, C), np.int64)
    for a in range(k):
        for b in range(k):
            v = xp[:, a:a + stride * (Ho - 1) + 1:stride, b:b + stride * (Wo - 1) + 1:stride]
            better = v > out
            out = np.where(better, v, out)
            arg = np.where(better, a * k + b, arg)
    return out, (x.shape, arg, k, stride, pad)


def maxpool_bwd(dy, cache):
    (N, H, W, C), arg, k, stride, pad = cache
    _, Ho, Wo, _ = dy.shape
    dxp = np.zeros((N, H + 2 * pad, W + 2 * pad, C))
    for a in range(k):
        for b in range(k):
            sl = (slice(None), slice(a, a + stride * (Ho - 1) + 1, stride),
                  slice(b, b + stride * (Wo - 1) + 1, stride))
            dxp[sl] += np.where(arg == a * k + b, dy, 0.0)
    return dxp[:, pad:pad + H, pad:pad + W]


# ----------------------------------------------------------------------------
# Model
# ----------------------------------------------------------------------------

def forward(cfg, P, images, labels):
    """images [B, C, H, W], labels [B].  Returns (loss, cache); cache["acts"][i]
    is the input of block i (NHWC) and cache["acts"][n_blocks] the last block's
    output."""
    eps = cfg.ln_eps
    rnd = None if getattr(cfg, "operands", "fp64") == "fp64" else _rounder(cfg)
    x = np.transpose(np.asarray(images, np.float64), (0, 2, 3, 1))
    c = {"acts": [], "blocks": []}
    y, c["stem_conv"] = conv_fwd(x, P["stem.conv.w"], 7, 2, 3, rnd)
    y, c["stem_bn"] = bn_fwd(y, P["stem.bn.g"], P["stem.bn.b"], eps)
    c["stem_relu"] = y > 0
    y = np.maximum(y, 0.0)
    y, c["pool"] = maxpool_fwd(y)
    for i, _, cin, mid, cout, stride, proj in block_specs(cfg):
        p = f"b{i}."
        c["acts"].append(y)
        bc = {}
        h, bc["c1"] = conv_fwd(y, P[p + "conv1.w"], 1, 1, 0, rnd)
        h, bc["n1"] = bn_fwd(h, P[p + "bn1.g"], P[p + "bn1.b"], eps)
        bc["r1"] = h > 0
        h = np.maximum(h, 0.0)
        h, bc["c2"] = conv_fwd(h, P[p + "conv2.w"], 3, stride, 1, rnd)
        h, bc["n2"] = bn_fwd(h, P[p + "bn2.g"], P[p + "bn2.b"], eps)
        bc["r2"] = h > 0
        h = np.maximum(h, 0.0)
        h, bc["c3"] = conv_fwd(h, P[p + "conv3.w"], 1, 1, 0, rnd)
        h, bc["n3"] = bn_fwd(h, P[p + "bn3.g"], P[p + "bn3.b"], eps)
        if proj:
            s, bc["cd"] = conv_fwd(y, P[p + "down.w"], 1, stride, 0, rnd)
            s, bc["nd"] = bn_fwd(s, P[p + "down.bn.g"], P[p + "down.bn.b"], eps)
        else:
            s = y
        o = h + s
        bc["ro"] = o > 0
        y = np.maximum(o, 0.0)
        c["blocks"].append(bc)
    c["acts"].append(y)
    N, Hf, Wf, F = y.shape
    R_ = _rounder(cfg)
    feat = R_(y.reshape(N, Hf * Wf, F).mean(axis=1))
    c["feat_hw"] = (Hf, Wf)
    c["feat"] = feat
    z = feat @ R_(P["fc.w"]).T + P["fc.b"]
    c["logits"] = z
    loss, dz = L.cross_entropy(z, np.asarray(labels))
    c["dz"] = dz
    return loss, c


def backward(cfg, P, c):
    """Gradients of the trainable tensors (frozen ones are absent)."""
    k = cfg.frozen_layers
    G = {}
    R_ = _rounder(cfg)
    dz = R_(c["dz"])
    G["fc.w"] = dz.T @ c["feat"]
    G["fc.b"] = dz.sum(axis=0)
    dfeat = dz @ R_(P["fc.w"])
    Hf, Wf = c["feat_hw"]
    N, F = dfeat.shape
    dy = np.broadcast_to(dfeat[:, None, None, :] / (Hf * Wf), (N, Hf, Wf, F)).copy()
    specs = block_specs(cfg)
    for i, _, cin, mid, cout, stride, proj in reversed(specs):
        if i < k:
            return G
        p = f"b{i}."
        bc = c["blocks"][i]
        do = dy * bc["ro"]
        dh, G[p + "bn3.g"], G[p + "bn3.b"] = bn_bwd(do, bc["n3"])
        dh, G[p + "conv3.w"] = conv_bwd(dh, bc["c3"])
        dh = dh * bc["r2"]
        dh, G[p + "bn2.g"], G[p + "bn2.b"] = bn_bwd(dh, bc["n2"])
        dh, G[p + "conv2.w"] = conv_bwd(dh, bc["c2"])
        dh = dh * bc["r1"]
        dh, G[p + "bn1.g"], G[p + "bn1.b"] = bn_bwd(dh, bc["n1"])
        dx, G[p + "conv1.w"] = conv_bwd(dh, bc["c1"])
        if proj:
            ds, G[p + "down.bn.g"], G[p + "down.bn.b"] = bn_bwd(do, bc["nd"])
            dsx, G[p + "down.w"] = conv_bwd(ds, bc["cd"])
            dx = dx + dsx
        else:
            dx = dx + do
        dy = dx
    if k > 0:
        return G
    dy = maxpool_bwd(dy, c["pool"])
    dy = dy * c["stem_relu"]
    dy, G["stem.bn.g"], G["stem.bn.b"] = bn_bwd(dy, c["stem_bn"])
    _, G["stem.conv.w"] = conv_bwd(dy, c["stem_conv"])
    return G


def train_step(cfg, P, state, images, labels):
    """One step: forward, backward, AdamW on the trainable tensors.
    state: {} initially; holds m, v, t.  Returns (loss, grads, P', state, cache)."""
    loss, cache = forward(cfg, P, images, labels)
    G = backward(cfg, P, cache)
    train = trainable_mask(cfg)
    if not state:
        state = {"m": {n: np.zeros_like(v) for n, v in P.items()},
                 "v": {n: np.zeros_like(v) for n, v in P.items()}, "t": 0}
    t = state["t"] + 1
    newP, m, v = dict(P), dict(state["m"]), dict(state["v"])
    for n in P:
        if train[n]:
            newP[n], m[n], v[n] = adamw_update(cfg, P[n], G[n], state["m"][n], state["v"][n], t)
    return loss, G, newP, {"m": m, "v": v, "t": t}, cache


def eval_loss(cfg, P, images, labels):
    return forward(cfg, P, images, labels)[0]


def _flop_parts(cfg):
    """(stem, [per block], head) forward FLOPs, 2 per multiply-add."""
    H = cfg.img_size
    B = cfg.batch
    hs = (H + 6 - 7) // 2 + 1
    stem = 2.0 * B * hs * hs * 7 * 7 * cfg.channels * cfg.width
    hw = (hs + 2 - 3) // 2 + 1
    per_block = []
    for i, _, cin, mid, cout, stride, proj in block_specs(cfg):
        ho = (hw - 1) // stride + 1
        per_block.append(2.0 * B * (hw * hw * cin * mid + ho * ho * 9 * mid * mid + ho * ho * mid * cout
                                    + (ho * ho * cin * cout if proj else 0.0)))
        hw = ho
    feat = 4 * cfg.width * 2 ** (len(cfg.blocks) - 1)
    return stem, per_block, 2.0 * B * feat * cfg.classes


def forward_flops(cfg):
    stem, blocks, head = _flop_parts(cfg)
    return stem + sum(blocks) + head


def step_flops(cfg):
    """Algorithmic FLOPs of one step: 2 per multiply-add of every forward
    convolution and the head, twice that again for the input- and
    weight-gradient products of the trainable part (the stem's input gradient
    is never needed, so a trainable stem adds its weight gradient only)."""
    stem, blocks, head = _flop_parts(cfg)
    k = cfg.frozen_layers
    f = stem + sum(blocks) + head + 2.0 * sum(blocks[k:]) + 2.0 * head
    return f + (stem if k == 0 else 0.0)
