"""Kernel-level parity on the GPU against the float64 oracle references, on
seeded inputs that span several tiles and ragged tails, plus edge cases."""

import math

import numpy as np
import pytest
import torch

from oracle import ops as O
from tests.gpu_util import bf16_round, flush, host, rel, to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def ops():
    from paper_2309_01226_amd import ops as K
    return K


# ------------------------------------------------------------------ LayerNorm

# The wide-row forward runs at most 2048 workgroups that walk rows with a
# stride of the grid and load the next row before storing the current one:
# 4096 and 16448 rows (GPT-J, ViT-H/14 per step), 5000 and 2049 rows (not a
# multiple of 2048: the last rows of the walk belong to some workgroups only).
@pytest.mark.parametrize("rows,d", [(1, 64), (37, 768), (300, 1280), (64, 4096), (5, 16),
                                    (9, 1028), (4096, 4096), (16448, 1280), (5000, 1280),
                                    (2049, 4096)])
def test_layernorm_fwd_bwd(rows, d):
    flush(f"layernorm rows={rows} d={d}")
    rng = np.random.default_rng(rows + d)
    x = rng.normal(0.5, 2.0, size=(rows, d)).astype(np.float32)
    g = (1 + 0.3 * rng.normal(size=d)).astype(np.float32)
    b = (0.3 * rng.normal(size=d)).astype(np.float32)
    xd, gd, bd = to_dev_f32(x), to_dev_f32(g), to_dev_f32(b)
    y = torch.empty(rows, d, device="cuda", dtype=torch.bfloat16)
    mean = torch.empty(rows, device="cuda")
    rstd = torch.empty(rows, device="cuda")
    ops().layernorm_fwd(xd, gd, bd, y, mean, rstd, rows, d, 1e-5)
    dy = rng.normal(size=(rows, d)).astype(np.float32)
    r0 = rng.normal(size=(rows, d)).astype(np.float32)
    dres = to_dev_f32(r0)
    dg = torch.empty(d, device="cuda")
    db = torch.empty(d, device="cuda")
    ops().layernorm_bwd(to_dev_f32(dy), xd, gd, mean, rstd, dres, dg, db, rows, d)
    torch.cuda.synchronize()
    ry, rmean, rrstd = O.layernorm_fwd(x, g, b, 1e-5)
    assert rel(host(y), ry) < 4e-3
    assert rel(host(mean), rmean) < 1e-5 and rel(host(rstd), rrstd) < 1e-5
    rdx, rdg, rdb = O.layernorm_bwd(dy, x, g, 1e-5)
    assert rel(host(dres) - r0, rdx) < 1e-4
    assert rel(host(dg), rdg) < 1e-5 and rel(host(db), rdb) < 1e-5


def test_layernorm_fwd_widest():
    """The widest row the forward accepts (8192; the backward stops at 4096)."""
    rng = np.random.default_rng(11)
    rows, d = 3, 8192
    x = rng.normal(-0.2, 1.5, size=(rows, d)).astype(np.float32)
    g = (1 + 0.3 * rng.normal(size=d)).astype(np.float32)
    b = (0.3 * rng.normal(size=d)).astype(np.float32)
    y = torch.empty(rows, d, device="cuda", dtype=torch.bfloat16)
    mean = torch.empty(rows, device="cuda")
    rstd = torch.empty(rows, device="cuda")
    ops().layernorm_fwd(to_dev_f32(x), to_dev_f32(g), to_dev_f32(b), y, mean, rstd, rows, d, 1e-5)
    torch.cuda.synchronize()
    ry, rmean, rrstd = O.layernorm_fwd(x, g, b, 1e-5)
    assert rel(host(y), ry) < 4e-3
    assert rel(host(mean), rmean) < 1e-5 and rel(host(rstd), rrstd) < 1e-5


@pytest.mark.parametrize("d,B,S", [(128, 7, 5), (1280, 7, 5), (1280, 64, 257), (4096, 3000, 2)])
def test_layernorm_strided_rows(d, B, S):
    """Rows picked with a stride (the ViT head normalises only the CLS rows);
    widths below and above 1024 take the one-wave and one-workgroup row
    kernels; 3000 strided rows of 4096 run the multi-row walk of the latter."""
    flush(f"layernorm strided rows d={d} rows={B} stride={S}")
    rng = np.random.default_rng(3 + B)
    x = rng.normal(size=(B * S, d)).astype(np.float32)
    g = np.ones(d, np.float32)
    b = np.zeros(d, np.float32)
    y = torch.empty(B, d, device="cuda", dtype=torch.bfloat16)
    mean = torch.empty(B, device="cuda")
    rstd = torch.empty(B, device="cuda")
    ops().layernorm_fwd(to_dev_f32(x), to_dev_f32(g), to_dev_f32(b), y, mean, rstd, B, d, 1e-5,
                        row_stride=S)
    torch.cuda.synchronize()
    assert rel(host(y), O.layernorm_fwd(x[::S], g, b, 1e-5)[0]) < 4e-3


# ------------------------------------------------------------------ attention

def _qkv(rng, B, H, S, dh):
    d = H * dh
    buf = bf16_round(rng.normal(size=(B * S, 3 * d)))
    q = buf[:, :d].reshape(B, S, H, dh).transpose(0, 2, 1, 3)
    k = buf[:, d:2 * d].reshape(B, S, H, dh).transpose(0, 2, 1, 3)
    v = buf[:, 2 * d:].reshape(B, S, H, dh).transpose(0, 2, 1, 3)
    return buf, q, k, v


def _merge(x):
    B, H, S, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B * S, H * dh)


ATTN = [(2, 3, 100, 16, True), (1, 2, 257, 80, False), (2, 2, 300, 64, True), (1, 2, 160, 256, True),
        (1, 1, 1, 64, True), (1, 2, 129, 128, False), (2, 1, 70, 32, False),
        # pipelined kernels: several 32-row blocks, ragged tails, both masks
        (2, 1, 520, 256, True), (1, 2, 97, 256, False), (1, 1, 5, 256, True), (2, 2, 333, 128, True),
        (1, 3, 200, 64, False), (1, 1, 31, 128, True),
        # 64- and 80-wide heads: several 128-row workgroups, diagonal and tail
        # blocks, single-key tails (257 = 4 x 64 + 1), empty waves
        (2, 3, 640, 64, True), (1, 1, 33, 64, False), (1, 2, 257, 64, True), (3, 2, 513, 80, True),
        (2, 2, 190, 80, True), (2, 2, 1, 80, False), (1, 2, 385, 80, False)]


@pytest.mark.parametrize("B,H,S,dh,causal", ATTN)
def test_attention_fwd_bwd(B, H, S, dh, causal):
    flush(f"attention B={B} H={H} S={S} dh={dh} causal={causal}")
    rng = np.random.default_rng(S * dh + H)
    d = H * dh
    buf, q, k, v = _qkv(rng, B, H, S, dh)
    qkv = to_dev_bf16(buf)
    o = torch.empty(B * S, d, device="cuda", dtype=torch.bfloat16)
    lse = torch.empty(B * H * S, device="cuda")
    scale = 1.0 / math.sqrt(dh)
    K = ops()
    K.attention_fwd(qkv, qkv[:, d:], qkv[:, 2 * d:], o, lse, B, H, S, dh, causal, scale,
                    ldq=3 * d, ldk=3 * d, ldv=3 * d, ldo=d)
    torch.cuda.synchronize()
    ro, rlse, probs = O.attention(q, k, v, causal)
    assert rel(host(o), _merge(ro)) < 1e-2
    assert np.max(np.abs(host(lse).reshape(B, H, S) - rlse)) < 1e-4 * max(1.0, np.abs(rlse).max())
    do = bf16_round(rng.normal(size=(B * S, d)))
    dq = torch.empty(B * S, 3 * d, device="cuda", dtype=torch.bfloat16)
    K.attention_bwd(qkv, qkv[:, d:], qkv[:, 2 * d:], o, lse, to_dev_bf16(do), dq, dq[:, d:],
                    dq[:, 2 * d:], B, H, S, dh, causal, scale, ldq=3 * d, ldk=3 * d, ldv=3 * d,
                    ldo=d, lddo=d, lddq=3 * d, lddk=3 * d, lddv=3 * d)
    torch.cuda.synchronize()
    dos = do.reshape(B, S, H, dh).transpose(0, 2, 1, 3)
    rdq, rdk, rdv = O.attention_bwd(dos, q, k, v, probs)
    got = host(dq)
    # With one visible key the softmax is constant, so the true dq and dk are
    # exactly zero; the GPU returns rounding noise of dP - rowsum(dO * O).
    # Errors are therefore measured against max(|ref|, 1e-3 |dO| |K|).
    floor = 1e-3 * np.linalg.norm(do) * np.linalg.norm(buf[:, d:2 * d]) / math.sqrt(B * S)
    for part, ref in ((0, rdq), (1, rdk), (2, rdv)):
        err = np.linalg.norm(got[:, part * d:(part + 1) * d] - _merge(ref))
        assert err <= 2e-2 * max(np.linalg.norm(ref), floor), (part, err, np.linalg.norm(ref))


# Attention at the full per-layer shapes the step launches (GPT-J, GPT-2-small,
# ViT-H/14, a grid member at batch 16), checked on sampled heads (the first
# and the last (batch, head) plus one in between) against the oracle.
FULL_ATTN = [(2, 16, 2048, 256, True), (8, 12, 1024, 64, True), (64, 16, 257, 80, False),
             (16, 16, 512, 64, True)]


@pytest.mark.parametrize("B,H,S,dh,causal", FULL_ATTN)
def test_attention_full_size_sampled(B, H, S, dh, causal):
    flush(f"attention full size B={B} H={H} S={S} dh={dh} causal={causal}")
    rng = np.random.default_rng(B * H + S)
    d = H * dh
    buf = rng.standard_normal(size=(B * S, 3 * d), dtype=np.float32)
    buf = bf16_round(buf)
    qkv = to_dev_bf16(buf)
    o = torch.empty(B * S, d, device="cuda", dtype=torch.bfloat16)
    lse = torch.empty(B * H * S, device="cuda")
    scale = 1.0 / math.sqrt(dh)
    K = ops()
    K.attention_fwd(qkv, qkv[:, d:], qkv[:, 2 * d:], o, lse, B, H, S, dh, causal, scale,
                    ldq=3 * d, ldk=3 * d, ldv=3 * d, ldo=d)
    do = bf16_round(rng.standard_normal(size=(B * S, d), dtype=np.float32))
    dq = torch.empty(B * S, 3 * d, device="cuda", dtype=torch.bfloat16)
    K.attention_bwd(qkv, qkv[:, d:], qkv[:, 2 * d:], o, lse, to_dev_bf16(do), dq, dq[:, d:],
                    dq[:, 2 * d:], B, H, S, dh, causal, scale, ldq=3 * d, ldk=3 * d, ldv=3 * d,
                    ldo=d, lddo=d, lddq=3 * d, lddk=3 * d, lddv=3 * d)
    torch.cuda.synchronize()
    go, glse, gd = host(o), host(lse).reshape(B, H, S), host(dq)
    for b, h in ((0, 0), (B // 2, H // 3), (B - 1, H - 1)):
        rows = slice(b * S, (b + 1) * S)
        part = lambda x, j: x[rows, j * d + h * dh: j * d + (h + 1) * dh].astype(np.float64)[None, None]
        q, k, v = part(buf, 0), part(buf, 1), part(buf, 2)
        ro, rlse, probs = O.attention(q, k, v, causal)
        assert rel(go[rows, h * dh:(h + 1) * dh], ro[0, 0]) < 1e-2, (b, h)
        assert np.max(np.abs(glse[b, h] - rlse[0, 0])) < 1e-4 * max(1.0, np.abs(rlse).max()), (b, h)
        dos = do[rows, h * dh:(h + 1) * dh].astype(np.float64)[None, None]
        rdq, rdk, rdv = O.attention_bwd(dos, q, k, v, probs)
        for j, ref in ((0, rdq), (1, rdk), (2, rdv)):
            err = np.linalg.norm(gd[rows, j * d + h * dh: j * d + (h + 1) * dh] - ref[0, 0])
            assert err <= 2e-2 * np.linalg.norm(ref), (b, h, j, err, np.linalg.norm(ref))


# ------------------------------------------------------------------ rotary

# rd % 8 == 0 takes the 16-byte kernel, other even rd the per-pair one
@pytest.mark.parametrize("inverse", [False, True])
@pytest.mark.parametrize("dh,rd", [(32, 8), (32, 6), (256, 64)])
def test_rotary(inverse, dh, rd):
    rng = np.random.default_rng(21)
    B, S, H = 2, 300, 3
    d = H * dh
    buf = bf16_round(rng.normal(size=(B * S, 3 * d)))
    dev = to_dev_bf16(buf)
    ops().rotary(dev, 3 * d, B, S, H, dh, rd, inverse)
    torch.cuda.synchronize()
    got = host(dev)
    for part in range(2):
        x = buf[:, part * d:(part + 1) * d].reshape(B, S, H, dh).transpose(0, 2, 1, 3)
        ref = _merge(O.rope(x, rd, inverse))
        assert rel(got[:, part * d:(part + 1) * d], ref) < 4e-3
    assert np.array_equal(got[:, 2 * d:], buf[:, 2 * d:])  # v untouched


# ------------------------------------------------------------------ cross-entropy

# Rows of at most 53248 logits with 16-byte aligned rows stay in registers:
# 512 threads for up to 12 groups of 2048 and for exactly 25 (the GPT
# vocabularies, where only the last group can be ragged), 1024 threads for
# the rest; wider or unaligned rows take the streaming kernel.  `pad` gives
# the rows a leading dimension rounded up to 8 (as the model's logits have),
# whose padding columns the kernel zeroes in dz.
@pytest.mark.parametrize("N,V,pad", [
    (7, 50257, True), (7, 50400, False), (3, 49153, True),   # 512 x 25, last group ragged
    (64, 512, False), (3, 1000, False), (6, 6000, False),     # 512 x 1, 512 x 4
    (5, 16000, False), (3, 20481, True),                      # 512 x 8, 512 x 12
    (4, 40000, False), (5, 53248, False), (3, 51201, True),   # 1024 x 13
    (4, 53256, False), (7, 50257, False)])                    # streaming kernel
def test_cross_entropy(N, V, pad):
    flush(f"xent N={N} V={V} pad={pad}")
    rng = np.random.default_rng(N + V)
    z = rng.normal(0, 3, size=(N, V)).astype(np.float32)
    lab = rng.integers(0, V, size=N).astype(np.int32)
    lab[1] = -1
    lab[2] = V - 1
    ld = (V + 7) // 8 * 8 if pad else V
    zd = torch.zeros(N, ld, device="cuda")
    zd[:, :V] = to_dev_f32(z)
    row = torch.empty(N, device="cuda")
    dz = torch.full((N, ld), 7.0, device="cuda", dtype=torch.bfloat16)
    inv_n = torch.empty(1, device="cuda")
    ops().cross_entropy(zd, torch.as_tensor(lab).cuda(), row, dz, inv_n, N, V, ldz=ld, lddz=ld)
    torch.cuda.synchronize()
    rrow, rdz, _ = O.cross_entropy(z, lab)
    assert rel(host(row), rrow) < 1e-5
    got = host(dz)
    assert rel(got[:, :V], rdz) < 4e-3
    assert np.all(got[:, V:] == 0.0)
    assert abs(host(inv_n)[0] * (N - 1) - 1.0) < 1e-7


# ------------------------------------------------------------------ AdamW

@pytest.mark.parametrize("n", [1, 7, 4099, 1 << 20])
def test_adamw_against_oracle(n):
    rng = np.random.default_rng(n)
    p = rng.normal(0, 0.02, n).astype(np.float32)
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    m = rng.normal(0, 1e-4, n).astype(np.float32)
    v = np.abs(rng.normal(0, 1e-6, n)).astype(np.float32)
    pd, gd, md, vd = map(to_dev_f32, (p, g, m, v))
    sh = torch.empty(n, device="cuda", dtype=torch.bfloat16)
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01)
    ops().adamw(pd, gd, md, vd, sh, n, t=3, **hp)
    torch.cuda.synchronize()
    rp, rm, rv = O.adamw(p, g, m, v, 3, **hp)
    assert rel(host(pd), rp) < 1e-6 and rel(host(md), rm) < 1e-6 and rel(host(vd), rv) < 1e-6
    assert np.array_equal(host(sh), bf16_round(host(pd)))


# ------------------------------------------------------------------ embedding

# 40000 positions: three sort chunks of at most 16384, the later ones added in order
@pytest.mark.parametrize("T,d,V", [(64, 64, 512), (1000, 256, 97), (4096, 128, 50400), (40000, 64, 300)])
def test_embedding(T, d, V):
    flush(f"embedding T={T} d={d} V={V}")
    rng = np.random.default_rng(T)
    S = 32
    wte = rng.normal(size=(V, d)).astype(np.float32)
    wpe = rng.normal(size=(S, d)).astype(np.float32)
    tok = rng.integers(0, V, size=T).astype(np.int32)
    tok[:5] = tok[5]  # repeated ids
    h = torch.empty(T, d, device="cuda")
    tokd = torch.as_tensor(tok).cuda()
    ops().embed_fwd(tokd, to_dev_f32(wte), to_dev_f32(wpe), h, T, S, d, V)
    dh = rng.normal(size=(T, d)).astype(np.float32)
    dw = torch.full((V, d), 7.0, device="cuda")
    ops().embed_bwd(tokd, to_dev_f32(dh), dw, T, d, V)
    torch.cuda.synchronize()
    assert np.array_equal(host(h), (wte[tok] + wpe[np.arange(T) % S]).astype(np.float32))
    assert rel(host(dw), O.embed_bwd(tok, dh, V)) < 1e-6


def test_colsum():
    rng = np.random.default_rng(2)
    X = rng.normal(size=(1000, 333)).astype(np.float32)
    out = torch.empty(333, device="cuda")
    ops().colsum(to_dev_f32(X), out, 1000, 333)
    torch.cuda.synchronize()
    assert rel(host(out), X.astype(np.float64).sum(axis=0)) < 1e-5


# ------------------------------------------------------------------ transpose

@pytest.mark.parametrize("rows,cols,pad_s,pad_d", [(8, 8, 0, 0), (136, 72, 8, 0), (256, 384, 0, 16),
                                                   (1000, 24, 0, 0), (24, 1000, 8, 8)])
def test_transpose_bf16(rows, cols, pad_s, pad_d):
    flush(f"transpose rows={rows} cols={cols} pads={pad_s},{pad_d}")
    g = torch.Generator().manual_seed(rows * 7 + cols)
    lds, ldd = cols + pad_s, rows + pad_d
    src = torch.randn(rows, lds, generator=g).to(torch.bfloat16).cuda()
    # the padding columns of dst must be left as they were
    dst = torch.full((cols, ldd), 7.0, dtype=torch.bfloat16).cuda()
    ops().transpose_bf16(src, dst, rows, cols, lds=lds, ldd=ldd)
    torch.cuda.synchronize()
    s, d_ = src.cpu(), dst.cpu()
    assert torch.equal(d_[:, :rows], s[:, :cols].t())
    assert bool((d_[:, rows:] == 7.0).all())


def test_transpose_bf16_rejects_ragged():
    from paper_2309_01226_amd._lib import SatError
    src = torch.zeros(12, 16, dtype=torch.bfloat16, device="cuda")
    dst = torch.zeros(16, 16, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(SatError):
        ops().transpose_bf16(src, dst, 12, 16)
