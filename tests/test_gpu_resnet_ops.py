"""Kernel-level parity of the ResNet workload's kernels against the float64
oracle's layer functions (oracle/resnet.py), on seeded inputs with ragged
sizes: convolution as im2col + GEMM (forward, input gradient through col2im,
weight gradient), training-mode batch norm forward and backward (with and
without a ReLU mask, channel counts below and above one 256-column slab, a
large common offset that a plain sum of squares would cancel), and the
3 x 3 / 2 max pool with its tie rule (the first maximum in row-major tap
order) and its gradient routing.

Convolution operands are rounded to bfloat16 on the host first, so both sides
multiply the same values: the remaining difference is fp32 against fp64
accumulation."""

import numpy as np
import pytest
import torch

from oracle import resnet as OR
from tests.gpu_util import bf16_round, flush, host, rel, to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def K():
    from paper_2309_01226_amd import ops
    return ops


CONV = [(2, 9, 7, 16, 24, 3, 1, 1), (3, 10, 11, 8, 16, 3, 2, 1), (2, 8, 9, 32, 40, 1, 2, 0),
        (2, 15, 13, 8, 16, 7, 2, 3), (1, 5, 5, 64, 64, 3, 1, 1)]


@pytest.mark.parametrize("N,H,W,C,Co,k,s,p", CONV)
def test_conv_via_im2col_gemm(N, H, W, C, Co, k, s, p):
    flush(f"conv N={N} H={H} W={W} C={C} Co={Co} k={k} s={s} p={p}")
    ops = K()
    rng = np.random.default_rng(N * 100 + H + k)
    x = bf16_round(rng.normal(size=(N, H, W, C)))
    w = bf16_round(rng.normal(size=(Co, k * k * C)))
    ref, cache = OR.conv_fwd(x, w, k, s, p)
    Ho, Wo = ref.shape[1], ref.shape[2]
    col = ops.im2col(to_dev_bf16(x.reshape(-1, C)), N, H, W, C, k, s, p)
    Kc = k * k * C
    out = torch.empty(N * Ho * Wo, Co, device="cuda", dtype=torch.float32)
    ops.gemm(col, to_dev_bf16(w), N * Ho * Wo, Co, Kc, out, lda=Kc, ldb=Kc)
    torch.cuda.synchronize()
    assert rel(host(out), ref.reshape(-1, Co)) < 2e-6
    # backward: dcol = dy W, dx = col2im(dcol); dW = dy^T col
    dy = bf16_round(rng.normal(size=ref.shape))
    rdx, rdw = OR.conv_bwd(dy, cache)
    dyd = to_dev_bf16(dy.reshape(-1, Co))
    wt = to_dev_bf16(np.ascontiguousarray(w.T))  # [Kc, Co]
    dcol = torch.empty(N * Ho * Wo, Kc, device="cuda", dtype=torch.float32)
    ops.gemm(dyd, wt, N * Ho * Wo, Kc, Co, dcol, lda=Co, ldb=Co)
    dx = ops.col2im(dcol, N, H, W, C, k, s, p)
    base = to_dev_f32(np.full((N * H * W, C), 0.5))
    ops.col2im(dcol, N, H, W, C, k, s, p, dx=base)
    dw = torch.empty(Co, Kc, device="cuda", dtype=torch.float32)
    ops.gemm(dyd, col, Co, Kc, N * Ho * Wo, dw, lda=Co, ldb=Kc, a_layout=ops.LAY_MN, b_layout=ops.LAY_MN)
    torch.cuda.synchronize()
    assert rel(host(dx), rdx.reshape(-1, C)) < 2e-6
    assert rel(host(base) - 0.5, rdx.reshape(-1, C)) < 2e-6
    assert rel(host(dw), rdw) < 2e-6


# im2col written transposed (the weight-gradient operand): bitwise the
# transpose of im2col, for pixel counts that are multiples of 8, ragged maps,
# strides 1 and 2, 3 x 3 and 1 x 1 (the projection subsample), and column
# counts that end inside a workgroup's 512-column block
IM2COL_T = [(4, 9, 6, 16, 3, 1, 1), (4, 10, 11, 8, 3, 2, 1), (2, 8, 8, 24, 1, 2, 0),
            (8, 14, 14, 72, 3, 1, 1), (1, 16, 16, 64, 3, 1, 1)]


@pytest.mark.parametrize("N,H,W,C,k,s,p", IM2COL_T)
def test_im2col_transposed(N, H, W, C, k, s, p):
    flush(f"im2col_t N={N} H={H} W={W} C={C} k={k} s={s} p={p}")
    ops = K()
    rng = np.random.default_rng(N + H + C + k)
    x = to_dev_bf16(rng.normal(size=(N * H * W, C)))
    col = ops.im2col(x, N, H, W, C, k, s, p)
    colT = ops.im2col_t(x, N, H, W, C, k, s, p)
    torch.cuda.synchronize()
    assert col.shape[0] % 8 == 0
    assert torch.equal(colT, col.t().contiguous())


BN = [(1000, 64, 0.0), (37, 8, 0.0), (5000, 512, 0.0), (200, 200, 0.0), (3000, 96, 1000.0)]


@pytest.mark.parametrize("P,C,offset", BN)
@pytest.mark.parametrize("relu", [0, 1])
def test_batchnorm_fwd_bwd(P, C, offset, relu):
    flush(f"batchnorm P={P} C={C} offset={offset} relu={relu}")
    ops = K()
    rng = np.random.default_rng(P + C + relu)
    x = (offset + rng.normal(0.3, 2.0, size=(P, C)) * rng.uniform(0.5, 2.0, size=C)).astype(np.float32)
    g = (1 + 0.3 * rng.normal(size=C)).astype(np.float32)
    b = (0.3 * rng.normal(size=C)).astype(np.float32)
    xd, gd, bd = to_dev_f32(x), to_dev_f32(g), to_dev_f32(b)
    y, yf, mean, rstd = ops.batchnorm_fwd(xd, gd, bd, 1e-5, relu=bool(relu))
    ry, cache = OR.bn_fwd(x.astype(np.float64), g, b, 1e-5)
    pre = ry
    if relu:
        ry = np.maximum(ry, 0.0)
    torch.cuda.synchronize()
    assert rel(host(mean), x.astype(np.float64).mean(axis=0)) < 1e-6
    assert rel(host(rstd), cache[1]) < 1e-5
    assert rel(host(yf), ry) < 2e-5
    assert rel(host(y), ry) < 4e-3
    dy = rng.normal(size=(P, C)).astype(np.float32)
    if relu:
        # through the ReLU, with the bf16 output (kind 1) and the fp32 one (kind 2) as the mask
        for mask in (y, yf):
            dx, dg, db = ops.batchnorm_bwd(to_dev_f32(dy), xd, mean, rstd, gd, mask=mask)
            gm = dy * (host(mask) > 0)
            rdx, rdg, rdb = OR.bn_bwd(gm.astype(np.float64), cache)
            torch.cuda.synchronize()
            assert rel(host(dx), rdx) < 4e-3 and rel(host(dg), rdg) < 1e-4 and rel(host(db), rdb) < 1e-5
        assert np.array_equal(host(y) > 0, pre > 0) or np.mean((host(y) > 0) != (pre > 0)) < 1e-4
    else:
        dx, dg, db = ops.batchnorm_bwd(to_dev_f32(dy), xd, mean, rstd, gd)
        rdx, rdg, rdb = OR.bn_bwd(dy.astype(np.float64), cache)
        torch.cuda.synchronize()
        assert rel(host(dx), rdx) < 4e-3 and rel(host(dg), rdg) < 1e-4 and rel(host(db), rdb) < 1e-5


POOL = [(2, 8, 8, 16), (3, 9, 7, 8), (1, 112, 112, 4), (2, 2, 3, 5)]


@pytest.mark.parametrize("N,H,W,C", POOL)
def test_maxpool(N, H, W, C):
    flush(f"maxpool N={N} H={H} W={W} C={C}")
    ops = K()
    rng = np.random.default_rng(N + H + W + C)
    for x in (rng.normal(size=(N, H, W, C)).astype(np.float32),
              np.maximum(rng.normal(size=(N, H, W, C)), 0).astype(np.float32),  # ties at zero
              np.full((N, H, W, C), 0.25, np.float32)):                         # all ties
        ry, cache = OR.maxpool_fwd(x.astype(np.float64))
        y, yb, arg = ops.maxpool_fwd(to_dev_f32(x.reshape(-1, C)), N, H, W, C)
        dy = rng.normal(size=ry.shape).astype(np.float32)
        dx = ops.maxpool_bwd(to_dev_f32(dy.reshape(-1, C)), arg, N, H, W, C)
        torch.cuda.synchronize()
        assert np.array_equal(host(y), ry.reshape(-1, C))
        assert np.array_equal(arg.cpu().numpy().astype(np.int64), cache[1].reshape(-1, C))
        assert rel(host(dx), OR.maxpool_bwd(dy.astype(np.float64), cache).reshape(-1, C)) < 1e-6
