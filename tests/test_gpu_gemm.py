"""GEMM kernel parity against the float64 matmul of the same bf16 operands,
over all operand layouts and epilogues, at shapes that span several tiles with
ragged edges, and the unaligned (scalar-load) path."""

import numpy as np
import pytest
import torch

from oracle import ops as O
from tests.gpu_util import bf16_round, flush, host, rel, to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def _operands(rng, M, N, K, a_layout, b_layout):
    A = bf16_round(rng.normal(size=(M, K)))
    B = bf16_round(rng.normal(size=(N, K)))
    Ad = to_dev_bf16(A if a_layout == 0 else A.T.copy())
    Bd = to_dev_bf16(B if b_layout == 0 else B.T.copy())
    lda = K if a_layout == 0 else M
    ldb = K if b_layout == 0 else N
    return A, B, Ad, Bd, lda, ldb


SHAPES = [(64, 64, 64), (300, 200, 136), (513, 257, 520), (256, 128, 64), (8, 8, 8), (1000, 40, 16)]


@pytest.mark.parametrize("a_layout,b_layout", [(0, 0), (0, 1), (1, 1), (1, 0)])
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_f32_layouts(a_layout, b_layout, M, N, K):
    from paper_2309_01226_amd import ops
    flush(f"gemm f32 lay=({a_layout},{b_layout}) M={M} N={N} K={K}")
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, a_layout, b_layout)
    bias = rng.normal(size=N)
    out = torch.empty(M, N, device="cuda", dtype=torch.float32)
    ops.gemm(Ad, Bd, M, N, K, out, lda=lda, ldb=ldb, a_layout=a_layout, b_layout=b_layout,
             bias=to_dev_f32(bias))
    torch.cuda.synchronize()
    ref = O.gemm(A, B) + bias
    assert rel(host(out), ref) < 2e-6


@pytest.mark.parametrize("M,N,K", [(300, 200, 100), (77, 45, 588), (129, 65, 37)])
def test_gemm_unaligned_scalar_path(M, N, K):
    from paper_2309_01226_amd import ops
    flush(f"gemm unaligned M={M} N={N} K={K}")
    rng = np.random.default_rng(5)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, 0, 0)
    out = torch.empty(M, N, device="cuda", dtype=torch.float32)
    ops.gemm(Ad, Bd, M, N, K, out, lda=lda, ldb=ldb)
    torch.cuda.synchronize()
    assert rel(host(out), O.gemm(A, B)) < 2e-6


@pytest.mark.parametrize("erf_form", [0, 1])
def test_gemm_epilogues(erf_form):
    from paper_2309_01226_amd import ops
    M, N, K = 390, 272, 200
    flush(f"gemm epilogues erf={erf_form}")
    rng = np.random.default_rng(11)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, 0, 0)
    C = O.gemm(A, B)
    bias = rng.normal(size=N - 40)
    # residual add into fp32, resid aliasing out
    R = rng.normal(size=(M, N))
    out = to_dev_f32(R)
    ops.gemm(Ad, Bd, M, N, K, out, lda=lda, ldb=ldb, epilogue=1, resid=out,
             bias=to_dev_f32(bias), bias_col0=40)
    torch.cuda.synchronize()
    ref = R + C
    ref[:, 40:] += bias
    assert rel(host(out), ref) < 2e-6
    # bf16 store with bias from column 40 and GELU of columns >= 100 into out2
    o1 = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
    o2 = torch.empty(M, N - 100, device="cuda", dtype=torch.bfloat16)
    ops.gemm(Ad, Bd, M, N, K, o1, lda=lda, ldb=ldb, epilogue=2, bias=to_dev_f32(bias),
             bias_col0=40, out2=o2, ldo2=N - 100, gelu_col0=100, gelu_erf=erf_form)
    torch.cuda.synchronize()
    pre = C.copy()
    pre[:, 40:] += bias
    assert rel(host(o1), pre) < 4e-3
    assert rel(host(o2), O.gelu(pre[:, 100:], erf_form)) < 4e-3
    # GELU-backward epilogue
    U = bf16_round(rng.normal(size=(M, N)))
    o3 = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
    ops.gemm(Ad, Bd, M, N, K, o3, lda=lda, ldb=ldb, epilogue=3, aux=to_dev_bf16(U), ldaux=N,
             gelu_erf=erf_form)
    torch.cuda.synchronize()
    assert rel(host(o3), C * O.gelu_grad(U, erf_form)) < 4e-3


@pytest.mark.parametrize("a_layout,b_layout", [(0, 0), (0, 1), (1, 1), (1, 0)])
@pytest.mark.parametrize("epi", [0, 1, 2, 3])
def test_gemm_large_tiles_sampled(a_layout, b_layout, epi):
    """Shapes large enough for the 256 x 256 four-stage path (>= 256 tiles),
    with ragged M and N edges and a K tail, every epilogue; checked on 300
    sampled rows (always including the last) against float64."""
    from paper_2309_01226_amd import ops
    M, N, K = 4100, 4104, 584
    flush(f"gemm large lay=({a_layout},{b_layout}) epi={epi}")
    rng = np.random.default_rng(17 + a_layout + 2 * b_layout + 4 * epi)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, a_layout, b_layout)
    bias = rng.normal(size=N - 8)
    rows = np.sort(rng.choice(M - 1, size=299, replace=False))
    rows = np.append(rows, M - 1)
    C = O.gemm(A[rows], B)
    pre = C.copy()
    pre[:, 8:] += bias
    kw = dict(lda=lda, ldb=ldb, a_layout=a_layout, b_layout=b_layout, epilogue=epi)
    if epi == 0:
        out = torch.empty(M, N, device="cuda", dtype=torch.float32)
        ops.gemm(Ad, Bd, M, N, K, out, bias=to_dev_f32(bias), bias_col0=8, **kw)
        torch.cuda.synchronize()
        assert rel(host(out)[rows], pre) < 2e-6
    elif epi == 1:
        R = rng.normal(size=(M, N)).astype(np.float32)
        out = to_dev_f32(R)
        ops.gemm(Ad, Bd, M, N, K, out, resid=out, bias=to_dev_f32(bias), bias_col0=8, **kw)
        torch.cuda.synchronize()
        assert rel(host(out)[rows], R[rows] + pre) < 2e-6
    elif epi == 2:
        o1 = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        o2 = torch.empty(M, N - 512, device="cuda", dtype=torch.bfloat16)
        ops.gemm(Ad, Bd, M, N, K, o1, bias=to_dev_f32(bias), bias_col0=8, out2=o2, ldo2=N - 512,
                 gelu_col0=512, **kw)
        torch.cuda.synchronize()
        assert rel(host(o1)[rows], pre) < 4e-3
        assert rel(host(o2)[rows], O.gelu(pre[:, 512:], 0)) < 4e-3
    else:
        U = bf16_round(rng.normal(size=(M, N)))
        o3 = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        ops.gemm(Ad, Bd, M, N, K, o3, aux=to_dev_bf16(U), ldaux=N, gelu_erf=1, **kw)
        torch.cuda.synchronize()
        assert rel(host(o3)[rows], C * O.gelu_grad(U[rows], 1)) < 4e-3


# Split-K: fp32-output products with fewer than 256 tiles of 256 x 256 and
# K >= 1024, given a workspace.  Shapes: one tile, ragged M / N, a K that is
# not a multiple of the slice depth (last slice shorter) and not a multiple of
# 64, and a residual + bias epilogue with the residual aliasing the output.
SPLITK = [(256, 256, 2048, 0), (300, 520, 4160, 0), (768, 768, 8192, 0), (520, 264, 3008, 1),
          (1000, 40, 1032, 1)]


@pytest.mark.parametrize("M,N,K,resid", SPLITK)
def test_gemm_splitk(M, N, K, resid):
    from paper_2309_01226_amd import ops
    flush(f"gemm split-K M={M} N={N} K={K} resid={resid}")
    rng = np.random.default_rng(M + N + K)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, 0, 0)
    bias = rng.normal(size=N)
    R = rng.normal(size=(M, N))
    ws = torch.full((16 * M * N,), float("nan"), device="cuda", dtype=torch.float32)
    out = to_dev_f32(R) if resid else torch.empty(M, N, device="cuda", dtype=torch.float32)
    kw = dict(bias=to_dev_f32(bias), epilogue=ops.EPI_RESID_F32 if resid else ops.EPI_F32)
    if resid:
        kw.update(resid=out, ldr=N)
    ops.gemm(Ad, Bd, M, N, K, out, lda=lda, ldb=ldb, splitk_ws=ws, **kw)
    # the same product without a workspace (no split)
    out1 = to_dev_f32(R) if resid else torch.empty(M, N, device="cuda", dtype=torch.float32)
    if resid:
        kw.update(resid=out1)
    ops.gemm(Ad, Bd, M, N, K, out1, lda=lda, ldb=ldb, **kw)
    torch.cuda.synchronize()
    ref = O.gemm(A, B) + bias + (R if resid else 0.0)
    got = host(out)
    assert np.isfinite(got).all()
    assert rel(got, ref) < 2e-6
    assert rel(got, host(out1)) < 2e-6
    # the split path ran: at least two slices of partial products were written
    n_used = int(torch.isfinite(ws).sum().item())
    assert n_used >= 2 * M * N, n_used


# Tail split: fp32-output products with more than 256 tiles of 256 x 256 whose
# last round would run mostly empty (ViT-H/14's 16448 x 1280 products have 325
# tiles), given a workspace: whole rounds of rows unsplit, the remaining rows
# split-K, then the reduction with bias and residual.  Shapes: the ViT-H
# products, a ragged last row tile, ragged columns, and a second shape family.
TAIL = [(16448, 1280, 5120, 1), (16448, 1280, 1280, 0), (16400, 1280, 3840, 1),
        (16448, 1272, 5120, 0), (9000, 2048, 2048, 1)]


@pytest.mark.parametrize("M,N,K,resid", TAIL)
def test_gemm_tail_split(M, N, K, resid):
    from paper_2309_01226_amd import ops
    flush(f"gemm tail split M={M} N={N} K={K} resid={resid}")
    rng = np.random.default_rng(M + N + K + 1)
    A, B, Ad, Bd, lda, ldb = _operands(rng, M, N, K, 0, 0)
    bias = rng.normal(size=N)
    R = rng.normal(size=(M, N)).astype(np.float32)
    ws = torch.full((16 * 1024 * 1024,), float("nan"), device="cuda", dtype=torch.float32)
    out = to_dev_f32(R) if resid else torch.empty(M, N, device="cuda", dtype=torch.float32)
    kw = dict(bias=to_dev_f32(bias), epilogue=ops.EPI_RESID_F32 if resid else ops.EPI_F32)
    if resid:
        kw.update(resid=out, ldr=N)
    ops.gemm(Ad, Bd, M, N, K, out, lda=lda, ldb=ldb, splitk_ws=ws, **kw)
    out1 = to_dev_f32(R) if resid else torch.empty(M, N, device="cuda", dtype=torch.float32)
    if resid:
        kw.update(resid=out1)
    ops.gemm(Ad, Bd, M, N, K, out1, lda=lda, ldb=ldb, **kw)
    torch.cuda.synchronize()
    got = host(out)
    assert np.isfinite(got).all()
    # rows from the unsplit head, from the split tail and the last row
    head_rows = rng.choice(M // 2, size=150, replace=False)
    tail_rows = M - 1 - rng.choice(2048, size=150, replace=False)
    rows = np.unique(np.concatenate([head_rows, tail_rows, [M - 1]]))
    ref = O.gemm(A[rows], B) + bias + (R[rows].astype(np.float64) if resid else 0.0)
    assert rel(got[rows], ref) < 2e-6
    assert rel(got, host(out1)) < 2e-6
    # the tail ran split-K: partials of at least two slices were written, but
    # fewer than a split of every row would write
    n_used = int(torch.isfinite(ws).sum().item())
    assert 2 * N * 16 <= n_used < 2 * M * N, n_used
