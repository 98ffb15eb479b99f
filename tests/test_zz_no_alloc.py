"""sat_op_gemm_noalloc: the split-K product without a caller workspace.

The call keeps its split-K partials in the library's per-device scratch
array instead of a workspace argument.  Its result must be bitwise that of
sat_op_gemm given a workspace (same slice plan, same kernels, same summation
order), and within the split-K test's tolerance of the float64 product.
Two calls in a row, the second on a smaller product, check that nothing of
the first call's partials leaks into the second.  A product whose partials
would not fit the scratch is refused on the host, before any launch.
"""

import numpy as np
import pytest
import torch

from oracle import ops as O
from tests.gpu_util import bf16_round, flush, host, rel, to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def _case(rng, M, N, K, resid):
    from paper_2309_01226_amd import ops
    A = bf16_round(rng.normal(size=(M, K)))
    B = bf16_round(rng.normal(size=(N, K)))
    bias = rng.normal(size=N)
    R = rng.normal(size=(M, N))
    Ad, Bd = to_dev_bf16(A), to_dev_bf16(B)
    kw = dict(lda=K, ldb=K, bias=to_dev_f32(bias),
              epilogue=ops.EPI_RESID_F32 if resid else ops.EPI_F32)

    def fresh():
        return to_dev_f32(R) if resid else torch.empty(M, N, device="cuda", dtype=torch.float32)

    ref = O.gemm(A, B) + bias + (R if resid else 0.0)
    return Ad, Bd, kw, fresh, ref


def _check(M, N, K, resid, seed):
    from paper_2309_01226_amd import ops
    flush(f"no-alloc gemm M={M} N={N} K={K} resid={resid}")
    rng = np.random.default_rng(seed)
    Ad, Bd, kw, fresh, ref = _case(rng, M, N, K, resid)
    out_na = fresh()
    extra = dict(resid=out_na, ldr=N) if resid else {}
    ops.gemm_noalloc(Ad, Bd, M, N, K, out_na, **kw, **extra)
    ws = torch.full((16 * M * N,), float("nan"), device="cuda", dtype=torch.float32)
    out_ws = fresh()
    extra = dict(resid=out_ws, ldr=N) if resid else {}
    ops.gemm(Ad, Bd, M, N, K, out_ws, splitk_ws=ws, **kw, **extra)
    torch.cuda.synchronize()
    got = host(out_na)
    assert np.isfinite(got).all()
    assert torch.equal(out_na, out_ws), "differs from sat_op_gemm with a workspace"
    assert rel(got, ref) < 2e-6
    # the workspace path really split K (so the scratch path was exercised)
    assert int(torch.isfinite(ws).sum().item()) >= 2 * M * N


def test_noalloc_two_calls_second_smaller():
    # 6 output tiles, K 8192: 16 slices of 512, 6.3 M partials (of the 8 M scratch)
    _check(512, 768, 8192, resid=True, seed=1)
    # smaller, ragged, plain epilogue: fewer partials in the same scratch
    _check(300, 520, 4160, resid=False, seed=2)


def test_noalloc_tail_split():
    """A product with 288 tiles (one whole round of rows, then 32 tiles split
    four ways: 6.6 M partials) takes the same plan as sat_op_gemm with a
    workspace, and gives the same bits."""
    from paper_2309_01226_amd import ops
    M, N, K = 9000, 2048, 2048
    flush(f"no-alloc gemm tail split M={M} N={N} K={K}")
    rng = np.random.default_rng(5)
    Ad, Bd, kw, fresh, ref = _case(rng, M, N, K, resid=True)
    out_na = fresh()
    ops.gemm_noalloc(Ad, Bd, M, N, K, out_na, resid=out_na, ldr=N, **kw)
    ws = torch.full((8 * 1024 * 1024,), float("nan"), device="cuda", dtype=torch.float32)
    out_ws = fresh()
    ops.gemm(Ad, Bd, M, N, K, out_ws, splitk_ws=ws, resid=out_ws, ldr=N, **kw)
    torch.cuda.synchronize()
    assert torch.equal(out_na, out_ws), "differs from sat_op_gemm with a workspace"
    assert rel(host(out_na), ref) < 2e-6
    assert int(torch.isfinite(ws).sum().item()) > 0
    # 16448 x 1280 x 1280 (325 tiles): its tail plan needs 8.7 M partials,
    # beyond the scratch, so it runs unsplit, as sat_op_gemm without a workspace
    M, N, K = 16448, 1280, 1280
    flush(f"no-alloc gemm tail split beyond the scratch M={M} N={N} K={K}")
    rng = np.random.default_rng(6)
    Ad, Bd, kw, fresh, ref = _case(rng, M, N, K, resid=False)
    out_na = fresh()
    ops.gemm_noalloc(Ad, Bd, M, N, K, out_na, **kw)
    out_plain = fresh()
    ops.gemm(Ad, Bd, M, N, K, out_plain, **kw)
    torch.cuda.synchronize()
    assert torch.equal(out_na, out_plain)
    assert rel(host(out_na), ref) < 2e-6


def test_noalloc_unsplit_product():
    """A product that never splits K (K < 1024) uses no scratch and equals
    sat_op_gemm."""
    from paper_2309_01226_amd import ops
    rng = np.random.default_rng(3)
    M, N, K = 520, 264, 512
    Ad, Bd, kw, fresh, ref = _case(rng, M, N, K, resid=False)
    a, b = fresh(), fresh()
    ops.gemm_noalloc(Ad, Bd, M, N, K, a, **kw)
    ops.gemm(Ad, Bd, M, N, K, b, **kw)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert rel(host(a), ref) < 2e-6


def test_noalloc_refuses_oversized_partials():
    """16 slices of a 1024 x 1024 product need 16.8 M partials: refused on the
    host with SAT_EINVAL, output untouched."""
    from paper_2309_01226_amd import _lib, ops
    M = N = 1024
    K = 16384
    A = torch.zeros(M, K, device="cuda", dtype=torch.bfloat16)
    B = torch.zeros(N, K, device="cuda", dtype=torch.bfloat16)
    out = torch.full((M, N), 7.0, device="cuda")
    with pytest.raises(_lib.SatError) as e:
        ops.gemm_noalloc(A, B, M, N, K, out, lda=K, ldb=K)
    assert e.value.status == _lib.SAT_EINVAL and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
