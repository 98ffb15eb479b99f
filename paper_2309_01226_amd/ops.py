"""Kernel-level entry points on torch device tensors (marshalling only).

Each function checks shapes on the host, then calls one sat_op_* entry point
of libsaturn.so on the current torch stream.  torch provides device memory and
the stream; every element of every output is computed by the HIP kernels.
"""

import ctypes as C

import torch

from . import _lib

LAY_K, LAY_MN = 0, 1
EPI_F32, EPI_RESID_F32, EPI_BF16, EPI_DGELU_BF16 = 0, 1, 2, 3


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t, dtype, name):
    if t is None:
        return
    if not t.is_cuda or t.dtype != dtype:
        raise TypeError(f"{name}: expected a CUDA tensor of {dtype}, got {t.device} {t.dtype}")


def _gemm_desc(A, B, M, N, K, out, lda, ldb, a_layout, b_layout, epilogue, ldo, bias, bias_col0,
               resid, ldr, out2, ldo2, gelu_col0, aux, ldaux, gelu_erf, splitk_ws):
    _need(A, torch.bfloat16, "A")
    _need(B, torch.bfloat16, "B")
    _need(bias, torch.float32, "bias")
    _need(resid, torch.float32, "resid")
    _need(aux, torch.bfloat16, "aux")
    _need(splitk_ws, torch.float32, "splitk_ws")
    need_a = (M - 1) * lda + K if a_layout == LAY_K else (K - 1) * lda + M
    need_b = (N - 1) * ldb + K if b_layout == LAY_K else (K - 1) * ldb + N
    if A.numel() < need_a or B.numel() < need_b:
        raise ValueError("gemm: operand smaller than its sizes imply")
    ldo = N if ldo is None else ldo
    if out.numel() < (M - 1) * ldo + N:
        raise ValueError("gemm: out too small")
    return _lib.sat_gemm_desc(
        A=A.data_ptr(), B=B.data_ptr(), M=M, N=N, K=K, lda=lda, ldb=ldb,
        a_layout=a_layout, b_layout=b_layout, epilogue=epilogue,
        out=out.data_ptr(), ldo=ldo,
        bias=None if bias is None else bias.data_ptr(), bias_col0=bias_col0,
        resid=None if resid is None else resid.data_ptr(), ldr=ldo if ldr is None else ldr,
        out2=None if out2 is None else out2.data_ptr(), ldo2=ldo2, gelu_col0=gelu_col0,
        aux=None if aux is None else aux.data_ptr(), ldaux=ldaux, gelu_erf=gelu_erf,
        splitk_ws=None if splitk_ws is None else splitk_ws.data_ptr(),
        splitk_ws_elems=0 if splitk_ws is None else splitk_ws.numel())


def gemm(A, B, M, N, K, out, *, lda, ldb, a_layout=LAY_K, b_layout=LAY_K, epilogue=EPI_F32,
         ldo=None, bias=None, bias_col0=0, resid=None, ldr=None, out2=None, ldo2=0, gelu_col0=0,
         aux=None, ldaux=0, gelu_erf=0, splitk_ws=None):
    """C[m, n] = sum_k A(m, k) B(n, k) with the chosen epilogue (see saturn_ops.h);
    splitk_ws: optional fp32 scratch that lets a small fp32-output product run split-K."""
    d = _gemm_desc(A, B, M, N, K, out, lda, ldb, a_layout, b_layout, epilogue, ldo, bias, bias_col0,
                   resid, ldr, out2, ldo2, gelu_col0, aux, ldaux, gelu_erf, splitk_ws)
    _lib.call("sat_op_gemm", C.byref(d), _stream())
    return out


def gemm_noalloc(A, B, M, N, K, out, *, lda, ldb, a_layout=LAY_K, b_layout=LAY_K, epilogue=EPI_F32,
                 ldo=None, bias=None, bias_col0=0, resid=None, ldr=None, out2=None, ldo2=0,
                 gelu_col0=0, aux=None, ldaux=0, gelu_erf=0):
    """The same product through sat_op_gemm_noalloc: split-K partials go to the
    library's own per-device scratch, and the call allocates nothing."""
    d = _gemm_desc(A, B, M, N, K, out, lda, ldb, a_layout, b_layout, epilogue, ldo, bias, bias_col0,
                   resid, ldr, out2, ldo2, gelu_col0, aux, ldaux, gelu_erf, None)
    _lib.call("sat_op_gemm_noalloc", C.byref(d), _stream())
    return out


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def layernorm_fwd(x, g, b, y, mean, rstd, rows, d, eps, *, ldx=None, row_stride=1, ldy=None):
    _need(x, torch.float32, "x")
    _need(y, torch.bfloat16, "y")
    _lib.call("sat_op_layernorm_fwd", _p(x), ldx or d, row_stride, _p(g), _p(b), _p(y), ldy or d,
              _p(mean), _p(rstd), rows, d, C.c_float(eps), _stream())


def layernorm_bwd(dy, x, g, mean, rstd, dres, dg, db, rows, d, *, lddy=None, ldx=None, row_stride=1,
                  ldres=None):
    n_part = min(rows, 1024)
    work = torch.empty(2 * n_part * d, device=dy.device, dtype=torch.float32)
    _lib.call("sat_op_layernorm_bwd", _p(dy), lddy or d, _p(x), ldx or d, row_stride, _p(g),
              _p(mean), _p(rstd), _p(dres), ldres or d, _p(dg), _p(db), _p(work), rows, d, _stream())
    return work


def attention_fwd(q, k, v, o, lse, B, H, S, dh, causal, scale, *, ldq, ldk, ldv, ldo):
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        _need(t, torch.bfloat16, n)
    _need(lse, torch.float32, "lse")
    if lse.numel() < B * H * S:
        raise ValueError("lse too small")
    _lib.call("sat_op_attention_fwd", _p(q), _p(k), _p(v), ldq, ldk, ldv, _p(o), ldo, _p(lse),
              B, H, S, dh, int(causal), C.c_float(scale), _stream())


def attention_bwd(q, k, v, o, lse, dout, dq, dk, dv, B, H, S, dh, causal, scale, *, ldq, ldk, ldv,
                  ldo, lddo, lddq, lddk, lddv):
    delta = torch.empty(B * H * S, device=q.device, dtype=torch.float32)
    _lib.call("sat_op_attention_bwd", _p(q), _p(k), _p(v), ldq, ldk, ldv, _p(o), ldo, _p(lse),
              _p(dout), lddo, _p(delta), _p(dq), _p(dk), _p(dv), lddq, lddk, lddv, B, H, S, dh,
              int(causal), C.c_float(scale), _stream())
    return delta


def rotary(qk, ld, B, S, H, dh, rd, inverse=False):
    _need(qk, torch.bfloat16, "qk")
    _lib.call("sat_op_rotary", _p(qk), ld, B, S, H, dh, rd, int(inverse), _stream())


def cross_entropy(z, labels, row_loss, dz, inv_n, N, V, *, ldz=None, lddz=None):
    _need(z, torch.float32, "z")
    _need(dz, torch.bfloat16, "dz")
    _need(labels, torch.int32, "labels")
    _lib.call("sat_op_cross_entropy", _p(z), ldz or V, _p(labels), N, V, _p(row_loss), _p(dz),
              lddz or V, _p(inv_n), _stream())


def adamw(p, g, m, v, shadow, n, lr, beta1, beta2, eps, wd, t):
    for name, t_ in (("p", p), ("g", g), ("m", m), ("v", v)):
        _need(t_, torch.float32, name)
    _need(shadow, torch.bfloat16, "shadow")
    _lib.call("sat_op_adamw", _p(p), _p(g), _p(m), _p(v), _p(shadow), n, float(lr), float(beta1),
              float(beta2), float(eps), float(wd), t, _stream())


def embed_fwd(tok, wte, wpe, h, T, S, d, V):
    _need(tok, torch.int32, "tok")
    _lib.call("sat_op_embed_fwd", _p(tok), _p(wte), _p(wpe), _p(h), T, S, d, V, _stream())


def embed_bwd(tok, dh, dwte, T, d, V):
    work = torch.empty(max(min(T, 16384), 1), device=dh.device, dtype=torch.int32)
    _lib.call("sat_op_embed_bwd", _p(tok), _p(dh), _p(dwte), T, d, V, _p(work), _stream())


def colsum(X, out, rows, cols, ldx=None):
    work = torch.empty(min(rows, 256) * max(cols, 1), device=X.device, dtype=torch.float32)
    _lib.call("sat_op_colsum", _p(X), ldx or cols, rows, cols, _p(out), _p(work), _stream())


def transpose_bf16(src, dst, rows, cols, *, lds=None, ldd=None):
    """dst[c, r] = src[r, c] (bf16, rows and cols multiples of 8)."""
    _need(src, torch.bfloat16, "src")
    _need(dst, torch.bfloat16, "dst")
    _lib.call("sat_op_transpose_bf16", _p(src), lds or cols, _p(dst), ldd or rows, rows, cols,
              _stream())


# ---------------------------------------------------------------- ResNet kernels

def _hw(H, k, stride, pad):
    return (H + 2 * pad - k) // stride + 1


def im2col(x, N, H, W, C, k, stride, pad):
    """x bf16 [N*H*W, C] -> col bf16 [N*Ho*Wo, k*k*C]."""
    _need(x, torch.bfloat16, "x")
    Ho, Wo = _hw(H, k, stride, pad), _hw(W, k, stride, pad)
    if x.numel() < N * H * W * C:
        raise ValueError("im2col: x too small")
    col = torch.empty(N * Ho * Wo, k * k * C, device=x.device, dtype=torch.bfloat16)
    _lib.call("sat_op_im2col", _p(x), _p(col), N, H, W, C, k, stride, pad, _stream())
    return col


def im2col_t(x, N, H, W, C, k, stride, pad):
    """x bf16 [N*H*W, C] -> colT bf16 [k*k*C, N*Ho*Wo] (im2col transposed)."""
    _need(x, torch.bfloat16, "x")
    Ho, Wo = _hw(H, k, stride, pad), _hw(W, k, stride, pad)
    if x.numel() < N * H * W * C:
        raise ValueError("im2col_t: x too small")
    P = N * Ho * Wo
    colT = torch.empty(k * k * C, P, device=x.device, dtype=torch.bfloat16)
    _lib.call("sat_op_im2col_t", _p(x), _p(colT), P, N, H, W, C, k, stride, pad, _stream())
    return colT


def col2im(dcol, N, H, W, C, k, stride, pad, dx=None):
    """dcol fp32 [N*Ho*Wo, k*k*C] -> dx fp32 [N*H*W, C] (accumulated into dx when given)."""
    _need(dcol, torch.float32, "dcol")
    Ho, Wo = _hw(H, k, stride, pad), _hw(W, k, stride, pad)
    if dcol.numel() < N * Ho * Wo * k * k * C:
        raise ValueError("col2im: dcol too small")
    acc = dx is not None
    if dx is None:
        dx = torch.empty(N * H * W, C, device=dcol.device, dtype=torch.float32)
    _lib.call("sat_op_col2im", _p(dcol), _p(dx), N, H, W, C, k, stride, pad, int(acc), _stream())
    return dx


def batchnorm_fwd(x, g, b, eps, relu=False):
    """Training-mode batch norm of x fp32 [P, C]: (y bf16, yf fp32, mean, rstd)."""
    _need(x, torch.float32, "x")
    P, Cc = x.shape
    part = torch.empty(2 * 1024 * Cc, device=x.device, dtype=torch.float32)
    mean = torch.empty(Cc, device=x.device, dtype=torch.float32)
    rstd = torch.empty_like(mean)
    y = torch.empty(P, Cc, device=x.device, dtype=torch.bfloat16)
    yf = torch.empty(P, Cc, device=x.device, dtype=torch.float32)
    _lib.call("sat_op_batchnorm_fwd", _p(x), P, Cc, _p(g), _p(b), C.c_float(eps), int(relu), _p(part),
              _p(mean), _p(rstd), _p(y), _p(yf), _stream())
    return y, yf, mean, rstd


def batchnorm_bwd(dy, x, mean, rstd, g, mask=None):
    """Backward of batchnorm_fwd (through a ReLU whose output is `mask`, bf16 or
    fp32, when given): (dx bf16, dg, db)."""
    _need(dy, torch.float32, "dy")
    P, Cc = dy.shape
    kind = 0 if mask is None else (1 if mask.dtype == torch.bfloat16 else 2)
    part = torch.empty(2 * 1024 * Cc, device=dy.device, dtype=torch.float32)
    dg = torch.empty(Cc, device=dy.device, dtype=torch.float32)
    db = torch.empty_like(dg)
    dx = torch.empty(P, Cc, device=dy.device, dtype=torch.bfloat16)
    _lib.call("sat_op_batchnorm_bwd", _p(dy), kind, _p(mask), _p(x), _p(mean), _p(rstd), _p(g), P, Cc,
              _p(part), _p(dg), _p(db), _p(dx), _stream())
    return dx, dg, db


def maxpool_fwd(x, N, H, W, C):
    """3 x 3 / 2 max pool (padding 1) of x fp32 [N*H*W, C]: (y fp32, y bf16, arg uint8)."""
    _need(x, torch.float32, "x")
    Ho, Wo = _hw(H, 3, 2, 1), _hw(W, 3, 2, 1)
    y = torch.empty(N * Ho * Wo, C, device=x.device, dtype=torch.float32)
    yb = torch.empty(N * Ho * Wo, C, device=x.device, dtype=torch.bfloat16)
    arg = torch.empty(N * Ho * Wo, C, device=x.device, dtype=torch.uint8)
    _lib.call("sat_op_maxpool_fwd", _p(x), N, H, W, C, _p(y), _p(yb), _p(arg), _stream())
    return y, yb, arg


def maxpool_bwd(dy, arg, N, H, W, C):
    _need(dy, torch.float32, "dy")
    dx = torch.empty(N * H * W, C, device=dy.device, dtype=torch.float32)
    _lib.call("sat_op_maxpool_bwd", _p(dy), _p(arg), N, H, W, C, _p(dx), _stream())
    return dx
