"""Helpers for the GPU parity tests: bf16 rounding on the host (to feed both
sides identical operand values) and relative Frobenius error."""

import numpy as np
import torch


def bf16_round(x):
    """Round a float array to bfloat16 values (returned as float64)."""
    return torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def to_dev_bf16(x):
    return torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16).cuda()


def to_dev_f32(x):
    return torch.as_tensor(np.asarray(x, np.float32)).cuda()


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def flush(*msg):
    print(*msg, flush=True)
