"""Python handle of one model of the C ABI (include/saturn.h).

torch supplies the device arena (a uint8 tensor) and the HIP stream; every
step runs in libsaturn.so's kernels.  Host accessors return numpy arrays.
"""

import ctypes as C

import numpy as np
import torch

from . import _lib


def make_config(arch, n_layers, d_model=0, n_heads=0, d_mlp=0, vocab=2, seq_len=0, batch=1,
                frozen_layers=0, rotary_dim=0, img_size=0, patch=0, channels=3, lr=1e-3,
                beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, init_std=0.02, ln_eps=1e-5,
                seed=0, checkpoint=0, res_blocks=(0, 0, 0, 0), res_width=0):
    c = _lib.sat_config()
    c.struct_size = C.sizeof(_lib.sat_config)
    c.arch = _lib.ARCH[arch]
    c.n_layers, c.d_model, c.n_heads, c.d_mlp = n_layers, d_model, n_heads, d_mlp
    c.vocab, c.seq_len = vocab, seq_len
    c.img_size, c.patch, c.channels = img_size, patch, channels
    c.rotary_dim, c.batch, c.frozen_layers = rotary_dim, batch, frozen_layers
    c.checkpoint = int(checkpoint)
    c.lr, c.beta1, c.beta2, c.eps, c.weight_decay = lr, beta1, beta2, eps, weight_decay
    c.init_std, c.ln_eps, c.seed = init_std, ln_eps, seed
    for i, b in enumerate(res_blocks):
        c.res_blocks[i] = int(b)
    c.res_width = res_width
    return c


def arena_bytes(cfg):
    n = C.c_size_t()
    _lib.call("sat_model_arena_bytes", C.byref(cfg), C.byref(n))
    return n.value


class Model:
    """One fine-tuning task: a model, its hyper-parameters and its stream."""

    def __init__(self, cfg_kwargs, stream=None, device="cuda", own_arena=False):
        self.kw = dict(cfg_kwargs)
        self.cfg = make_config(**self.kw)
        self.stream = stream if stream is not None else torch.cuda.current_stream(device)
        self.nbytes = arena_bytes(self.cfg)
        if own_arena:
            self.arena = None
            ptr = None
        else:
            self.arena = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
            base = self.arena.data_ptr()
            ptr = (base + 255) // 256 * 256
        h = C.c_void_p()
        _lib.call("sat_model_create", C.byref(self.cfg), None if ptr is None else C.c_void_p(ptr),
                  self.nbytes, C.c_void_p(self.stream.cuda_stream), C.byref(h))
        self.h = h
        self._names = None

    # ---------------------------------------------------------------- lifecycle
    def close(self):
        if getattr(self, "h", None):
            _lib.lib().sat_model_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- steps
    @staticmethod
    def _check_inputs(inputs, labels):
        if not (inputs.is_cuda and labels.is_cuda):
            raise TypeError("inputs and labels must be device tensors")
        if labels.dtype != torch.int32:
            raise TypeError("labels must be int32")
        if not (inputs.is_contiguous() and labels.is_contiguous()):
            raise ValueError("inputs and labels must be contiguous")

    def train_step(self, inputs, labels, sync=True):
        """Enqueue one step; with sync=True wait and return the loss."""
        self._check_inputs(inputs, labels)
        if sync:
            loss = C.c_float()
            _lib.call("sat_train_step", self.h, C.c_void_p(inputs.data_ptr()),
                      C.c_void_p(labels.data_ptr()), C.byref(loss))
            return loss.value
        _lib.call("sat_train_step", self.h, C.c_void_p(inputs.data_ptr()),
                  C.c_void_p(labels.data_ptr()), None)
        return None

    def eval_loss(self, inputs, labels):
        self._check_inputs(inputs, labels)
        loss = C.c_float()
        _lib.call("sat_eval_loss", self.h, C.c_void_p(inputs.data_ptr()),
                  C.c_void_p(labels.data_ptr()), C.byref(loss))
        return loss.value

    # ---------------------------------------------------------------- table
    def param_table(self):
        """[(name, shape, trainable)] in arena order."""
        if self._names is None:
            out = []
            for i in range(_lib.lib().sat_num_params(self.h)):
                name = C.c_char_p()
                shape = (C.c_int64 * 2)()
                tr = C.c_int32()
                _lib.call("sat_param_info", self.h, i, C.byref(name), shape, C.byref(tr))
                shp = (shape[0],) if shape[1] == 1 else (shape[0], shape[1])
                out.append((name.value.decode(), shp, bool(tr.value)))
            self._names = out
        return self._names

    def _read(self, fn, i, shape):
        buf = np.empty(shape, np.float32)
        _lib.call(fn, self.h, i, buf.ctypes.data_as(C.c_void_p))
        return buf

    def params(self):
        return {n: self._read("sat_param_read", i, s) for i, (n, s, _) in enumerate(self.param_table())}

    def grads(self):
        return {n: self._read("sat_grad_read", i, s) for i, (n, s, _) in enumerate(self.param_table())}

    def set_param(self, name, value):
        for i, (n, s, _) in enumerate(self.param_table()):
            if n == name:
                v = np.ascontiguousarray(np.asarray(value, np.float32).reshape(s))
                _lib.call("sat_param_write", self.h, i, v.ctypes.data_as(C.c_void_p))
                return
        raise KeyError(name)

    def state(self):
        out, t = {}, C.c_int64()
        for i, (n, s, _) in enumerate(self.param_table()):
            m = np.empty(s, np.float32)
            v = np.empty(s, np.float32)
            _lib.call("sat_state_read", self.h, i, m.ctypes.data_as(C.c_void_p),
                      v.ctypes.data_as(C.c_void_p), C.byref(t))
            out[n] = (m, v)
        return out, t.value

    def set_state(self, name, m, v, t):
        for i, (n, s, _) in enumerate(self.param_table()):
            if n == name:
                m = np.ascontiguousarray(np.asarray(m, np.float32).reshape(s))
                v = np.ascontiguousarray(np.asarray(v, np.float32).reshape(s))
                _lib.call("sat_state_write", self.h, i, m.ctypes.data_as(C.c_void_p),
                          v.ctypes.data_as(C.c_void_p), t)
                return
        raise KeyError(name)

    def activation(self, layer):
        shape = (C.c_int64 * 2)()
        _lib.call("sat_activation_shape", self.h, layer, shape)
        return self._read("sat_activation_read", layer, (shape[0], shape[1]))

    def logits(self):
        R = self.kw["batch"] if self.kw["arch"] in ("vit", "resnet") else self.rows()
        buf = np.empty((R, self.kw["vocab"]), np.float32)
        _lib.call("sat_logits_read", self.h, buf.ctypes.data_as(C.c_void_p))
        return buf

    def rows(self):
        """Rows entering the loss per step (tokens; images for the ResNet)."""
        if self.kw["arch"] == "resnet":
            return self.kw["batch"]
        if self.kw["arch"] == "vit":
            g = self.kw["img_size"] // self.kw["patch"]
            return self.kw["batch"] * (g * g + 1)
        return self.kw["batch"] * self.kw["seq_len"]

    def stats(self):
        n, nt, fl = C.c_int64(), C.c_int64(), C.c_double()
        _lib.call("sat_model_stats", self.h, C.byref(n), C.byref(nt), C.byref(fl))
        return n.value, nt.value, fl.value

    # ---------------------------------------------------------------- timing
    def set_option(self, name, value):
        """sat_model_set_option: "fused_adamw", "keep_grads" or "overlap_wgrad", value 0 / 1."""
        _lib.call("sat_model_set_option", self.h, _lib.OPTIONS[name], int(value))

    def set_timing(self, kind, max_launches=4096):
        _lib.call("sat_model_set_timing", self.h, kind, max_launches)

    def timing_read(self):
        ms, n, w = C.c_double(), C.c_int64(), C.c_double()
        _lib.call("sat_model_timing_read", self.h, C.byref(ms), C.byref(n), C.byref(w))
        return ms.value, n.value, w.value


TIMING = {"off": 0, "qkv_fwd_gemm": 1, "all_gemm": 2, "adamw": 3, "attn_fwd": 4, "attn_bwd": 5,
          "ln_fwd": 6, "ln_bwd": 7, "xent": 8, "qkv_wgrad_gemm": 9}


def device_batch(cfg_kwargs, seed=0, step=0, rows=None, device="cuda"):
    """Seeded synthetic batch for this model as device tensors (inputs, labels)."""
    from .inputs import batch_for
    x, y = batch_for(cfg_kwargs, seed=seed, step=step, rows=rows)
    return torch.as_tensor(x).to(device), torch.as_tensor(y).to(device)
