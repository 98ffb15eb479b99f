"""ctypes binding of libsaturn.so (argument marshalling only).

Every computation happens in the library's HIP kernels; this module only
declares the C signatures of include/saturn.h and include/saturn_ops.h and
turns non-zero status codes into exceptions.  Loading fails loudly when the
library has not been built: there is no fallback.
"""

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# SAT_LIBRARY selects another build of the same library (for instance the
# AddressSanitizer build of the host code); by default the in-tree one.
LIB_PATH = os.environ.get("SAT_LIBRARY") or os.path.join(_PKG, "libsaturn.so")

SAT_OK, SAT_EINVAL, SAT_ENOMEM, SAT_EHIP, SAT_ESTATE, SAT_ENONFINITE, SAT_ENOTSUP = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {0: "SAT_OK", -1: "SAT_EINVAL", -2: "SAT_ENOMEM", -3: "SAT_EHIP", -4: "SAT_ESTATE",
                -5: "SAT_ENONFINITE", -6: "SAT_ENOTSUP"}
ARCH = {"gpt2": 0, "gptj": 1, "vit": 2, "resnet": 3}
OPTIONS = {"fused_adamw": 1, "keep_grads": 2, "overlap_wgrad": 3}
GEMM_NOALLOC_WS_ELEMS = 8 * 1024 * 1024   # SAT_GEMM_NOALLOC_WS_ELEMS in saturn_ops.h


class SatError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class sat_config(C.Structure):
    _fields_ = [
        ("struct_size", C.c_uint32), ("arch", C.c_int32),
        ("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32), ("d_mlp", C.c_int32),
        ("vocab", C.c_int32), ("seq_len", C.c_int32),
        ("img_size", C.c_int32), ("patch", C.c_int32), ("channels", C.c_int32),
        ("rotary_dim", C.c_int32), ("batch", C.c_int32), ("frozen_layers", C.c_int32),
        ("checkpoint", C.c_int32),
        ("lr", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
        ("weight_decay", C.c_double), ("init_std", C.c_float), ("ln_eps", C.c_float),
        ("seed", C.c_uint64), ("res_blocks", C.c_int32 * 4), ("res_width", C.c_int32),
    ]


class sat_gemm_desc(C.Structure):
    _fields_ = [
        ("A", C.c_void_p), ("B", C.c_void_p),
        ("M", C.c_int32), ("N", C.c_int32), ("K", C.c_int32),
        ("lda", C.c_int64), ("ldb", C.c_int64),
        ("a_layout", C.c_int32), ("b_layout", C.c_int32), ("epilogue", C.c_int32),
        ("out", C.c_void_p), ("ldo", C.c_int64),
        ("bias", C.c_void_p), ("bias_col0", C.c_int32),
        ("resid", C.c_void_p), ("ldr", C.c_int64),
        ("out2", C.c_void_p), ("ldo2", C.c_int64), ("gelu_col0", C.c_int32),
        ("aux", C.c_void_p), ("ldaux", C.c_int64),
        ("gelu_erf", C.c_int32),
        ("splitk_ws", C.c_void_p), ("splitk_ws_elems", C.c_int64),
    ]


class sat_profile_result(C.Structure):
    _fields_ = [
        ("struct_size", C.c_uint32), ("steps", C.c_int32),
        ("step_ms_mean", C.c_double), ("step_ms_min", C.c_double), ("step_ms_max", C.c_double),
        ("tokens_per_s", C.c_double), ("step_tflop", C.c_double), ("achieved_tflops", C.c_double),
        ("steps_per_epoch", C.c_int64), ("epoch_ms", C.c_double), ("arena_bytes", C.c_uint64),
        ("final_loss", C.c_float),
    ]


_VP, _I32, _I64, _F32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float

# name -> (restype, argtypes); restype int means a sat_status to check
SIGNATURES = {
    "sat_last_error": (C.c_char_p, []),
    "sat_model_arena_bytes": (C.c_int, [C.POINTER(sat_config), C.POINTER(C.c_size_t)]),
    "sat_model_create": (C.c_int, [C.POINTER(sat_config), _VP, C.c_size_t, _VP, C.POINTER(_VP)]),
    "sat_train_step": (C.c_int, [_VP, _VP, _VP, C.POINTER(C.c_float)]),
    "sat_eval_loss": (C.c_int, [_VP, _VP, _VP, C.POINTER(C.c_float)]),
    "sat_model_destroy": (C.c_int, [_VP]),
    "sat_num_params": (C.c_int32, [_VP]),
    "sat_param_info": (C.c_int, [_VP, _I32, C.POINTER(C.c_char_p), C.POINTER(C.c_int64), C.POINTER(_I32)]),
    "sat_param_read": (C.c_int, [_VP, _I32, _VP]),
    "sat_param_write": (C.c_int, [_VP, _I32, _VP]),
    "sat_grad_read": (C.c_int, [_VP, _I32, _VP]),
    "sat_activation_read": (C.c_int, [_VP, _I32, _VP]),
    "sat_activation_shape": (C.c_int, [_VP, _I32, C.POINTER(C.c_int64)]),
    "sat_logits_read": (C.c_int, [_VP, _VP]),
    "sat_state_read": (C.c_int, [_VP, _I32, _VP, _VP, C.POINTER(C.c_int64)]),
    "sat_state_write": (C.c_int, [_VP, _I32, _VP, _VP, C.c_int64]),
    "sat_model_stats": (C.c_int, [_VP, C.POINTER(C.c_int64), C.POINTER(C.c_int64), C.POINTER(C.c_double)]),
    "sat_model_set_timing": (C.c_int, [_VP, _I32, _I32]),
    "sat_model_set_option": (C.c_int, [_VP, _I32, _I32]),
    "sat_profile": (C.c_int, [C.POINTER(sat_config), _VP, _I32, _I32, _I64, C.POINTER(sat_profile_result)]),
    "sat_profile_batch": (C.c_int, [C.POINTER(sat_config), _VP, _VP, _VP]),
    "sat_model_timing_read": (C.c_int, [_VP, C.POINTER(C.c_double), C.POINTER(C.c_int64), C.POINTER(C.c_double)]),
    "sat_op_gemm": (C.c_int, [C.POINTER(sat_gemm_desc), _VP]),
    "sat_op_gemm_noalloc": (C.c_int, [C.POINTER(sat_gemm_desc), _VP]),
    "sat_op_layernorm_fwd": (C.c_int, [_VP, _I64, _I64, _VP, _VP, _VP, _I64, _VP, _VP, _I32, _I32, _F32, _VP]),
    "sat_op_layernorm_bwd": (C.c_int, [_VP, _I64, _VP, _I64, _I64, _VP, _VP, _VP, _VP, _I64, _VP, _VP, _VP,
                                       _I32, _I32, _VP]),
    "sat_op_attention_fwd": (C.c_int, [_VP, _VP, _VP, _I64, _I64, _I64, _VP, _I64, _VP,
                                       _I32, _I32, _I32, _I32, _I32, _F32, _VP]),
    "sat_op_attention_bwd": (C.c_int, [_VP, _VP, _VP, _I64, _I64, _I64, _VP, _I64, _VP, _VP, _I64, _VP,
                                       _VP, _VP, _VP, _I64, _I64, _I64, _I32, _I32, _I32, _I32, _I32,
                                       _F32, _VP]),
    "sat_op_rotary": (C.c_int, [_VP, _I64, _I32, _I32, _I32, _I32, _I32, _I32, _VP]),
    "sat_op_cross_entropy": (C.c_int, [_VP, _I64, _VP, _I32, _I32, _VP, _VP, _I64, _VP, _VP]),
    "sat_op_adamw": (C.c_int, [_VP, _VP, _VP, _VP, _VP, _I64, C.c_double, C.c_double, C.c_double,
                               C.c_double, C.c_double, _I64, _VP]),
    "sat_op_embed_fwd": (C.c_int, [_VP, _VP, _VP, _VP, _I32, _I32, _I32, _I32, _VP]),
    "sat_op_embed_bwd": (C.c_int, [_VP, _VP, _VP, _I32, _I32, _I32, _VP, _VP]),
    "sat_op_colsum": (C.c_int, [_VP, _I64, _I32, _I32, _VP, _VP, _VP]),
    "sat_op_transpose_bf16": (C.c_int, [_VP, _I64, _VP, _I64, _I32, _I32, _VP]),
    "sat_op_im2col": (C.c_int, [_VP, _VP, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _VP]),
    "sat_op_im2col_t": (C.c_int, [_VP, _VP, _I64, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _VP]),
    "sat_op_col2im": (C.c_int, [_VP, _VP, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _VP]),
    "sat_op_batchnorm_fwd": (C.c_int, [_VP, _I64, _I32, _VP, _VP, _F32, _I32, _VP, _VP, _VP, _VP, _VP,
                                       _VP]),
    "sat_op_batchnorm_bwd": (C.c_int, [_VP, _I32, _VP, _VP, _VP, _VP, _VP, _I64, _I32, _VP, _VP, _VP,
                                       _VP, _VP]),
    "sat_op_maxpool_fwd": (C.c_int, [_VP, _I32, _I32, _I32, _I32, _VP, _VP, _VP, _VP]),
    "sat_op_maxpool_bwd": (C.c_int, [_VP, _VP, _I32, _I32, _I32, _I32, _VP, _VP]),
}

_lib = None


def lib():
    """The loaded library (raises if it is missing: there is no CPU fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2309_01226_amd.build")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            if hasattr(L, name):
                f = getattr(L, name)
                f.restype = res
                f.argtypes = args
        _lib = L
    return _lib


def last_error():
    return lib().sat_last_error().decode(errors="replace")


def check(status):
    if status != SAT_OK:
        raise SatError(status, last_error())
    return status


def call(name, *args):
    """Call a sat_* function that returns a status; raise on failure."""
    return check(getattr(lib(), name)(*args))
