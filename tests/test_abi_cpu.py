"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function the headers declare, validates configurations and sizes arenas
(these calls make no HIP call)."""

import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    from paper_2309_01226_amd import _lib
    return _lib


def _declared():
    names = set()
    for h in ("saturn.h", "saturn_ops.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(sat_[a-z0-9_]+)\s*\(", src))
    return names


def test_every_declared_symbol_is_exported():
    L = _lib().lib()
    declared = _declared()
    assert len(declared) >= 20
    for n in sorted(declared):
        assert hasattr(L, n), n
    # and the binding declares a signature for each
    assert declared <= set(_lib().SIGNATURES), declared - set(_lib().SIGNATURES)


def _cfg(**kw):
    from paper_2309_01226_amd.model import make_config
    base = dict(arch="gpt2", n_layers=2, d_model=64, n_heads=4, d_mlp=256, vocab=512, seq_len=32,
                batch=2)
    base.update(kw)
    return make_config(**base)


def _bytes(cfg):
    n = C.c_size_t()
    st = _lib().lib().sat_model_arena_bytes(C.byref(cfg), C.byref(n))
    return st, n.value


def test_arena_bytes_valid_configs():
    st, n = _bytes(_cfg())
    assert st == 0 and n > 0
    st2, n2 = _bytes(_cfg(n_layers=4))
    assert st2 == 0 and n2 > n
    # frozen layers share one activation set: less memory
    st3, n3 = _bytes(_cfg(n_layers=4, frozen_layers=3))
    assert st3 == 0 and n3 < n2
    for arch_kw in (dict(arch="gptj", rotary_dim=8), dict(arch="vit", img_size=28, patch=14)):
        st, n = _bytes(_cfg(**arch_kw))
        assert st == 0 and n > 0


def test_arena_bytes_gptj_full_fits_hbm():
    from paper_2309_01226_amd.configs import PRESETS
    st, n = _bytes(_cfg(**PRESETS["gptj"]))
    assert st == 0
    assert 100e9 < n < 200e9  # fp32 p, g, m, v + bf16 shadow ~109 GB, plus activations


@pytest.mark.parametrize("bad", [
    dict(d_model=60),                    # not a multiple of 8
    dict(n_heads=3),                     # d % H != 0
    dict(n_heads=1, d_model=64 * 9),     # head dim 576 unsupported
    dict(frozen_layers=3),               # k > L
    dict(frozen_layers=-1),
    dict(n_layers=0),
    dict(vocab=1),
    dict(batch=0),
    dict(seq_len=0),
    dict(arch="gptj", rotary_dim=3),     # odd rotary
    dict(arch="gptj", rotary_dim=32),    # > head dim 16
    dict(rotary_dim=4),                  # rotary on GPT-2
    dict(arch="vit", img_size=30, patch=14),
    dict(beta1=1.0),
    dict(eps=0.0),
    dict(vocab=70000),                   # token ids of the embedding backward: 16 bits
])
def test_invalid_configs_rejected(bad):
    st, _ = _bytes(_cfg(**bad))
    assert st == -1
    assert _lib().last_error()


def test_struct_size_checked():
    cfg = _cfg()
    cfg.struct_size = 4
    st, _ = _bytes(cfg)
    assert st == -1 and "struct_size" in _lib().last_error()


def test_destroy_null_and_null_args():
    L = _lib().lib()
    assert L.sat_model_destroy(None) == 0
    assert L.sat_num_params(None) == 0
    assert L.sat_train_step(None, None, None, None) == -1
    assert L.sat_model_arena_bytes(None, None) == -1


def test_embedding_limits():
    # more than 16384 positions: the embedding backward takes them in chunks
    st, _ = _bytes(_cfg(seq_len=20000, batch=1))
    assert st == 0
    # the 16-bit token ids of its sort keys bound the vocabulary, unless the
    # embedding is frozen
    st, _ = _bytes(_cfg(vocab=70000, frozen_layers=1))
    assert st == 0


def test_op_argument_checks_make_no_launch():
    from paper_2309_01226_amd import _lib as B
    L = B.lib()
    d = B.sat_gemm_desc()
    assert L.sat_op_gemm(C.byref(d), None) == -1          # null operands
    assert L.sat_op_adamw(None, None, None, None, None, 0, 0, 0, 0, 0, 0, 1, None) == -1
    assert L.sat_op_attention_fwd(C.c_void_p(16), C.c_void_p(16), C.c_void_p(16), 8, 8, 8,
                                  C.c_void_p(16), 8, C.c_void_p(16), 1, 1, 4, 48, 1,
                                  C.c_float(1.0), None) == -1  # head dim 48 unsupported
    # head dims 64, 80, 256: q must be 16-byte aligned (here 2 bytes off)
    for dh in (64, 80, 256):
        assert L.sat_op_attention_fwd(C.c_void_p(18), C.c_void_p(16), C.c_void_p(16), 3 * dh, 3 * dh,
                                      3 * dh, C.c_void_p(16), dh, C.c_void_p(16), 1, 1, 4, dh, 1,
                                      C.c_float(1.0), None) == -1, dh
        assert "aligned" in B.last_error()
        p = [C.c_void_p(16)] * 3
        assert L.sat_op_attention_bwd(C.c_void_p(18), *p[:2], 3 * dh, 3 * dh, 3 * dh, p[0], dh, p[0],
                                      p[0], dh, p[0], p[0], p[0], p[0], dh, dh, dh, 1, 1, 4, dh, 1,
                                      C.c_float(1.0), None) == -1, dh
        assert "aligned" in B.last_error()


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without the built library every entry point raises: no CPU fallback."""
    from paper_2309_01226_amd import _lib as L
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "libsaturn.so"))
    monkeypatch.setattr(L, "_lib", None)
    with pytest.raises(ImportError):
        L.lib()
    with pytest.raises(ImportError):
        L.call("sat_model_destroy", None)
