"""The AdamW step applied in the epilogue of the weight-gradient products.

A weight whose weight-gradient product runs in the 256 x 256 GEMM kernel (at
least 256 output tiles) is updated inside that product, so its fp32 gradient
makes no round trip through the gradient arena.  The main case is a one-block
GPT-J-shaped decoder at d_model 2048, MLP 8192 and vocabulary 8200: the fused
q|k|v + fc1 weight (448 tiles), fc2 (256) and the head (264 tiles, the last
tile-row holding 8 of its 256 rows) take the fused path; the out-projection
(64 tiles), the vectors and the embedding take the separate pass.

  * fused and separate updates (SAT_OPT_FUSED_ADAMW 1 / 0) give bitwise equal
    losses, parameters and moments over three steps: the same fp32 AdamW
    arithmetic on the same fp32 gradient, and the transposed bf16 copies the
    next step's input-gradient products read;
  * with SAT_OPT_KEEP_GRADS the fused path stores gradients bitwise equal to
    the separate path's; without it, reading a fused weight's gradient fails
    with SAT_ENOTSUP while every other tensor's gradient is readable;
  * one fused step against the float64 oracle on a smaller decoder (MLP 2048,
    vocabulary 512: only the q|k|v + fc1 weight, 256 tiles, is fused), with the
    tolerances of the end-to-end parity test (loss 2e-2; parameters 1e-2
    relative, zero-started ones within 2 lr of the oracle).
"""

import numpy as np
import pytest

import oracle
from tests.gpu_util import flush, rel

pytestmark = pytest.mark.gpu

KW = dict(arch="gptj", n_layers=1, d_model=2048, n_heads=8, d_mlp=8192, vocab=8200, seq_len=256,
          batch=2, rotary_dim=64, lr=1e-3)
KW_ORACLE = dict(KW, d_mlp=2048, vocab=512, seq_len=128)
FUSED = ("h0.attn.qkv.w", "h0.mlp.fc1.w", "h0.mlp.fc2.w", "head.w")


def _models(*opts, kw=KW):
    from paper_2309_01226_amd.model import Model
    out = []
    for o in opts:
        m = Model(kw)
        for k, v in o.items():
            m.set_option(k, v)
        out.append(m)
    return out


# The weight-gradient products run with K = batch x seq_len tokens: 512, 4096
# (the GPT-J step's K) and 8192.
@pytest.mark.parametrize("seq_len", [256, 2048, 4096])
def test_fused_equals_separate(seq_len):
    from paper_2309_01226_amd.model import device_batch
    kw = dict(KW, seq_len=seq_len)
    a, b = _models({}, {"fused_adamw": 0}, kw=kw)
    Pa0, Pb0 = a.params(), b.params()
    for n in Pa0:
        assert np.array_equal(Pa0[n], Pb0[n]), n
    for step in range(3):
        x, y = device_batch(kw, seed=0, step=step)
        la, lb = a.train_step(x, y), b.train_step(x, y)
        flush(f"step {step}: fused {la!r} separate {lb!r}")
        assert la == lb, (step, la, lb)
    Pa, Pb = a.params(), b.params()
    Sa, ta = a.state()
    Sb, tb = b.state()
    assert ta == tb == 3
    for n in Pa:
        assert np.array_equal(Pa[n], Pb[n]), ("param", n, float(np.abs(Pa[n] - Pb[n]).max()))
        assert np.array_equal(Sa[n][0], Sb[n][0]) and np.array_equal(Sa[n][1], Sb[n][1]), ("state", n)
    for n in FUSED:  # the fused weights did move
        assert not np.array_equal(Pa[n], Pa0[n]), n
    x, y = device_batch(kw, seed=0, step=3)
    assert a.eval_loss(x, y) == b.eval_loss(x, y)
    a.close()
    b.close()


def test_keep_grads_and_missing_grads():
    from paper_2309_01226_amd import _lib
    from paper_2309_01226_amd.model import device_batch
    a, b, c = _models({"keep_grads": 1}, {"fused_adamw": 0}, {})
    x, y = device_batch(KW, seed=1, step=0)
    for m in (a, b, c):
        m.train_step(x, y)
    Ga, Gb = a.grads(), b.grads()
    for n in Ga:
        assert np.array_equal(Ga[n], Gb[n]), ("grad", n)
    table = c.param_table()
    for i, (n, shape, _) in enumerate(table):
        if n in FUSED:
            with pytest.raises(_lib.SatError) as e:
                c._read("sat_grad_read", i, shape)
            assert e.value.status == _lib.SAT_ENOTSUP, n
        else:
            assert np.array_equal(c._read("sat_grad_read", i, shape), Gb[n]), n
    # SAT_OPT_KEEP_GRADS on a model that had it off makes the next step's gradients readable
    c.set_option("keep_grads", 1)
    x, y = device_batch(KW, seed=1, step=1)
    c.train_step(x, y)
    b.train_step(x, y)
    Gc, Gb = c.grads(), b.grads()
    for n in FUSED:
        assert np.array_equal(Gc[n], Gb[n]), n
    for m in (a, b, c):
        m.close()


def test_fused_step_vs_oracle():
    from paper_2309_01226_amd import _lib
    from paper_2309_01226_amd.inputs import batch_for
    from paper_2309_01226_amd.model import Model, device_batch
    KW = KW_ORACLE
    m = Model(KW)
    keys = ("arch", "n_layers", "d_model", "n_heads", "d_mlp", "vocab", "seq_len", "batch",
            "rotary_dim", "lr")
    ocfg = oracle.Config(**{k: KW[k] for k in keys})
    P = {n: v.astype(np.float64) for n, v in m.params().items()}
    x, y = device_batch(KW, seed=2, step=0)
    xh, yh = batch_for(KW, seed=2, step=0)
    gl = m.train_step(x, y)
    newP = m.params()
    i = [n for n, _, _ in m.param_table()].index("h0.attn.qkv.w")
    with pytest.raises(_lib.SatError):  # the fused path was taken
        m._read("sat_grad_read", i, m.param_table()[i][1])
    loss, _, P1, _, _ = oracle.train_step(ocfg, P, {}, xh, yh)
    flush(f"fused step: gpu loss {gl:.6f} oracle {loss:.6f}")
    assert abs(gl - loss) / abs(loss) < 2e-2
    num = den = 0.0
    lr = KW["lr"]
    for n, p in newP.items():
        num += float(np.sum((p - P1[n]) ** 2))
        den += float(np.sum(P1[n] ** 2))
        if n.endswith(".b"):
            assert float(np.abs(p - P1[n]).max()) <= 2 * lr, n
        else:
            assert rel(p, P1[n]) < 1e-2, (n, rel(p, P1[n]))
    assert (num / den) ** 0.5 < 1e-2
    m.close()
