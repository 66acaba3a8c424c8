"""Why the free-running bf16 parity bar is looser than the per-layer one.

The oracle accumulates every product in fp64.  Any implementation that
accumulates in fp32 (every GPU GEMM here) lands on the other side of a bf16
rounding tie now and then; each flip is one bf16 ulp of one element, but the
residual stream carries it into every later layer, so at the depth of the
So400m-shaped model (27 layers, D = 1152) the max-abs relative error of the
deep hidden states grows past 2e-2 with no mistake anywhere.

This test shows it on the CPU with no GPU code at all: the same layers as the
oracle (same rounding points, fp64 LayerNorm, softmax and GELU), with only the
GEMM accumulation switched to fp32, drift from the oracle past the per-layer
bar (2e-2) and stay inside the free-running bound the GPU tests use (4e-2).  The per-layer
(teacher-forced) GPU checks keep the strict 2e-2 bar, since one layer alone
does not compound.
"""
import numpy as np
import pytest

from oracle import vit
from paper_2607_12287_amd import synth
from tests.gpu_util import FREE_TOL, TOL


def _encode_fp32_gemms(model, t0):
    """Full forward of one frame, as the oracle's full encode, except that every
    matrix product accumulates in fp32."""
    m = model.shape
    D, H = m.dim, m.heads
    S = vit.round_bf16

    def mm(a, b):
        return (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64)

    Z = S(t0)
    xs = [Z]
    for l in range(m.depth):
        p = lambda n: model.w[f"l{l}.{n}"]  # noqa: E731
        A = S(vit.layer_norm(Z, p("ln1_g"), p("ln1_b"), m.ln_eps))
        qkv = S(mm(A, p("w_qkv")) + p("b_qkv"))
        O = S(vit.attention(qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], H))
        Hr = S(Z + S(mm(O, p("w_o")) + p("b_o")))
        A2 = S(vit.layer_norm(Hr, p("ln2_g"), p("ln2_b"), m.ln_eps))
        G = S(vit.gelu_tanh(S(mm(A2, p("w_1")) + p("b_1"))))
        Z = S(Hr + S(mm(G, p("w_2")) + p("b_2")))
        xs.append(Z)
    return xs


@pytest.mark.slow
def test_fp32_accumulation_alone_drifts_past_the_per_layer_bar():
    wl = synth.workload("so400m")
    m = wl.model
    model = vit.Model(m, wl.weights())
    frame = next(iter(wl.patch_frames(1)))[0]
    cache = vit.full_encode(model, frame)
    xs = _encode_fp32_gemms(model, cache.ref.astype(np.float64))
    errs = [float(np.abs(xs[l] - cache.X[l]).max() / np.abs(cache.X[l]).max()) for l in range(m.depth + 1)]
    assert errs[0] == 0.0                       # same embedding, same rounding
    assert errs[1] <= TOL["bf16"]               # one layer: inside the strict bar
    print("fp32-accumulation drift per layer:", " ".join(f"{e:.2e}" for e in errs))
    assert max(errs) > TOL["bf16"]              # depth: the drift passes the per-layer bar
    assert max(errs) <= FREE_TOL["bf16"]        # and inside the free-running bound
