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
bar (2e-2).  How far depends on the summation order and the workload: on the
1024-token 448x448 frame, fp32 accumulation with the MLP down projection's K
summed in three fp32 partial sums (as the split-K GPU form does) drifts past
4e-2.  The free-running bound the GPU tests use (5e-2) is about 1.2x the
largest such drift.  The per-layer (teacher-forced) GPU checks keep the strict
2e-2 bar, since one layer alone does not compound.
"""
import numpy as np
import pytest

from oracle import vit
from paper_2607_12287_amd import synth
from tests.gpu_util import FREE_TOL, TOL


def _mm32(a, b):
    return (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64)


def _mm32_split3(a, b):
    """fp32 product whose K (in 32-deep chunks) is split into three ranges,
    each summed in fp32, the three partial sums then added in order in fp32."""
    K = a.shape[1]
    kper = -(-(-(-K // 32)) // 3) * 32
    acc = None
    for lo in range(0, K, kper):
        p = a[:, lo:lo + kper].astype(np.float32) @ b[lo:lo + kper].astype(np.float32)
        acc = p if acc is None else (acc + p).astype(np.float32)
    return acc.astype(np.float64)


def _encode_fp32_gemms(model, t0, mm_down=_mm32):
    """Full forward of one frame, as the oracle's full encode, except that every
    matrix product accumulates in fp32 (the MLP down projection by mm_down)."""
    m = model.shape
    D, H = m.dim, m.heads
    S = vit.round_bf16
    mm = _mm32

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
        Z = S(Hr + S(mm_down(G, p("w_2")) + p("b_2")))
        xs.append(Z)
    return xs


@pytest.mark.slow
def test_fp32_accumulation_drifts_past_the_per_layer_bar_and_inside_the_free_running_bound():
    """1024 tokens, 27 layers: fp32 accumulation with the down projection's K
    split in three stays inside the per-layer bar for one layer, drifts past
    it (and past 4e-2) with depth, and stays inside the free-running bound."""
    wl = synth.workload("so400m_448")
    m = wl.model
    model = vit.Model(m, wl.weights())
    frame = next(iter(wl.patch_frames(1)))[0]
    cache = vit.full_encode(model, frame)
    xs = _encode_fp32_gemms(model, cache.ref.astype(np.float64), mm_down=_mm32_split3)
    errs = [float(np.abs(xs[l] - cache.X[l]).max() / np.abs(cache.X[l]).max()) for l in range(m.depth + 1)]
    print("fp32 split-K drift per layer:", " ".join(f"{e:.2e}" for e in errs))
    assert errs[0] == 0.0                       # same embedding, same rounding
    assert errs[1] <= TOL["bf16"]               # one layer: inside the per-layer bar
    assert max(errs) > TOL["bf16"]              # depth: past the per-layer bar
    assert max(errs) > 4e-2                     # and past the earlier 4e-2 free-running bar
    assert max(errs) <= FREE_TOL["bf16"]        # inside the free-running bound
