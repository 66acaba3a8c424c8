"""Where the oracle rounds to bf16, pinned against PyTorch's own bf16 modules.

The reading (oracle/vit.py, module text): the paper's encoder runs in half
precision under PyTorch (Appendix A), where every operation computes
internally at higher precision and stores its output in the storage type.
PyTorch's CPU bf16 modules are that pipeline: F.layer_norm, F.linear (the
bias inside the one rounding), the math backend of
F.scaled_dot_product_attention, F.gelu and the residual `+` each round their
result once.  A dense layer built from them on bf16 tensors is therefore an
independent statement of the rounding points.  Both sides compute internally
at different precisions (fp32 in torch, fp64 in the oracle), so a result that
sits within an fp32 rounding of a bf16 tie may come out one bf16 ulp apart;
everything else must agree bit for bit.

The mutation checks plant one mistake at a time in the oracle (one call of
``S`` made the identity, by call order inside a layer) and show that the pin
catches each: a dropped rounding anywhere in the layer moves many outputs.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.nn.attention import SDPBackend, sdpa_kernel

from oracle import vit
from paper_2607_12287_amd import synth

BF = torch.bfloat16


def _model(seed=5, scale=True):
    """A one-layer bf16 model whose activations are O(1), so that every
    rounding point matters: weights ~ N(0, 1/fan_in) instead of N(0, 0.02)."""
    m = synth.small_model(dim=64, depth=1, heads=2, mlp=96, img=32, patch=8, dtype="bf16")
    w = synth.make_weights(m, seed)
    if scale:
        rng = np.random.default_rng(seed + 1)
        for name in ("w_qkv", "w_o", "w_1", "w_2"):
            k = f"l0.{name}"
            fan_in = w[k].shape[0]
            w[k] = vit.round_bf16(rng.standard_normal(w[k].shape) / np.sqrt(fan_in)).astype(np.float32)
        for name in ("b_qkv", "b_o", "b_1", "b_2"):
            k = f"l0.{name}"
            w[k] = vit.round_bf16(0.3 * rng.standard_normal(w[k].shape)).astype(np.float32)
    return m, w


def _x(m, seed=9):
    rng = np.random.default_rng(seed)
    return vit.round_bf16(rng.standard_normal((m.n_tokens, m.dim)))


def torch_bf16_layer(m, w, x: np.ndarray):
    """One encoder layer over all rows, every operation a PyTorch bf16 module.
    Returns the layer output, K and V (as float64 arrays)."""
    D, h = m.dim, m.heads
    dh = D // h
    t = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float32)).to(BF)  # noqa: E731 (exact: values are bf16)
    p = lambda n: t(w[f"l0.{n}"])  # noqa: E731
    X = t(x)
    A = F.layer_norm(X, (D,), p("ln1_g"), p("ln1_b"), m.ln_eps)
    qkv = F.linear(A, p("w_qkv").T.contiguous(), p("b_qkv"))
    q, k, v = qkv.split(D, dim=-1)
    heads = lambda a: a.reshape(-1, h, dh).transpose(0, 1).contiguous()[None]  # noqa: E731
    with sdpa_kernel(SDPBackend.MATH):
        O = F.scaled_dot_product_attention(heads(q), heads(k), heads(v))[0]
    O = O.transpose(0, 1).reshape(-1, D)
    H = X + F.linear(O, p("w_o").T.contiguous(), p("b_o"))
    A2 = F.layer_norm(H, (D,), p("ln2_g"), p("ln2_b"), m.ln_eps)
    G = F.gelu(F.linear(A2, p("w_1").T.contiguous(), p("b_1")), approximate="tanh")
    out = H + F.linear(G, p("w_2").T.contiguous(), p("b_2"))
    f = lambda a: a.to(torch.float64).numpy()  # noqa: E731
    return f(out), f(k), f(v)


def oracle_layer(m, w, x):
    model = vit.Model(m, w)
    K = np.zeros((m.n_tokens, m.dim))
    V = np.zeros((m.n_tokens, m.dim))
    out = vit.layer_rows(model, 0, x, np.arange(m.n_tokens), K, V)
    return out, K, V


def _ulps(a, b):
    """Distance in bf16 ulps of b (elementwise, b nonzero)."""
    _, e = np.frexp(np.where(b == 0, 1.0, b))
    return np.abs(a - b) / np.ldexp(1.0, e - 8)


def agreement(ours, theirs):
    """(fraction of elements equal bit for bit, max distance in bf16 ulps)."""
    eq = np.mean([np.mean(a == b) for a, b in zip(ours, theirs)])
    return float(eq), float(max(_ulps(a, b).max() for a, b in zip(ours, theirs)))


@pytest.mark.parametrize("seed", [5, 17, 29])
def test_oracle_rounds_where_torch_bf16_modules_round(seed):
    m, w = _model(seed)
    x = _x(m, seed + 4)
    ours = oracle_layer(m, w, x)
    theirs = torch_bf16_layer(m, w, x)
    for a in ours:
        assert np.array_equal(a, vit.round_bf16(a))   # every stored value is a bf16 number
    eq, ulp = agreement(ours, theirs)
    assert eq >= 0.995, eq
    assert ulp <= 1.0, ulp


def _mutated(m, w, x, drop: int):
    """The oracle's layer with the drop-th call of S (in call order inside the
    layer) made the identity."""
    real = vit.S
    n = [0]

    def S(v, dt):
        n[0] += 1
        return np.asarray(v, dtype=np.float64) if n[0] == drop + 1 else real(v, dt)

    vit.S = S
    try:
        out = oracle_layer(m, w, x)
    finally:
        vit.S = real
    return out, n[0]


def test_every_rounding_point_is_detected():
    """Dropping any one of the layer's ten roundings breaks the agreement with
    the torch pipeline: the bit-equal fraction falls well below the pin's bar
    or some output moves by more than one ulp."""
    m, w = _model(5)
    x = _x(m, 9)
    theirs = torch_bf16_layer(m, w, x)
    _, calls = _mutated(m, w, x, drop=10 ** 6)
    assert calls == 10          # A, QKV, O, B, H, A2, F, G, M, X'
    for drop in range(calls):
        ours, _ = _mutated(m, w, x, drop)
        eq, ulp = agreement(ours, theirs)
        assert eq < 0.95 or ulp > 1.0, (drop, eq, ulp)


def test_both_mlp_readings_share_the_full_encode():
    """With every row refreshed the two MLP readings are the same computation,
    so their full encodes are identical bit for bit."""
    m = synth.small_model(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype="bf16")
    w = synth.make_weights(m, 13)
    x = synth.random_patches(m, 14)[0]
    a = vit.full_encode(vit.Model(m, w, mlp="reuse"), x)
    b = vit.full_encode(vit.Model(m, w, mlp="all"), x)
    for name in ("X", "K", "V", "Y"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
