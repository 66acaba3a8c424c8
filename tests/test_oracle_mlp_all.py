"""Pins of the oracle's non-exact reading of the MLP statement of §III-B
(every token goes through the MLP): reused rows add their cached attention-branch output
to their current residual stream, and the MLP runs over every row.

* 100% refresh is the plain full forward of the same reading;
* an identical frame is a fixed point: nothing in the cache changes;
* a frame that selects nothing still moves every reused row with the new
  embedding, while K, V and the references stay cached;
* the rows equal an independent torch float64 dense formulation of the layer
  in which the attention branch of the reused rows is replaced by its cached
  value;
* the attention-branch cache holds S(O W_o + b_o) as the dense forward
  computes it.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import vit
from paper_2607_12287_amd import synth
from tests import torch_ref


def stream(dtype="bf16", seed=61, frames=4, depth=2):
    m = synth.small_model(dim=64, depth=depth, heads=2, mlp=96, img=32, patch=8,
                          dtype="bf16" if dtype == "bf16" else "f32")
    w = synth.make_weights(m, seed)
    fr = [synth.patchify(f, m.patch) for f in synth.RefillRectStream(m, seed + 1, 0, 16, 16).frames(frames)]
    return m, w, vit.Model(m, w, dtype=dtype, mlp="all"), fr


@pytest.mark.parametrize("dtype", ["bf16", "f32", "f64"])
def test_full_refresh_equals_full_encode(dtype):
    m, w, model, frames = stream(dtype)
    cache = vit.full_encode(model, frames[0])
    res = vit.step(model, frames[1], cache, np.inf, m.n_tokens)
    ref = vit.full_encode(model, frames[1])
    assert res.count == m.n_tokens
    for name in ("ref", "X", "K", "V", "Y", "A"):
        assert np.array_equal(getattr(cache, name), getattr(ref, name)), name


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_identical_frame_is_a_fixed_point(dtype):
    m, w, model, frames = stream(dtype)
    cache = vit.full_encode(model, frames[0])
    before = cache.copy()
    res = vit.step(model, frames[0], cache, 0.98, m.n_tokens)
    assert res.count == 0
    for name in ("ref", "X", "K", "V", "Y", "A"):
        assert np.array_equal(getattr(cache, name), getattr(before, name)), name


def test_reused_rows_follow_the_new_frame():
    m, w, model, frames = stream("bf16")
    cache = vit.full_encode(model, frames[0])
    before = cache.copy()
    res = vit.step(model, frames[1], cache, 0.0, m.n_tokens)   # tau = 0 selects nothing
    assert res.count == 0
    for name in ("ref", "K", "V", "A"):
        assert np.array_equal(getattr(cache, name), getattr(before, name)), name
    assert np.array_equal(cache.X[0], vit.S(res.t0.astype(np.float64), "bf16"))
    moved = np.any(cache.Y != before.Y, axis=1)
    assert moved.mean() > 0.5          # most rows' outputs move with the new embedding
    # the exact reading leaves everything in place on the same frame
    exact = vit.Model(m, w)
    c2 = vit.full_encode(exact, frames[0])
    b2 = c2.copy()
    vit.step(exact, frames[1], c2, 0.0, m.n_tokens)
    assert np.array_equal(c2.Y, b2.Y)


def test_rows_equal_dense_formulation_with_cached_branch():
    m, w, model, frames = stream("f64", depth=3)
    cache = vit.full_encode(model, frames[0])
    for f in frames[1:3]:
        vit.step(model, f, cache, 0.98, m.n_tokens)
    before = cache.copy()
    res = vit.step(model, frames[3], cache, 0.98, m.n_tokens)
    U = res.idx
    assert 0 < U.size < m.n_tokens
    D, h = m.dim, m.heads
    dh = D // h
    t = torch_ref.t64
    x = t(vit.S(res.t0.astype(np.float64), "f64"))
    for l in range(m.depth):
        g = lambda n: t(w[f"l{l}.{n}"])  # noqa: E731
        k, v = t(before.K[l]).clone(), t(before.V[l]).clone()
        a = F.layer_norm(x[U], (D,), g("ln1_g"), g("ln1_b"), m.ln_eps)
        q, kn, vn = F.linear(a, g("w_qkv").T, g("b_qkv")).split(D, dim=-1)
        k[U], v[U] = kn, vn
        heads = lambda z: z.reshape(-1, h, dh).transpose(0, 1)  # noqa: E731
        o = F.scaled_dot_product_attention(heads(q)[None], heads(k)[None], heads(v)[None])[0]
        branch = t(before.A[l]).clone()
        branch[U] = F.linear(o.transpose(0, 1).reshape(-1, D), g("w_o").T, g("b_o"))
        hres = x + branch
        a2 = F.layer_norm(hres, (D,), g("ln2_g"), g("ln2_b"), m.ln_eps)
        x = hres + F.linear(F.gelu(F.linear(a2, g("w_1").T, g("b_1")), approximate="tanh"), g("w_2").T, g("b_2"))
        assert np.allclose(cache.A[l], branch.numpy(), rtol=0, atol=1e-10), l
        assert np.allclose(cache.X[l + 1], x.numpy(), rtol=0, atol=1e-10 * max(1.0, float(x.abs().max()))), l
        assert np.allclose(cache.K[l], k.numpy(), rtol=0, atol=1e-10), l


def test_branch_cache_of_full_encode_matches_dense_forward():
    m, w, model, frames = stream("f64")
    cache = vit.full_encode(model, frames[0])
    xs, y = torch_ref.forward_from_tokens(m, w, torch_ref.t64(cache.X[0]))
    for l in range(m.depth):
        # in a full forward the branch is X^{l} -> H - X^{l}
        D = m.dim
        g = lambda n: torch_ref.t64(w[f"l{l}.{n}"])  # noqa: E731
        hres = xs[l] + torch.tensor(cache.A[l])
        a2 = F.layer_norm(hres, (D,), g("ln2_g"), g("ln2_b"), m.ln_eps)
        out = hres + F.linear(F.gelu(F.linear(a2, g("w_1").T, g("b_1")), approximate="tanh"), g("w_2").T, g("b_2"))
        assert np.allclose(out.numpy(), xs[l + 1].numpy(), rtol=0, atol=1e-10)
    assert np.allclose(cache.Y, y.numpy(), rtol=0, atol=1e-10)
