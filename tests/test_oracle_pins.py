"""Pins of the CPU oracle against things other than itself.

* library routines: torch float64 functional ops (conv2d, layer_norm, linear,
  scaled_dot_product_attention, gelu) -- ``torch_ref``;
* exact arithmetic: the fixed fp32 embedding and cosine redone with rationals;
* closed forms and textbook special cases;
* brute-force selection.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pinned, vit
from paper_2607_12287_amd import synth
from tests import exact_fp32, torch_ref


def small(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype="f64"):
    return synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch,
                             dtype="f32" if dtype == "f64" else dtype)


# ----------------------------------------------------------------------------
# storage rounding
# ----------------------------------------------------------------------------


def test_round_bf16_matches_torch_on_fp32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 3,
                        rng.standard_normal(2000).astype(np.float32) * 1e-3])
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(vit.round_bf16(x.astype(np.float64)), ref)


def test_round_bf16_ties_to_even():
    # 1 + 2^-8 lies half way between 1 and 1 + 2^-7: ties go to the even 1.0;
    # 1 + 3*2^-8 lies half way between 1 + 2^-7 and 1 + 2^-6: goes to 1 + 2^-6.
    x = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), 0.0, 2.0 ** -20 * 1.5])
    assert vit.round_bf16(x).tolist() == [1.0, 1 + 2.0 ** -6, -1.0, 0.0, 2.0 ** -20 * 1.5]


def test_storage_modes():
    x = np.array([1 / 3, -2.5e-4, 7.0])
    assert np.array_equal(vit.S(x, "f64"), x)
    assert np.array_equal(vit.S(x, "f32"), x.astype(np.float32).astype(np.float64))


# ----------------------------------------------------------------------------
# elementary ops vs torch and closed forms
# ----------------------------------------------------------------------------


def test_layer_norm_vs_torch_and_constant_row():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96)) * 3 + 1
    g = rng.standard_normal(96)
    b = rng.standard_normal(96)
    ref = F.layer_norm(torch.tensor(x), (96,), torch.tensor(g), torch.tensor(b), 1e-6).numpy()
    assert np.allclose(vit.layer_norm(x, g, b, 1e-6), ref, rtol=0, atol=1e-12)
    const = np.full((1, 96), 5.0)
    assert np.allclose(vit.layer_norm(const, g, b, 1e-6), b, atol=0)


def test_gelu_tanh_vs_torch_and_closed_forms():
    x = np.linspace(-8, 8, 1001)
    ref = F.gelu(torch.tensor(x), approximate="tanh").numpy()
    assert np.allclose(vit.gelu_tanh(x), ref, rtol=0, atol=1e-14)
    assert vit.gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(vit.gelu_tanh(np.array([30.0]))[0] - 30.0) < 1e-12


def test_attention_vs_sdpa_and_uniform_case():
    rng = np.random.default_rng(2)
    h, dh, n, m = 3, 16, 11, 5
    q = rng.standard_normal((m, h * dh))
    k = rng.standard_normal((n, h * dh))
    v = rng.standard_normal((n, h * dh))
    split = lambda t: torch.tensor(t).reshape(-1, h, dh).transpose(0, 1)[None]
    ref = F.scaled_dot_product_attention(split(q), split(k), split(v))[0].transpose(0, 1).reshape(m, -1)
    assert np.allclose(vit.attention(q, k, v, h), ref.numpy(), rtol=0, atol=1e-12)
    # zero queries: every key scores the same, so the output is the mean of V
    out = vit.attention(np.zeros((2, h * dh)), k, v, h)
    assert np.allclose(out, np.broadcast_to(v.mean(axis=0), out.shape), atol=1e-13)


# ----------------------------------------------------------------------------
# the fixed-order fp32 embedding and cosine
# ----------------------------------------------------------------------------


def test_pinned_embed_matches_exact_fmaf_chain():
    m = small(dim=64, img=16, patch=4)
    w = synth.make_weights(m, 5, names=("w_pe", "b_pe", "pos"))
    x = synth.random_patches(m, 3)[0]
    t0 = pinned.embed_f32(x, w["w_pe"], w["b_pe"], w["pos"])
    for i in (0, 7, 15):
        exact = exact_fp32.embed_token(x[i], w["w_pe"], w["b_pe"], w["pos"][i])
        assert np.array_equal(t0[i], exact), i


def test_pinned_cosine_matches_exact_order():
    rng = np.random.default_rng(4)
    a = rng.standard_normal((4, 128)).astype(np.float32)
    b = (a + 0.01 * rng.standard_normal((4, 128))).astype(np.float32)
    b[3] = rng.standard_normal(128).astype(np.float32)
    sim = pinned.cosine_f32(a, b)
    for i in range(4):
        assert sim[i] == exact_fp32.cosine(a[i], b[i]), i


def test_pinned_embed_vs_conv2d_fp64():
    for m in (small(dim=64, img=32, patch=8), synth.TINY):
        w = synth.make_weights(m, 6, names=("w_pe", "b_pe", "pos"))
        rng = np.random.default_rng(9)
        frame = synth.add_pixel_noise(rng, synth.smooth_noise(rng, m.channels, m.img_h, m.img_w))
        t0 = pinned.embed_f32(synth.patchify(frame, m.patch), w["w_pe"], w["b_pe"], w["pos"])
        ref = torch_ref.conv_embed(m, w, frame).numpy()
        # a chain of P fp32 fmaf roundings: |err| <= (P + 1) * 2^-24 * sum|terms|
        bound = (m.patch_dim + 1) * 2.0 ** -24 * (np.abs(synth.patchify(frame, m.patch)) @ np.abs(w["w_pe"])
                                                   + np.abs(w["b_pe"]) + np.abs(w["pos"]))
        assert np.all(np.abs(t0 - ref) <= bound)


def test_pinned_cosine_accuracy_and_special_cases():
    rng = np.random.default_rng(7)
    a = rng.standard_normal((50, 192)).astype(np.float32)
    b = (a + 0.05 * rng.standard_normal((50, 192))).astype(np.float32)
    sim = pinned.cosine_f32(a, b)
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    ref = (a64 * b64).sum(1) / np.linalg.norm(a64, axis=1) / np.linalg.norm(b64, axis=1)
    assert np.max(np.abs(sim - ref)) <= 1e-5
    self_sim = pinned.cosine_f32(a, a)
    assert np.all(np.abs(self_sim - 1.0) <= 4 * 2.0 ** -24 * 2)
    assert np.all(np.abs(pinned.cosine_f32(a, -a) + 1.0) <= 8 * 2.0 ** -24)
    zero = np.zeros((1, 192), np.float32)
    assert pinned.cosine_f32(zero, a[:1])[0] == 0.0


# ----------------------------------------------------------------------------
# selection
# ----------------------------------------------------------------------------


def brute_select(sim, tau, cap):
    n = len(sim)
    cand = [i for i in range(n) if np.float32(sim[i]) < np.float32(tau)]
    cand.sort(key=lambda i: (float(sim[i]), i))
    return sorted(cand[:max(0, min(cap, n))])


@pytest.mark.parametrize("seed", range(40))
def test_select_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 70))
    # few distinct values so that ties are common
    sim = rng.choice(np.float32([0.5, 0.9, 0.97, 0.98, 0.99, 1.0]), n).astype(np.float32)
    tau = float(rng.choice([0.98, 0.99, np.inf, 0.0, 1.5]))
    cap = int(rng.integers(0, n + 3))
    assert vit.select(sim, tau, cap).tolist() == brute_select(sim, tau, cap)


def test_select_strict_threshold_and_nan():
    sim = np.float32([0.98, 0.97, 0.99])
    assert vit.select(sim, 0.98, 10).tolist() == [1]
    with pytest.raises(ValueError):
        vit.select(np.float32([0.5, np.nan]), 0.98, 10)


# ----------------------------------------------------------------------------
# full forward vs an independent torch float64 ViT
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("shape", ["small", "dh72", "tiny"])
def test_full_encode_f64_matches_torch(shape):
    if shape == "small":
        m = small(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8)
    elif shape == "dh72":
        m = small(dim=144, depth=2, heads=2, mlp=100, img=28, patch=7)
    else:
        m = synth.TINY
    w = synth.make_weights(m, 11)
    x = synth.random_patches(m, 12)[0]
    model = vit.Model(m, w, dtype="f64")
    cache = vit.full_encode(model, x)
    xs, y = torch_ref.forward_from_tokens(m, w, torch_ref.t64(cache.ref))
    for l in range(m.depth + 1):
        assert np.allclose(cache.X[l], xs[l].numpy(), rtol=0, atol=1e-10 * max(1, np.abs(cache.X[l]).max()))
    assert np.allclose(cache.Y, y.numpy(), rtol=0, atol=1e-10)
    for l in range(m.depth):
        k, v = torch_ref.kv_of(m, w, l, xs[l])
        assert np.allclose(cache.K[l], k.numpy(), rtol=0, atol=1e-10)
        assert np.allclose(cache.V[l], v.numpy(), rtol=0, atol=1e-10)


def test_storage_rounding_stays_close_to_f64():
    m = small(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype="bf16")
    w = synth.make_weights(m, 13)
    x = synth.random_patches(m, 14)[0]
    y64 = vit.full_encode(vit.Model(m, w, dtype="f64"), x).Y
    y16 = vit.full_encode(vit.Model(m, w, dtype="bf16"), x).Y
    assert np.array_equal(y16, vit.round_bf16(y16))      # stored values are bf16 numbers
    err = np.abs(y16 - y64).max() / np.abs(y64).max()
    assert 1e-4 < err < 3e-2
