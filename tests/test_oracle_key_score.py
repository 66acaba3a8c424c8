"""Pins of the oracle's first-layer key score and of the refresh schedule.

The paper scores tokens by the cosine of their current and cached first-layer
keys (§III-B, eq. 3) and refreshes the cache with a full pass on odd chunks
(the odd/even schedule of §III-B).  Pinned here against:

* exact arithmetic: the fixed-order fp32 key score redone with rationals;
* a library routine: torch float64 LayerNorm + key projection (the first
  layer's keys as a dense forward defines them), within the fp32 error bound,
  and the oracle's own bf16 forward within the storage precision;
* special cases: zero key weights give the bias bit for bit, a constant token
  reduces LayerNorm to beta;
* invariants of the method in key mode: full refresh is the full forward, an
  identical frame selects nothing, the reference is the last refresh's key;
* the schedule: period 1 is a full forward per frame, period 2 compares every
  incremental frame with the keys of the full pass just before it, and a
  period longer than the stream is the rolling incremental stream.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pinned, vit
from paper_2607_12287_amd import synth
from tests import exact_fp32, torch_ref


def small(dtype, dim=128, heads=2, mlp=96, depth=2, img=32, patch=8):
    return synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch, dtype=dtype)


def torch_bf16(x: np.ndarray) -> np.ndarray:
    return torch.tensor(np.asarray(x, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_key_score_matches_exact_order(dtype):
    m = small(dtype)
    w = synth.make_weights(m, 41)
    model = vit.Model(m, w, score="key")
    t0 = vit.embed(model, synth.random_patches(m, 42)[0])
    key = vit.key_score(model, t0)
    D = m.dim
    for i in (0, 5, m.n_tokens - 1):
        x = torch_bf16(t0[i]) if dtype == "bf16" else t0[i]
        exact = exact_fp32.key_token(x, w["l0.ln1_g"], w["l0.ln1_b"], w["l0.w_qkv"][:, D:2 * D],
                                     w["l0.b_qkv"][D:2 * D], m.ln_eps)
        assert np.array_equal(key[i], exact), i


def test_key_score_is_the_first_layer_key_fp32():
    m = small("f32", dim=192, heads=3)
    w = synth.make_weights(m, 43)
    model = vit.Model(m, w, score="key")
    t0 = vit.embed(model, synth.random_patches(m, 44)[0])
    key = vit.key_score(model, t0).astype(np.float64)
    D = m.dim
    x = torch.tensor(t0.astype(np.float64))
    n = F.layer_norm(x, (D,), torch.tensor(w["l0.ln1_g"], dtype=torch.float64),
                     torch.tensor(w["l0.ln1_b"], dtype=torch.float64), m.ln_eps)
    wk = torch.tensor(w["l0.w_qkv"][:, D:2 * D], dtype=torch.float64)
    bk = torch.tensor(w["l0.b_qkv"][D:2 * D], dtype=torch.float64)
    ref = (n @ wk + bk).numpy()
    # the same keys through the independent dense forward of the test suite
    k_dense, _ = torch_ref.kv_of(m, w, 0, x)
    assert np.allclose(k_dense.numpy(), ref, rtol=0, atol=1e-12)
    # a chain of D fmaf roundings after a LayerNorm good to a few ulps
    bound = (D + 64) * 2.0 ** -24 * (np.abs(n.numpy()) @ np.abs(wk.numpy()) + np.abs(bk.numpy()))
    assert np.all(np.abs(key - ref) <= bound)


def test_key_score_is_the_first_layer_key_bf16():
    m = small("bf16")
    w = synth.make_weights(m, 45)
    model = vit.Model(m, w, score="key")
    x = synth.random_patches(m, 46)[0]
    cache = vit.full_encode(vit.Model(m, w), x)      # the model's own stored layer-0 keys
    key = vit.key_score(model, vit.embed(model, x)).astype(np.float64)
    err = np.abs(key - cache.K[0]).max() / np.abs(cache.K[0]).max()
    assert err < 2e-2


def test_key_score_special_cases():
    m = small("f32")
    D = m.dim
    w = synth.make_weights(m, 47)
    rng = np.random.default_rng(48)
    t0 = rng.standard_normal((4, D)).astype(np.float32)
    # zero key weights: every fmaf adds an exact zero, the key is the bias
    zero = dict(w)
    zero["l0.w_qkv"] = w["l0.w_qkv"].copy()
    zero["l0.w_qkv"][:, D:2 * D] = 0.0
    key = vit.key_score(vit.Model(m, zero, score="key"), t0)
    assert np.array_equal(key, np.broadcast_to(w["l0.b_qkv"][D:2 * D], key.shape))
    # a constant token: mean exact, variance 0, LayerNorm gives beta
    const = np.full((1, D), 0.5, np.float32)
    key = vit.key_score(vit.Model(m, w, score="key"), const).astype(np.float64)
    beta = w["l0.ln1_b"].astype(np.float64)
    wk, bk = w["l0.w_qkv"][:, D:2 * D].astype(np.float64), w["l0.b_qkv"][D:2 * D].astype(np.float64)
    ref = beta @ wk + bk
    bound = (D + 1) * 2.0 ** -24 * (np.abs(beta) @ np.abs(wk) + np.abs(bk))
    assert np.all(np.abs(key[0] - ref) <= bound)


def key_stream(dtype="bf16", seed=51, frames=5):
    m = synth.small_model(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype=dtype)
    w = synth.make_weights(m, seed)
    fr = [synth.patchify(f, m.patch) for f in synth.RefillRectStream(m, seed + 1, 0, 16, 16).frames(frames)]
    return m, w, vit.Model(m, w, score="key"), fr


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_key_mode_full_refresh_equals_full_encode(dtype):
    m, w, model, frames = key_stream(dtype)
    cache = vit.full_encode(model, frames[0])
    res = vit.step(model, frames[1], cache, np.inf, m.n_tokens)
    ref = vit.full_encode(model, frames[1])
    assert res.count == m.n_tokens
    for name in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(getattr(cache, name), getattr(ref, name)), name
    # the reference the next frame is scored against is this frame's key
    assert np.array_equal(cache.ref, vit.key_score(model, vit.embed(model, frames[1])))


def test_key_mode_identical_frame_and_reference_update():
    m, w, model, frames = key_stream()
    cache = vit.full_encode(model, frames[0])
    before = cache.copy()
    res = vit.step(model, frames[0], cache, 0.98, m.n_tokens)
    assert res.count == 0
    for name in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(getattr(cache, name), getattr(before, name)), name
    res = vit.step(model, frames[1], cache, 0.98, m.n_tokens)
    U = res.idx
    assert 0 < U.size < m.n_tokens
    # the cosine is taken between this frame's keys and the cached keys
    assert np.array_equal(res.sim, pinned.cosine_f32(res.sv, before.ref))
    assert np.array_equal(res.sv, vit.key_score(model, res.t0))
    R = np.setdiff1d(np.arange(m.n_tokens), U)
    assert np.array_equal(cache.ref[U], res.sv[U]) and np.array_equal(cache.ref[R], before.ref[R])
    # same threshold rule as the embedding score, on the key cosines
    assert np.array_equal(U, np.nonzero(res.sim < np.float32(0.98))[0])


def test_schedule_period_one_is_full_forward_each_frame():
    m, w, model, frames = key_stream(frames=3)
    cache, out = vit.run_schedule(model, frames, 1, 0.98, m.n_tokens)
    for f, r in zip(frames, out):
        full = vit.full_encode(model, f)
        assert r.count == m.n_tokens and np.array_equal(r.refreshed, full.Y)
    assert np.array_equal(cache.Y, vit.full_encode(model, frames[-1]).Y)


def test_schedule_odd_even_scores_against_the_last_full_pass():
    m, w, model, frames = key_stream(frames=5)
    cache, out = vit.run_schedule(model, frames, 2, 0.98, m.n_tokens)
    for t in (1, 3):
        k_now = vit.key_score(model, vit.embed(model, frames[t]))
        k_full = vit.key_score(model, vit.embed(model, frames[t - 1]))
        assert np.array_equal(out[t].sim, pinned.cosine_f32(k_now, k_full)), t
        assert 0 < out[t].count < m.n_tokens
    for t in (0, 2, 4):
        assert out[t].count == m.n_tokens


def test_schedule_long_period_is_the_rolling_stream():
    m, w, model, frames = key_stream(frames=4)
    cache, out = vit.run_schedule(model, frames, 100, 0.98, m.n_tokens)
    roll = vit.full_encode(model, frames[0])
    for t in range(1, 4):
        r = vit.step(model, frames[t], roll, 0.98, m.n_tokens)
        assert np.array_equal(r.idx, out[t].idx) and np.array_equal(r.refreshed, out[t].refreshed)
    for name in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(getattr(cache, name), getattr(roll, name)), name
