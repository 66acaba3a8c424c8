"""Invariants the method fixes, checked on the oracle (paper §III-B).

* a 100% refresh (tau = +inf, cap = N) is the plain full forward;
* an identical repeated frame selects nothing and leaves the cache unchanged;
* reused rows (R) keep every cached value bit for bit; only rows of U change,
  and the same rows at every layer (selection happens once, before layer 1);
* the caches stay self-consistent: K^l and V^l are what layer l computes from
  its cached input rows X^l;
* a second formulation: the dense layer applied to the mixed matrix (new rows
  U, cached rows R) gives the step's rows U;
* with W_Q = W_K = 0 the attention is uniform, so an updated token's attention
  output is the mean of V over all N rows (new for U, cached for R).
"""
import numpy as np
import pytest

from oracle import vit
from paper_2607_12287_amd import synth
from tests import torch_ref


def model_and_frames(dtype="bf16", seed=21, dim=64, heads=2, mlp=96, depth=2, img=32, patch=8,
                     overrides=None):
    m = synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch,
                          dtype="bf16" if dtype == "bf16" else "f32")
    w = synth.make_weights(m, seed, overrides=overrides)
    frames = list(synth.RefillRectStream(m, seed + 1, 0, 2 * patch, 2 * patch).frames(4))
    return m, w, vit.Model(m, w, dtype=dtype), [synth.patchify(f, m.patch) for f in frames]


@pytest.mark.parametrize("dtype", ["bf16", "f32", "f64"])
def test_full_refresh_equals_full_encode(dtype):
    m, w, model, frames = model_and_frames(dtype)
    cache = vit.full_encode(model, frames[0])
    res = vit.step(model, frames[1], cache, np.inf, m.n_tokens)
    assert res.count == m.n_tokens
    ref = vit.full_encode(model, frames[1])
    for name in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(getattr(cache, name), getattr(ref, name)), name
    assert np.array_equal(res.refreshed, ref.Y)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_identical_frame_selects_nothing(dtype):
    m, w, model, frames = model_and_frames(dtype)
    cache = vit.full_encode(model, frames[0])
    before = cache.copy()
    res = vit.step(model, frames[0], cache, 0.98, m.n_tokens)
    assert res.count == 0
    assert np.all(res.sim > np.float32(0.98))
    for name in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(getattr(cache, name), getattr(before, name)), name


@pytest.mark.parametrize("dtype", ["bf16", "f32", "f64"])
def test_only_selected_rows_change(dtype):
    m, w, model, frames = model_and_frames(dtype)
    cache = vit.full_encode(model, frames[0])
    for f in frames[1:]:
        before = cache.copy()
        res = vit.step(model, f, cache, 0.98, m.n_tokens)
        U = set(res.idx.tolist())
        assert 0 < len(U) < m.n_tokens
        R = np.array(sorted(set(range(m.n_tokens)) - U))
        Ua = res.idx
        for name in ("ref", "Y"):
            a, b = getattr(cache, name), getattr(before, name)
            assert np.array_equal(a[R], b[R]), name
            assert np.all(np.any(a[Ua] != b[Ua], axis=-1)), name
        for name, depth in (("X", m.depth + 1), ("K", m.depth), ("V", m.depth)):
            a, b = getattr(cache, name), getattr(before, name)
            for l in range(depth):
                changed = np.nonzero(np.any(a[l] != b[l], axis=-1))[0].tolist()
                assert set(changed) == U, (name, l)   # the same rows at every layer


@pytest.mark.parametrize("dtype", ["bf16", "f64"])
def test_caches_stay_self_consistent(dtype):
    m, w, model, frames = model_and_frames(dtype)
    cache = vit.full_encode(model, frames[0])
    for f in frames[1:]:
        vit.step(model, f, cache, 0.98, m.n_tokens)
    for l in range(m.depth):
        if dtype == "f64":
            k, v = torch_ref.kv_of(m, w, l, torch_ref.t64(cache.X[l]))
            k, v = k.numpy(), v.numpy()
        else:  # same formula with the bf16 rounding of the LN output and of K, V
            D = m.dim
            a = vit.round_bf16(vit.layer_norm(cache.X[l], w[f"l{l}.ln1_g"], w[f"l{l}.ln1_b"], m.ln_eps))
            qkv = vit.round_bf16(a @ w[f"l{l}.w_qkv"].astype(np.float64) + w[f"l{l}.b_qkv"])
            k, v = qkv[:, D:2 * D], qkv[:, 2 * D:]
        tol = 1e-10 if dtype == "f64" else 0
        assert np.allclose(cache.K[l], k, rtol=0, atol=tol), l
        assert np.allclose(cache.V[l], v, rtol=0, atol=tol), l


def test_step_rows_equal_dense_layer_on_mixed_matrix():
    m, w, model, frames = model_and_frames("f64", depth=3)
    cache = vit.full_encode(model, frames[0])
    for f in frames[1:3]:
        vit.step(model, f, cache, 0.98, m.n_tokens)
    res = vit.step(model, frames[3], cache, 0.98, m.n_tokens)
    U = res.idx
    assert 0 < U.size < m.n_tokens
    for l in range(m.depth):
        dense = torch_ref.layer(m, w, l, torch_ref.t64(cache.X[l])).numpy()
        assert np.allclose(dense[U], cache.X[l + 1][U], rtol=0, atol=1e-10), l


def test_uniform_attention_mixes_cached_and_new_values():
    D = 64
    over = {}
    m0 = synth.small_model(dim=D, depth=2, heads=2, mlp=96, img=32, patch=8)
    for l in range(m0.depth):
        wq = synth.make_weights(m0, 31, names=(f"l{l}.w_qkv", f"l{l}.b_qkv"))
        a, b = wq[f"l{l}.w_qkv"].copy(), wq[f"l{l}.b_qkv"].copy()
        a[:, :2 * D] = 0.0
        b[:2 * D] = 0.0
        over[f"l{l}.w_qkv"], over[f"l{l}.b_qkv"] = a, b
    m, w, model, frames = model_and_frames("f64", seed=31, overrides=over)
    cache = vit.full_encode(model, frames[0])
    trace = {}
    res = vit.step(model, frames[1], cache, 0.98, m.n_tokens, trace=trace)
    assert 0 < res.count < m.n_tokens
    for l in range(m.depth):
        mean_v = cache.V[l].mean(axis=0)          # all N rows, after the scatter of U
        assert np.allclose(trace["O"][l], np.broadcast_to(mean_v, trace["O"][l].shape), atol=1e-12)
        U = res.idx
        mean_u_only = cache.V[l][U].mean(axis=0)  # what "attend among U only" would give
        assert not np.allclose(mean_v, mean_u_only, atol=1e-6)


# ----------------------------------------------------------------------------
# the workloads' streams refresh the intended share of tokens
# ----------------------------------------------------------------------------


def _counts(name, frames, rho=0.10):
    wl = synth.workload(name, rho=rho)
    m = wl.model
    w = synth.make_weights(m, wl.weight_seed, names=("w_pe", "b_pe", "pos"))
    from oracle import pinned
    counts, ref = [], None
    for t, batch in enumerate(wl.patch_frames(frames)):
        t0 = [pinned.embed_f32(batch[v], w["w_pe"], w["b_pe"], w["pos"]) for v in range(wl.views)]
        if ref is None:
            ref = t0
            continue
        row = []
        for v in range(wl.views):
            sim = pinned.cosine_f32(t0[v], ref[v])
            U = vit.select(sim, wl.tau, wl.caps[v])
            ref[v][U] = t0[v][U]
            row.append(U.size)
        counts.append(row)
    return wl, np.array(counts)


def test_tiny_stream_refresh():
    wl, c = _counts("tiny", 6)
    assert np.all(c >= 1) and np.all(c <= 20)


@pytest.mark.slow
def test_so400m_stream_refresh_is_about_ten_percent():
    wl, c = _counts("so400m", 8)
    frac = c / wl.model.n_tokens
    assert np.all(frac > 0.05) and np.all(frac < 0.16), c.ravel().tolist()


@pytest.mark.slow
def test_three_view_stream_refresh_matches_rectangles():
    wl, c = _counts("so400m_x3", 4)
    # a patch-aligned rectangle of 12 / 25 / 64 tokens is refilled each frame
    assert np.all(c == np.array([12, 25, 64])), c.tolist()


@pytest.mark.slow
def test_448_top_k_takes_exactly_the_cap():
    for rho in (0.02, 0.10):
        wl, c = _counts("so400m_448", 3, rho=rho)
        assert np.all(c == wl.caps[0]), (rho, c.tolist())
