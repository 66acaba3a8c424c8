"""Parity of the key score (eq. 3 on first-layer keys) and of the refresh
schedule (odd/even chunks) with the CPU oracle, through the C ABI.

The cached references are the first-layer keys in key mode, computed in the
same fixed fp32 order on both sides, so `ref` is compared bit for bit, and
with it every selected index; layers and outputs keep the usual bars.
"""
import numpy as np
import pytest
import torch

from oracle import vit
from paper_2607_12287_amd import incvit, synth
from tests.gpu_util import FREE_TOL, Pair, rel_err, say, workspace_arrays

pytestmark = pytest.mark.gpu

SMALL = {
    # name: (dim, depth, heads, mlp, img, patch, dtype, B)
    "f32_d64_n16": (64, 2, 2, 96, 32, 8, "f32", 1),
    "bf16_d64_n49": (64, 2, 2, 96, 28, 4, "bf16", 2),
    "bf16_d256_n100": (256, 2, 4, 200, 40, 4, "bf16", 2),
    "bf16_d288_n64": (288, 2, 4, 300, 32, 4, "bf16", 1),
    "f32_d256_n100": (256, 2, 4, 200, 40, 4, "f32", 3),
}


def small_frames(m, B, count, seed=500):
    its = [synth.RefillRectStream(m, seed + v, v, 2 * m.patch + 3, 3 * m.patch).frames(count) for v in range(B)]
    return [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(count)]


@pytest.mark.parametrize("name", sorted(SMALL))
def test_key_score_small_models(name):
    dim, depth, heads, mlp, img, patch, dtype, B = SMALL[name]
    m = synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch, dtype=dtype)
    w = synth.make_weights(m, 200 + dim)
    say(f"[key {name}] N={m.n_tokens} D={dim} B={B}")
    frames = small_frames(m, B, 6)
    p = Pair(m, w, B, score="key")
    p.full_encode(frames[0])
    p.check_layers(None, f"{name} full")
    p.check_caches(f"{name} full")
    rng = np.random.default_rng(9)
    for t in range(1, 6):
        tau = [0.98, 0.99, np.inf, 0.98, 0.995][t - 1]
        caps = [int(rng.integers(0, m.n_tokens + 2)) if t % 2 else m.n_tokens for _ in range(B)]
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: tau={tau} caps={caps} count={count.tolist()}")
        p.check_step(idx, count, refreshed, res, f"{name} step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"{name} step {t}")
        p.check_caches(f"{name} step {t}")


def _workload_key(name, steps, oracle_views=None, rho=0.10):
    wl = synth.workload(name, rho=rho)
    m = wl.model
    say(f"[key {name}] rho={rho} views={wl.views} steps={steps}")
    p = Pair(m, wl.weights(), wl.views, oracle_views, score="key")
    frames = list(wl.patch_frames(steps + 1))
    p.full_encode(frames[0])
    p.check_layers(None, f"{name} full")
    p.check_caches(f"{name} full")
    for t in range(1, steps + 1):
        idx, count, refreshed, res = p.step(frames[t], wl.tau, wl.caps)
        p.check_step(idx, count, refreshed, res, f"{name} step {t}")
        tf = p.check_layers(lambda v: idx[v, :count[v]], f"{name} step {t}")
        worst = p.check_caches(f"{name} step {t}")
        say(f"  step {t}: count={count.tolist()} per-layer worst {tf:.2e}, free-running worst {worst:.2e}")


def test_key_score_tiny():
    _workload_key("tiny", 4)


def test_key_score_so400m():
    _workload_key("so400m", 3)


def test_key_score_so400m_448_top_k():
    _workload_key("so400m_448", 1)


def test_key_score_vitl_sampled_streams():
    _workload_key("vitl_x8", 1, oracle_views=[0, 3])


@pytest.mark.parametrize("score", ["embed", "key"])
@pytest.mark.parametrize("period", [1, 2, 3])
def test_schedule_matches_oracle(score, period):
    m = synth.small_model(dim=256, depth=2, heads=4, mlp=200, img=40, patch=4, dtype="bf16")
    w = synth.make_weights(m, 321)
    B, T = 2, 6
    frames = small_frames(m, B, T, seed=700)
    say(f"[schedule {score} period {period}] N={m.n_tokens} B={B} frames={T}")
    enc = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=B, score=score)
    buf, caches = enc.new_caches(B)
    model = vit.Model(m, w, score=score)
    caps = [m.n_tokens, 40]
    outs = [vit.run_schedule(model, [f[v] for f in frames], period, 0.98, caps[v]) for v in range(B)]
    for t in range(T):
        idx, count, refreshed = enc.encode_frame(torch.from_numpy(frames[t]).cuda(), caches, t, period, 0.98, caps)
        torch.cuda.synchronize()
        idx, count, refreshed = idx.cpu().numpy(), count.cpu().numpy(), refreshed.float().cpu().numpy()
        for v in range(B):
            r = outs[v][1][t]
            assert int(count[v]) == r.count, (t, v)
            assert np.array_equal(idx[v, :r.count], r.idx), (t, v)
            if r.count:
                assert rel_err(refreshed[v, :r.count], r.refreshed) <= FREE_TOL["bf16"], (t, v)
        say(f"  frame {t}: count={count.tolist()}")
    for v in range(B):
        g = enc.export(caches[v])
        assert np.array_equal(g["ref"], outs[v][0].ref)
        assert rel_err(g["Y"], outs[v][0].Y) <= FREE_TOL["bf16"]
    enc.close()


def test_schedule_arguments_and_mixed_modes():
    m = synth.small_model(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype="bf16")
    w = synth.make_weights(m, 77)
    x = torch.from_numpy(synth.random_patches(m, 78)).cuda()
    key = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=1, score="key")
    emb = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=1, score="embed")
    buf, caches = key.new_caches(1)
    with pytest.raises(incvit.IncvitError) as e:
        key.encode_frame(x, caches, 0, 0, 0.98, [m.n_tokens])
    assert e.value.status == incvit.INCVIT_ERR_ARG
    with pytest.raises(incvit.IncvitError) as e:
        key.encode_frame(x, caches, -1, 2, 0.98, [m.n_tokens])
    assert e.value.status == incvit.INCVIT_ERR_ARG
    # a cache encoded with the embedding score is another model's cache for the key score
    emb.full_encode(x, caches)
    torch.cuda.synchronize()
    before = key.export(caches[0])
    idx, count, _ = key.step(x, caches, np.inf, [m.n_tokens])
    assert key.status(caches[0]) == incvit.INCVIT_ERR_STATE
    assert int(count.cpu()[0]) == 0
    after = key.export(caches[0])
    for k in ("ref", "X", "K", "V", "Y"):
        assert np.array_equal(before[k], after[k]), k
    # bad score value in the config
    cfg = incvit.make_config(m)
    cfg.score = 7
    st, h = incvit.incvit_create(cfg, key.packed.data_ptr())
    assert st == incvit.INCVIT_ERR_ARG
    key.close()
    emb.close()


@pytest.mark.parametrize("score", ["embed", "key"])
@pytest.mark.parametrize("name", ["small", "so400m"])
def test_similarities_are_bit_exact(score, name):
    """The cosines themselves (not only the indices they select) equal the
    oracle's bit for bit: embedding, LayerNorm, key projection and cosine all
    follow the same fixed fp32 order with correctly rounded sqrt and divide."""
    if name == "small":
        m = synth.small_model(dim=256, depth=2, heads=4, mlp=200, img=40, patch=4, dtype="bf16")
        w = synth.make_weights(m, 901)
        frames = small_frames(m, 2, 3, seed=902)
        tau, caps = 0.98, [m.n_tokens, m.n_tokens]
    else:
        wl = synth.workload("so400m")
        m, w = wl.model, wl.weights()
        frames = list(wl.patch_frames(3))
        tau, caps = wl.tau, wl.caps
    B = frames[0].shape[0]
    say(f"[sims {score} {name}] N={m.n_tokens} D={m.dim} B={B}")
    p = Pair(m, w, B, score=score)
    p.full_encode(frames[0])
    for t in (1, 2):
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        arr = workspace_arrays(p.enc, B)
        for v in range(B):
            assert np.array_equal(arr["t0"][v], res[v].t0), (t, v, "t0")
            if score == "key":
                assert np.array_equal(arr["key"][v], res[v].sv), (t, v, "key")
            bad = np.nonzero(arr["sim"][v].view(np.int32) != res[v].sim.view(np.int32))[0]
            assert bad.size == 0, (t, v, bad[:8], arr["sim"][v][bad[:4]], res[v].sim[bad[:4]])
        p.check_step(idx, count, refreshed, res, f"sims {score} {name} {t}")
