"""Parity of the all-rows MLP reading (every row through the MLP each frame,
reused rows with their cached attention branch) with the CPU oracle, through
the C ABI; plus its invariants on the GPU: the identical frame is a fixed
point, and a stream whose step must not run is left untouched while the others
of the batch run.
"""
import numpy as np
import pytest
import torch

from paper_2607_12287_amd import incvit, synth
from tests.gpu_util import Pair, say

pytestmark = pytest.mark.gpu

SMALL = {
    # name: (dim, depth, heads, mlp, img, patch, dtype, B, score)
    "bf16_d64_n49": (64, 2, 2, 96, 28, 4, "bf16", 2, "embed"),
    "bf16_d256_n100": (256, 2, 4, 200, 40, 4, "bf16", 2, "embed"),
    "bf16_d288_n64_key": (288, 2, 4, 300, 32, 4, "bf16", 1, "key"),
    "f32_d256_n100": (256, 2, 4, 200, 40, 4, "f32", 3, "embed"),
}


def frames_of(m, B, count, seed):
    its = [synth.RefillRectStream(m, seed + v, v, 2 * m.patch + 3, 3 * m.patch).frames(count) for v in range(B)]
    return [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(count)]


@pytest.mark.parametrize("name", sorted(SMALL))
def test_all_rows_small_models(name):
    dim, depth, heads, mlp, img, patch, dtype, B, score = SMALL[name]
    m = synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch, dtype=dtype)
    w = synth.make_weights(m, 400 + dim)
    say(f"[mlp all {name}] N={m.n_tokens} D={dim} B={B} score={score}")
    frames = frames_of(m, B, 6, 800)
    p = Pair(m, w, B, score=score, mlp="all")
    p.full_encode(frames[0])
    p.check_layers(None, f"{name} full")
    p.check_caches(f"{name} full")
    rng = np.random.default_rng(11)
    for t in range(1, 6):
        tau = [0.98, 0.99, np.inf, 0.98, 0.0][t - 1]
        caps = [int(rng.integers(0, m.n_tokens + 2)) if t % 2 else m.n_tokens for _ in range(B)]
        if t == 3:
            caps[0] = 0   # a stream that refreshes nothing still moves every row
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: tau={tau} caps={caps} count={count.tolist()}")
        p.check_step(idx, count, refreshed, res, f"{name} step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"{name} step {t}")
        p.check_caches(f"{name} step {t}")


@pytest.mark.parametrize("name,steps", [("tiny", 3), ("so400m", 2)])
def test_all_rows_workloads(name, steps):
    wl = synth.workload(name)
    m = wl.model
    say(f"[mlp all {name}] views={wl.views} steps={steps}")
    p = Pair(m, wl.weights(), wl.views, mlp="all")
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


def test_all_rows_large_row_gemm():
    """600 rows per call (6 streams of 100 tokens): the MLP of every call runs
    the large-row GEMM, its down projection split over K into partial sums for
    the row kernel, in full encodes and in threshold steps alike."""
    m = synth.small_model(dim=256, depth=2, heads=4, mlp=520, img=40, patch=4, dtype="bf16")
    B = 6
    w = synth.make_weights(m, 2610)
    say(f"[mlp all, large-row GEMM] N={m.n_tokens} B={B} rows={B * m.n_tokens}")
    frames = frames_of(m, B, 3, 2620)
    p = Pair(m, w, B, mlp="all")
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    p.check_caches("full")
    for t, (tau, caps) in enumerate([(0.98, [m.n_tokens] * B), (np.inf, [30, 0, 100, 7, 64, 1])], start=1):
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: count={count.tolist()}")
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        p.check_caches(f"step {t}")


def test_all_rows_eight_vitl_streams_sampled():
    """8 ViT-L streams, 2048 rows: the full encode's output projection writes
    the attention branch through the large-row GEMM (its 64-row tiles fill the
    chip); checked on streams 0 and 5."""
    wl = synth.workload("vitl_x8")
    m = wl.model
    say("[mlp all vitl_x8] views 8, oracle views [0, 5]")
    p = Pair(m, wl.weights(), wl.views, oracle_views=[0, 5], mlp="all")
    frames = list(wl.patch_frames(2))
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    p.check_caches("full")
    idx, count, refreshed, res = p.step(frames[1], wl.tau, wl.caps)
    p.check_step(idx, count, refreshed, res, "step 1")
    tf = p.check_layers(lambda v: idx[v, :count[v]], "step 1")
    worst = p.check_caches("step 1")
    say(f"  step 1: count={count.tolist()} per-layer worst {tf:.2e}, free-running worst {worst:.2e}")


def test_all_rows_identical_frame_is_a_fixed_point_and_invalid_stream_untouched():
    m = synth.small_model(dim=256, depth=2, heads=4, mlp=200, img=40, patch=4, dtype="bf16")
    w = synth.make_weights(m, 431)
    frames = frames_of(m, 2, 2, 830)
    enc = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=2, mlp="all")
    buf, caches = enc.new_caches(2)
    x0 = torch.from_numpy(frames[0]).cuda()
    enc.full_encode(x0, caches)
    torch.cuda.synchronize()
    before = [enc.export(c) for c in caches]
    idx, count, _ = enc.step(x0, caches, 0.98, [m.n_tokens, m.n_tokens])
    assert count.cpu().tolist() == [0, 0]
    for v in range(2):
        after = enc.export(caches[v])
        for k in ("ref", "X", "K", "V", "Y", "A"):
            assert np.array_equal(before[v][k], after[k]), (v, k)
    # stream 1 never encoded: its step is a no-op, stream 0 runs
    buf2, c2 = enc.new_caches(2)
    enc.full_encode(x0[:1].contiguous(), c2[:1])
    torch.cuda.synchronize()
    empty = enc.export(c2[1])
    enc.step(torch.from_numpy(frames[1]).cuda(), c2, 0.98, [m.n_tokens, m.n_tokens])
    assert enc.status(c2[1]) == incvit.INCVIT_ERR_STATE
    assert enc.status(c2[0]) == incvit.INCVIT_OK
    after = enc.export(c2[1])
    for k in ("ref", "X", "K", "V", "Y", "A"):
        assert np.array_equal(empty[k], after[k]), k
    moved = enc.export(c2[0])
    assert not np.array_equal(moved["Y"], before[0]["Y"])
    enc.close()
