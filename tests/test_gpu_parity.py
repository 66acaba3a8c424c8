"""Parity of the HIP path with the CPU oracle, through the C ABI.

Small models span several GEMM row/column tiles, K splits, head dims 32/64/72
and token counts with ragged tails; the five workloads run at full size on
sampled frames (and sampled streams where the oracle would be slow).
"""
import numpy as np
import pytest

from paper_2607_12287_amd import synth
from tests.gpu_util import Pair, say

pytestmark = pytest.mark.gpu

SMALL = {
    # name: (dim, depth, heads, mlp, img, patch, dtype, B)
    "f32_dh32_n16": (64, 2, 2, 96, 32, 8, "f32", 1),
    "bf16_dh32_n49": (64, 2, 2, 96, 28, 4, "bf16", 2),
    "bf16_dh64_n100_split": (256, 2, 4, 200, 40, 4, "bf16", 2),
    "bf16_dh72_n64": (288, 2, 4, 300, 32, 4, "bf16", 1),
    "f32_dh64_n100_split": (256, 2, 4, 200, 40, 4, "f32", 3),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_models_stream(name):
    dim, depth, heads, mlp, img, patch, dtype, B = SMALL[name]
    m = synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch, dtype=dtype)
    w = synth.make_weights(m, 100 + dim)
    say(f"[{name}] N={m.n_tokens} D={dim} dh={m.head_dim} F={mlp} B={B}")
    streams = [synth.RefillRectStream(m, 300 + v, v, 2 * patch + 3, 3 * patch) for v in range(B)]
    its = [s.frames(6) for s in streams]
    frames = [np.stack([synth.patchify(next(it), patch) for it in its]) for _ in range(6)]
    p = Pair(m, w, B)
    p.full_encode(frames[0])
    p.check_layers(None, f"{name} full")
    p.check_caches(f"{name} full")
    rng = np.random.default_rng(7)
    for t in range(1, 6):
        tau = [0.98, 0.99, np.inf, 0.98, 0.995][t - 1]
        caps = [int(rng.integers(0, m.n_tokens + 2)) if t % 2 else m.n_tokens for _ in range(B)]
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: tau={tau} caps={caps} count={count.tolist()}")
        p.check_step(idx, count, refreshed, res, f"{name} step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"{name} step {t}")
        p.check_caches(f"{name} step {t}")


def _workload_run(name, steps, oracle_views=None, rho=0.10, row_groups=0):
    """Full encode, then `steps` steps of the workload's stream, each checked
    per layer (teacher-forced) and free-running; prints the worst error of
    each step so that any growth over the stream shows."""
    wl = synth.workload(name, rho=rho)
    m = wl.model
    say(f"[{name}] rho={rho} views={wl.views} steps={steps} row_groups={row_groups}")
    w = wl.weights()
    p = Pair(m, w, wl.views, oracle_views)
    if row_groups:
        from paper_2607_12287_amd import incvit
        incvit._check(incvit.incvit_set_tuning(p.enc.h, row_groups=row_groups), p.enc.h)
    frames = list(wl.patch_frames(steps + 1))
    p.full_encode(frames[0])
    tf = p.check_layers(None, f"{name} full")
    worst = p.check_caches(f"{name} full")
    say(f"  full encode: per-layer worst {tf:.2e}, free-running worst {worst:.2e}")
    hist = []
    for t in range(1, steps + 1):
        idx, count, refreshed, res = p.step(frames[t], wl.tau, wl.caps)
        p.check_step(idx, count, refreshed, res, f"{name} step {t}")
        tf = p.check_layers(lambda v: idx[v, :count[v]], f"{name} step {t}")
        worst = p.check_caches(f"{name} step {t}")
        hist.append((tf, worst))
        say(f"  step {t}: count={count.tolist()} per-layer worst {tf:.2e}, free-running worst {worst:.2e}")
    if hist:
        say(f"  over {steps} steps: per-layer worst {max(h[0] for h in hist):.2e}, "
            f"free-running worst {max(h[1] for h in hist):.2e}")
    return hist


def test_tiny_workload():
    _workload_run("tiny", 8)


def test_so400m_full_stream():
    """The 64-frame stream of the So400m workload: a full encode and all 63 steps."""
    _workload_run("so400m", 63)


@pytest.mark.parametrize("row_groups,steps", [(0, 32), (4, 2)])
def test_so400m_three_views(row_groups, steps):
    """32 frames of the three-stream workload; row_groups 4 (two steps): the
    threshold steps' GEMM row groups that a caller expecting about a hundred
    rows sets (each GEMM then takes its own share of them)."""
    _workload_run("so400m_x3", steps, row_groups=row_groups)


@pytest.mark.parametrize("rho", [0.02, 0.05, 0.10, 0.25, 0.50, 1.0])
def test_so400m_448_top_k(rho):
    _workload_run("so400m_448", 1, rho=rho)


@pytest.mark.parametrize("row_groups,steps", [(0, 32), (6, 2)])
def test_vitl_eight_streams_sampled(row_groups, steps):
    _workload_run("vitl_x8", steps, oracle_views=[0, 5], row_groups=row_groups)


@pytest.mark.parametrize("waves", [2, 4, 8])
@pytest.mark.parametrize("qtiles", [1, 2])
def test_attention_tunings(waves, qtiles):
    """Every attention workgroup shape (waves splitting the keys, query tiles
    per workgroup) meets the parity bar: they differ only in the order of the
    fp32 partial sums."""
    from paper_2607_12287_amd import incvit
    m = synth.small_model(dim=288, depth=2, heads=4, mlp=300, img=64, patch=4, dtype="bf16")
    w = synth.make_weights(m, 951)
    say(f"[attn waves={waves} qtiles={qtiles}] N={m.n_tokens} dh={m.head_dim}")
    its = [synth.RefillRectStream(m, 960 + v, v, 21, 30).frames(3) for v in range(2)]
    frames = [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(3)]
    p = Pair(m, w, 2)
    incvit._check(incvit.incvit_set_tuning(p.enc.h, attn_qtiles=qtiles, attn_waves=waves), p.enc.h)
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    for t in (1, 2):
        idx, count, refreshed, res = p.step(frames[t], 0.98, [m.n_tokens, 40])
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_down_projection_modes(mode, dtype):
    """Both forms of the MLP down projection (K split with a row kernel; whole
    K with the residual and the cache write in the epilogue, on every layer but
    the last) meet the parity bar, in full encodes and steps."""
    from paper_2607_12287_amd import incvit
    m = synth.small_model(dim=256, depth=3, heads=4, mlp=520, img=40, patch=4, dtype=dtype)
    w = synth.make_weights(m, 971)
    say(f"[fc2 mode {mode} {dtype}] N={m.n_tokens} F={m.mlp_dim}")
    its = [synth.RefillRectStream(m, 980 + v, v, 15, 19).frames(3) for v in range(2)]
    frames = [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(3)]
    p = Pair(m, w, 2)
    incvit._check(incvit.incvit_set_tuning(p.enc.h, fc2_mode=mode), p.enc.h)
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    p.check_caches("full")
    for t in (1, 2):
        idx, count, refreshed, res = p.step(frames[t], [0.98, np.inf][t - 1], [m.n_tokens, 30])
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        p.check_caches(f"step {t}")


def test_down_projection_fused_so400m():
    from paper_2607_12287_amd import incvit
    wl = synth.workload("so400m")
    say("[fc2 mode 2 so400m]")
    p = Pair(wl.model, wl.weights(), 1)
    incvit._check(incvit.incvit_set_tuning(p.enc.h, fc2_mode=2), p.enc.h)
    frames = list(wl.patch_frames(3))
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    for t in (1, 2):
        idx, count, refreshed, res = p.step(frames[t], wl.tau, wl.caps)
        p.check_step(idx, count, refreshed, res, f"step {t}")
        tf = p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        worst = p.check_caches(f"step {t}")
        say(f"  step {t}: count={count.tolist()} per-layer worst {tf:.2e}, free-running worst {worst:.2e}")


@pytest.mark.parametrize("case", ["3x2", "4x2"])
@pytest.mark.parametrize("score", ["embed", "key"])
def test_patch16_register_tiles(case, score):
    """Patch 16 (P = 768, 12 LDS tiles of k) through each register tile of the
    fixed-order product that has an unrolled 12-tile form: one stream of 64
    tokens takes 3 tokens x 2 columns per thread, 8 streams of 256 tokens at
    D = 768 take 4 x 2 (fewer workgroup rounds); with the key score at
    D = 768 the key projection (K = 768, 12 tiles) takes the same tile, at
    D = 128 the tile loop.  Selection is checked bit-exactly, so the product
    must keep its fma order."""
    if case == "3x2":
        m = synth.small_model(dim=128, depth=1, heads=2, mlp=160, img=128, patch=16, dtype="bf16")
        B, views = 2, None
    else:
        m = synth.small_model(dim=768, depth=1, heads=8, mlp=256, img=256, patch=16, dtype="bf16")
        B, views = 8, [0, 7]
    assert m.patch_dim == 768
    w = synth.make_weights(m, 1501)
    say(f"[patch 16 {case} {score}] N={m.n_tokens} D={m.dim} B={B}")
    its = [synth.RefillRectStream(m, 1510 + v, v, 37, 45).frames(3) for v in range(B)]
    frames = [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(3)]
    p = Pair(m, w, B, oracle_views=views, score=score)
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    for t, (tau, cap) in enumerate([(0.98, m.n_tokens), (np.inf, 9)], start=1):
        idx, count, refreshed, res = p.step(frames[t], tau, [cap] * B)
        say(f"  step {t}: count={count.tolist()}")
        assert count.sum() > 0 if t == 1 else (count == 9).all()
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("cols", [(4, 4, 4, 4), (1, 2, 1, 2)])
def test_gemm_column_blocks(cols, mode):
    """GEMM workgroups of one, two and four 16-column blocks (every epilogue:
    QKV with the folded LayerNorm and the K/V scatter, output projection with
    the residual, MLP up with GELU, MLP down as K-split partial sums or whole
    K with the residual) in full encodes (8 row groups) and steps: the column
    count changes which workgroup computes a column, never its sum order."""
    from paper_2607_12287_amd import incvit
    m = synth.small_model(dim=256, depth=2, heads=4, mlp=512, img=64, patch=4, dtype="bf16")
    w = synth.make_weights(m, 1601)
    say(f"[gemm cols={cols} fc2 mode {mode}] N={m.n_tokens} D={m.dim} F={m.mlp_dim}")
    its = [synth.RefillRectStream(m, 1610 + v, v, 23, 29).frames(3) for v in range(2)]
    frames = [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(3)]
    p = Pair(m, w, 2)
    incvit._check(incvit.incvit_set_tuning(p.enc.h, cols=cols, fc2_mode=mode), p.enc.h)
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    p.check_caches("full")
    for t, (tau, caps) in enumerate([(0.98, [m.n_tokens, 50]), (np.inf, [200, 37])], start=1):
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: count={count.tolist()}")
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        p.check_caches(f"step {t}")
