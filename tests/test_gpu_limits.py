"""Parity at the library's limits, through the C ABI: the most streams a call
takes (64), the most tokens (4096, selection and attention over 128 key
blocks, threshold and top-k with many candidates), and the widest model
(D = 2048 with 128-wide heads, both score modes).  Every cache and the
workspace sit between guard bands of a fixed byte pattern that must survive
every call."""
import numpy as np
import pytest

from paper_2607_12287_amd import synth
from tests.gpu_util import Pair, say

pytestmark = pytest.mark.gpu


def frames_of(m, B, count, seed, rh, rw):
    its = [synth.RefillRectStream(m, seed + v, v, rh, rw).frames(count) for v in range(B)]
    return [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(count)]


GUARD = 8192  # guard bytes around every cache and the workspace


def run(p, frames, steps):
    p.full_encode(frames[0])
    p.check_guards("full")
    p.check_layers(None, "full")
    p.check_caches("full")
    for t, (tau, caps) in enumerate(steps, start=1):
        idx, count, refreshed, res = p.step(frames[t], tau, caps)
        say(f"  step {t}: tau={tau} counts {count.tolist()[:8]}{'...' if len(caps) > 8 else ''}")
        p.check_guards(f"step {t}")
        p.check_step(idx, count, refreshed, res, f"step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        p.check_caches(f"step {t}")


def test_sixty_four_streams():
    m = synth.small_model(dim=64, depth=2, heads=2, mlp=96, img=32, patch=8, dtype="bf16")
    w = synth.make_weights(m, 1201)
    B = 64
    say(f"[limits: {B} streams] N={m.n_tokens}")
    frames = frames_of(m, B, 3, 1210, 11, 13)
    rng = np.random.default_rng(3)
    caps = [int(c) for c in rng.integers(0, m.n_tokens + 1, B)]
    p = Pair(m, w, B, oracle_views=sorted(set(range(0, B, 7)) | {B - 1}), guard=GUARD)
    run(p, frames, [(0.98, [m.n_tokens] * B), (np.inf, caps)])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_four_thousand_tokens(dtype):
    m = synth.small_model(dim=64, depth=1, heads=2, mlp=96, img=256, patch=4, dtype=dtype)
    assert m.n_tokens == 4096
    w = synth.make_weights(m, 1301)
    say(f"[limits: N={m.n_tokens} {dtype}]")
    frames = frames_of(m, 1, 3, 1310, 60, 90)
    p = Pair(m, w, 1, guard=GUARD)
    run(p, frames, [(0.98, [m.n_tokens]), (np.inf, [1000])])


@pytest.mark.parametrize("score", ["embed", "key"])
def test_widest_model(score):
    m = synth.small_model(dim=2048, depth=1, heads=16, mlp=512, img=32, patch=8, dtype="bf16")
    assert m.head_dim == 128
    w = synth.make_weights(m, 1401)
    say(f"[limits: D={m.dim} dh={m.head_dim} score={score}]")
    frames = frames_of(m, 2, 3, 1410, 9, 17)
    p = Pair(m, w, 2, score=score, guard=GUARD)
    run(p, frames, [(0.98, [m.n_tokens, 5]), (np.inf, [3, m.n_tokens])])
