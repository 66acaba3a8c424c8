"""The large-row GEMM (bf16 calls with at least 512 rows known on the host:
full encodes, pure top-k steps) against the oracle, with ragged row tiles
(rows not a multiple of 64 or 128), a ragged column tile (the MLP width padded
to 544 = 4 x 128 + 32 columns), both tile heights (64 and 128 rows), and the
same calls on the weight-streaming GEMM (tuning tiled = 1) for comparison."""
import numpy as np
import pytest

from paper_2607_12287_amd import incvit, synth
from tests.gpu_util import Pair, say

pytestmark = pytest.mark.gpu

CASES = {
    # name: (dim, depth, heads, mlp, img, patch, B, top-k caps of the two steps)
    "rows600_cols544": (256, 2, 4, 520, 40, 4, 6, ([100, 100, 60, 100, 100, 100], [100, 37, 100, 100, 100, 100])),
    "rows2048_tile128": (768, 1, 12, 1024, 128, 4, 2, ([300, 200], [1024, 1])),
}


@pytest.mark.parametrize("tiled,fc2_mode", [(0, 0), (0, 2), (1, 0)])
@pytest.mark.parametrize("name", sorted(CASES))
def test_large_row_gemm(name, tiled, fc2_mode):
    """fc2_mode 0: the down projection split over K (its tiles are fewer than
    the CUs here); 2: unsplit, the residual and the cache write in its
    epilogue."""
    dim, depth, heads, mlp, img, patch, B, caps = CASES[name]
    m = synth.small_model(dim=dim, depth=depth, heads=heads, mlp=mlp, img=img, patch=patch, dtype="bf16")
    w = synth.make_weights(m, 2500 + dim)
    say(f"[large-row GEMM {name} tiled={tiled} fc2_mode={fc2_mode}] N={m.n_tokens} B={B} rows={B * m.n_tokens} "
        f"D={dim} F={mlp}")
    its = [synth.RefillRectStream(m, 2510 + v, v, 3 * patch + 1, 5 * patch).frames(3) for v in range(B)]
    frames = [np.stack([synth.patchify(next(it), patch) for it in its]) for _ in range(3)]
    p = Pair(m, w, B)
    incvit._check(incvit.incvit_set_tuning(p.enc.h, tiled=tiled, fc2_mode=fc2_mode), p.enc.h)
    p.full_encode(frames[0])
    tf = p.check_layers(None, "full")
    fr = p.check_caches("full")
    say(f"  full encode: per-layer worst {tf:.2e}, free-running worst {fr:.2e}")
    for t in (1, 2):
        idx, count, refreshed, res = p.step(frames[t], np.inf, caps[t - 1])
        p.check_step(idx, count, refreshed, res, f"step {t}")
        tf = p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        fr = p.check_caches(f"step {t}")
        say(f"  step {t}: rows {int(count.sum())} per-layer worst {tf:.2e}, free-running worst {fr:.2e}")

