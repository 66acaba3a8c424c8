"""The method's edge cases on the GPU, through the C ABI, against the oracle.

* Exact similarity ties straddling the cap (equal similarities go to the
  lower index, the top-rho*N rule after eq. 3), through both selection
  kernels (one wave up to 256 tokens, sixteen beyond), and a threshold equal
  to the tied value (strict comparison: none of the group is refreshed).
* Rows whose mean is twenty to eighty times their spread, through the
  LayerNorms folded into the QKV and MLP-up products (their statistics come
  from sums of x and x^2), in bf16 and fp32 models.
"""
import numpy as np
import pytest

from oracle import vit
from tests import edge_cases
from tests.gpu_util import Pair, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("img", [64, 80])
def test_tied_similarities_at_the_cap(img):
    m, w = edge_cases.tie_model(img)
    frames, grp, mov = edge_cases.tie_frames(m, 2300 + img)
    say(f"[ties] N={m.n_tokens} group={grp.tolist()} moved={mov.tolist()}")
    p = Pair(m, w, 1)
    p.full_encode(frames[0])
    p.check_layers(None, "full")
    # the tied value and the moved tokens below it, from the oracle's own cosine
    model = vit.Model(m, w)
    sim = vit.pinned.cosine_f32(vit.embed(model, frames[1][0]), p.ora[0].ref)
    tie = float(sim[grp][0])
    below = int((sim[mov] < sim[grp][0]).sum())
    # frame 2 changes the group's patch again: its five refreshed members and
    # its seven others now tie in two subgroups (different references)
    for t, cap in ((1, below + 5), (2, 9)):
        idx, count, refreshed, res = p.step(frames[t], np.inf, [cap])
        got = idx[0, :count[0]].tolist()
        say(f"  step {t}: cap={cap} count={count.tolist()} idx={got}")
        p.check_step(idx, count, refreshed, res, f"ties step {t}")
        p.check_layers(lambda v: idx[v, :count[v]], f"ties step {t}")
        if t == 1:
            assert set(grp[:5].tolist()) <= set(got) and not set(grp[5:].tolist()) & set(got)
    assert tie < 1.0


@pytest.mark.parametrize("img", [64, 80])
def test_threshold_equal_to_a_tied_similarity(img):
    m, w = edge_cases.tie_model(img)
    frames, grp, mov = edge_cases.tie_frames(m, 2300 + img)
    p = Pair(m, w, 1)
    p.full_encode(frames[0])
    sim = vit.pinned.cosine_f32(vit.embed(vit.Model(m, w), frames[1][0]), p.ora[0].ref)
    tie = float(sim[grp][0])
    idx, count, refreshed, res = p.step(frames[1], tie, [m.n_tokens])
    say(f"[tau = tied value {tie!r}] N={m.n_tokens} count={count.tolist()}")
    p.check_step(idx, count, refreshed, res, "tau = tie")
    p.check_layers(lambda v: idx[v, :count[v]], "tau = tie")
    assert not set(grp.tolist()) & set(idx[0, :count[0]].tolist())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_large_mean_rows(dtype):
    """Per layer every tensor meets the bar.  Free-running, fp32 models are
    held to the full check; bf16 models to the layer outputs X: stored in bf16
    such rows keep only a few levels across their spread, so a one-ulp
    difference in X^l moves the next LayerNorm's output (hence K, V and Y) by
    a tenth of its scale, and an fp64 implementation that differs from the
    oracle only by the LayerNorm folding drifts past the free-running bar on
    K, V and Y by itself (tests/test_oracle_edges.py)."""
    m, w = edge_cases.large_mean_model(dtype)
    from paper_2607_12287_amd import synth
    its = [synth.RefillRectStream(m, 2210 + v, v, 15, 19).frames(4) for v in range(2)]
    frames = [np.stack([synth.patchify(next(it), m.patch) for it in its]) for _ in range(4)]
    say(f"[large-mean rows {dtype}] N={m.n_tokens} D={m.dim}")
    free = ("X", "K", "V", "Y") if dtype == "f32" else ("X",)
    p = Pair(m, w, 2)
    p.full_encode(frames[0])
    tf = p.check_layers(None, "full")
    fr = p.check_caches("full", free)
    say(f"  full encode: per-layer worst {tf:.2e}, free-running worst ({'/'.join(free)}) {fr:.2e}")
    for t, caps in enumerate([[30, 60], [m.n_tokens, 7], [45, 45]], start=1):
        idx, count, refreshed, res = p.step(frames[t], np.inf, caps)
        p.check_step(idx, count, refreshed, res, f"step {t}", free_y="Y" in free)
        tf = p.check_layers(lambda v: idx[v, :count[v]], f"step {t}")
        fr = p.check_caches(f"step {t}", free)
        say(f"  step {t}: count={count.tolist()} per-layer worst {tf:.2e}, free-running worst {fr:.2e}")
