"""Inputs for the method's edge cases, shared by the CPU checks of their
construction and the GPU parity tests (data only; no arithmetic of the method).

* Tied similarities: every token gets the same position vector, so two tokens
  whose patches are equal have equal embeddings; a group of tokens with equal
  patches in both frames then has equal similarities, bit for bit, on both
  sides.  With a cap inside the group the rule "equal similarities go to the
  lower index" decides which members are refreshed.
* Large-mean rows: a constant offset on the patch-embedding bias makes every
  token's mean about twenty times its spread, the case where a one-pass
  variance loses precision.
"""
from __future__ import annotations

import numpy as np

from paper_2607_12287_amd import synth


def tie_model(img: int, dtype: str = "bf16"):
    m = synth.small_model(dim=64, depth=2, heads=2, mlp=96, img=img, patch=4, dtype=dtype)
    w = synth.make_weights(m, 2100 + img)
    w["pos"][:] = w["pos"][0]          # one position vector for every token
    return m, w


def tie_frames(m, seed: int, group: int = 12, moved: int = 3):
    """Three frames [1][N][P]: frame 0; frame 1 where `group` scattered tokens
    share one new patch (they also share one patch in frame 0) and `moved`
    other tokens get unrelated new patches; frame 2 = frame 1 with the group's
    patch changed again.  Returns (frames, group indices ascending, moved)."""
    rng = np.random.default_rng(seed)
    n = m.n_tokens
    base = synth.random_patches(m, seed)[0]
    perm = rng.permutation(n)
    grp = np.sort(perm[:group])
    mov = np.sort(perm[group:group + moved])
    f0 = base.copy()
    f0[grp] = base[grp[0]]
    f1 = f0.copy()
    fresh = synth.random_patches(m, seed + 1)[0]
    f1[grp] = fresh[0]
    f1[mov] = fresh[1:1 + moved]
    f2 = f1.copy()
    f2[grp] = fresh[moved + 1]
    return [f[None].astype(np.float32) for f in (f0, f1, f2)], grp, mov


def large_mean_model(dtype: str, offset: float = 6.0):
    m = synth.small_model(dim=256, depth=2, heads=4, mlp=512, img=40, patch=4, dtype=dtype)
    w = synth.make_weights(m, 2200)
    b = (w["b_pe"] + np.float32(offset)).astype(np.float32)
    if dtype == "bf16":                  # the weights of a bf16 model are bf16 numbers
        b = synth._round_to_bf16_values(b)
    w["b_pe"] = b
    return m, w
