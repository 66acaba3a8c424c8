"""Invariants of the HIP path, through the C ABI (paper §III-B: reused rows keep
their cached values; the selection is made once and applied to every layer).

Error paths are forced from the host (NaN frame, never-encoded cache, bad
arguments); every kernel still runs to completion.
"""
import math

import numpy as np
import pytest
import torch

from paper_2607_12287_amd import incvit, synth
from tests.gpu_util import TOL, Pair, rel_err, say

pytestmark = pytest.mark.gpu


def _setup(dtype="bf16", B=2, dim=256, heads=4, mlp=200, img=40, patch=4, frames=4, seed=5, score="embed",
           mlp_mode="reuse"):
    m = synth.small_model(dim=dim, depth=2, heads=heads, mlp=mlp, img=img, patch=patch, dtype=dtype)
    w = synth.make_weights(m, seed)
    enc = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=max(B, 2), score=score, mlp=mlp_mode)
    streams = [synth.RefillRectStream(m, seed + 10 + v, v, 2 * patch + 5, 3 * patch) for v in range(B)]
    its = [s.frames(frames) for s in streams]
    fr = [torch.from_numpy(np.stack([synth.patchify(next(it), patch) for it in its])).cuda() for _ in range(frames)]
    return m, w, enc, fr


def _raw(enc, caches):
    torch.cuda.synchronize()
    return [enc.export_raw(c).clone() for c in caches]


MODES = [("embed", "reuse", 1), ("key", "reuse", 1), ("embed", "all", 1), ("key", "all", 1), ("embed", "reuse", 3)]


@pytest.mark.parametrize("score,mlp_mode,row_groups", MODES)
def test_step_graph_replays_match_eager_steps(score, mlp_mode, row_groups):
    m, w, enc, fr = _setup(score=score, mlp_mode=mlp_mode)
    if row_groups > 1:
        incvit._check(incvit.incvit_set_tuning(enc.h, row_groups=row_groups), enc.h)
    B = 2
    caps = [m.n_tokens, 9]
    bufa, ca = enc.new_caches(B)
    bufb, cb = enc.new_caches(B)
    enc.full_encode(fr[0], ca)
    enc.full_encode(fr[0], cb)
    inp = torch.empty_like(fr[0])
    out_g = (torch.empty((B, m.n_tokens), dtype=torch.int32, device="cuda"),
             torch.empty((B,), dtype=torch.int32, device="cuda"),
             torch.empty((B, m.n_tokens, m.dim), dtype=enc.dtype, device="cuda"))
    g = enc.step_graph(inp, ca, 0.98, caps, out_g)
    try:
        for t in range(1, 4):
            say(f"replay {t}")
            inp.copy_(fr[t])
            enc.launch(g)
            idx, count, refreshed = enc.step(fr[t], cb, 0.98, caps)   # eager work between replays
            torch.cuda.synchronize()
            assert torch.equal(out_g[1], count)
            for v in range(B):
                k = int(count[v])
                assert torch.equal(out_g[0][v, :k], idx[v, :k])
                assert torch.equal(out_g[2][v, :k], refreshed[v, :k])
            for x, y in zip(_raw(enc, ca), _raw(enc, cb)):
                assert torch.equal(x, y)
    finally:
        enc.drop_graph(g)


@pytest.mark.parametrize("name,row_groups", [("so400m", 1), ("vitl_x8", 6), ("so400m_448", 0)])
def test_workload_graph_replays_match_eager_steps(name, row_groups):
    """The launch configuration the benchmark times: the full-size workload's
    step captured in a HIP graph (the bench's GEMM row groups) and replayed on
    consecutive frames gives bit for bit the outputs and caches of the eager
    steps, which the oracle parity tests check."""
    wl = synth.workload(name)
    m = wl.model
    B = wl.views
    enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=B)
    if row_groups > 1:
        incvit._check(incvit.incvit_set_tuning(enc.h, row_groups=row_groups), enc.h)
    fr = [torch.from_numpy(f).cuda() for f in wl.patch_frames(4)]
    bufa, ca = enc.new_caches(B)
    bufb, cb = enc.new_caches(B)
    enc.full_encode(fr[0], ca)
    enc.full_encode(fr[0], cb)
    inp = torch.empty_like(fr[0])
    out_g = (torch.empty((B, m.n_tokens), dtype=torch.int32, device="cuda"),
             torch.empty((B,), dtype=torch.int32, device="cuda"),
             torch.empty((B, m.n_tokens, m.dim), dtype=enc.dtype, device="cuda"))
    g = enc.step_graph(inp, ca, wl.tau, wl.caps, out_g)
    try:
        for t in range(1, 4):
            inp.copy_(fr[t])
            enc.launch(g)
            idx, count, refreshed = enc.step(fr[t], cb, wl.tau, wl.caps)
            torch.cuda.synchronize()
            say(f"[{name} graph] frame {t}: count={count.tolist()}")
            assert torch.equal(out_g[1], count)
            for v in range(B):
                k = int(count[v])
                assert torch.equal(out_g[0][v, :k], idx[v, :k])
                assert torch.equal(out_g[2][v, :k], refreshed[v, :k])
            for x, y in zip(_raw(enc, ca), _raw(enc, cb)):
                assert torch.equal(x, y)
    finally:
        enc.drop_graph(g)
        enc.close()


@pytest.mark.parametrize("score,mlp_mode", [("embed", "reuse"), ("key", "all")])
def test_full_graph_matches_eager(score, mlp_mode):
    m, w, enc, fr = _setup(B=1, score=score, mlp_mode=mlp_mode)
    bufa, ca = enc.new_caches(1)
    bufb, cb = enc.new_caches(1)
    inp = fr[1].clone()
    g = enc.full_graph(inp, ca)
    try:
        for _ in range(3):
            enc.launch(g)
            enc.full_encode(fr[1], cb)
            torch.cuda.synchronize()
            assert torch.equal(_raw(enc, ca)[0], _raw(enc, cb)[0])
    finally:
        enc.drop_graph(g)


def test_runs_are_bitwise_deterministic():
    m, w, enc, fr = _setup()
    outs = []
    for rep in range(2):
        buf, c = enc.new_caches(2)
        enc.full_encode(fr[0], c)
        res = []
        for t in (1, 2):
            idx, count, _ = enc.step(fr[t], c, 0.98, [m.n_tokens, 12])
            torch.cuda.synchronize()
            res.append([idx[v, :int(count[v])].clone() for v in range(2)])  # only count[v] are defined
        outs.append((_raw(enc, c), res))
    for x, y in zip(outs[0][0], outs[1][0]):
        assert torch.equal(x, y)
    for r0, r1 in zip(outs[0][1], outs[1][1]):
        for a, b in zip(r0, r1):
            assert torch.equal(a, b)


def test_identical_frame_and_zero_cap_write_nothing():
    m, w, enc, fr = _setup()
    buf, c = enc.new_caches(2)
    enc.full_encode(fr[0], c)
    before = _raw(enc, c)
    idx, count, _ = enc.step(fr[0], c, 0.98, [m.n_tokens, m.n_tokens])
    torch.cuda.synchronize()
    assert count.tolist() == [0, 0]
    for x, y in zip(before, _raw(enc, c)):
        assert torch.equal(x, y)
    idx, count, _ = enc.step(fr[1], c, 0.98, [0, 0])
    torch.cuda.synchronize()
    assert count.tolist() == [0, 0]
    for x, y in zip(before, _raw(enc, c)):
        assert torch.equal(x, y)


def test_only_selected_rows_change_on_gpu():
    m, w, enc, fr = _setup()
    buf, c = enc.new_caches(2)
    enc.full_encode(fr[0], c)
    before = [enc.export(x) for x in c]
    idx, count, _ = enc.step(fr[1], c, 0.98, [m.n_tokens, 7])
    torch.cuda.synchronize()
    after = [enc.export(x) for x in c]
    for v in range(2):
        U = set(idx[v, :int(count[v])].tolist())
        assert 0 < len(U) < m.n_tokens
        R = np.array(sorted(set(range(m.n_tokens)) - U))
        for name in ("ref", "Y"):
            assert np.array_equal(before[v][name][R], after[v][name][R])
        for name in ("X", "K", "V"):
            for l in range(after[v][name].shape[0]):
                assert np.array_equal(before[v][name][l][R], after[v][name][l][R]), (name, l)
                changed = set(np.nonzero(np.any(before[v][name][l] != after[v][name][l], axis=1))[0].tolist())
                assert changed <= U


def test_export_import_resume_is_bitwise():
    m, w, enc, fr = _setup()
    bufa, ca = enc.new_caches(2)
    bufb, cb = enc.new_caches(2)
    enc.full_encode(fr[0], ca)
    enc.step(fr[1], ca, 0.98, [m.n_tokens] * 2)
    snaps = _raw(enc, ca)
    for v in range(2):
        enc.import_raw(snaps[v], cb[v])
    assert enc.status(cb[0]) == incvit.INCVIT_OK
    ra = enc.step(fr[2], ca, 0.98, [m.n_tokens] * 2)
    rb = enc.step(fr[2], cb, 0.98, [m.n_tokens] * 2)
    torch.cuda.synchronize()
    assert torch.equal(ra[1], rb[1])
    for v in range(2):
        k = int(ra[1][v])
        assert torch.equal(ra[0][v, :k], rb[0][v, :k])
    for x, y in zip(_raw(enc, ca), _raw(enc, cb)):
        assert torch.equal(x, y)


def test_batched_call_equals_single_stream_calls():
    m, w, enc, fr = _setup(B=3)
    caps = [m.n_tokens, 5, 11]
    buf, cbat = enc.new_caches(3)
    enc.full_encode(fr[0], cbat)
    singles = []
    for v in range(3):
        b, c = enc.new_caches(1)
        enc.full_encode(fr[0][v:v + 1].contiguous(), c)
        singles.append((b, c))
    for t in (1, 2):
        idx, count, _ = enc.step(fr[t], cbat, 0.98, caps)
        for v in range(3):
            i1, c1, _ = enc.step(fr[t][v:v + 1].contiguous(), singles[v][1], 0.98, [caps[v]])
            torch.cuda.synchronize()
            assert int(c1[0]) == int(count[v])
            assert torch.equal(i1[0, :int(c1[0])], idx[v, :int(count[v])])
    tol = TOL[m.dtype]
    for v in range(3):
        a = enc.export(cbat[v])
        b = enc.export(singles[v][1][0])
        assert np.array_equal(a["ref"], b["ref"])
        for name in ("X", "K", "V", "Y"):
            assert rel_err(a[name], b[name]) <= tol, name


def test_full_refresh_step_matches_full_encode():
    m, w, enc, fr = _setup()
    bufa, ca = enc.new_caches(2)
    bufb, cb = enc.new_caches(2)
    enc.full_encode(fr[0], ca)
    idx, count, _ = enc.step(fr[1], ca, math.inf, [m.n_tokens] * 2)
    enc.full_encode(fr[1], cb)
    torch.cuda.synchronize()
    assert count.tolist() == [m.n_tokens] * 2
    for v in range(2):
        assert idx[v].tolist() == list(range(m.n_tokens))
        a, b = enc.export(ca[v]), enc.export(cb[v])
        assert np.array_equal(a["ref"], b["ref"])
        for name in ("X", "K", "V", "Y"):
            assert rel_err(a[name], b[name]) <= TOL[m.dtype], name


def test_448_full_refresh_equals_full_encode_on_every_frame():
    """The 448x448 stream at rho = 100% (top-k of all 1024 tokens): every step
    equals a full encode of the same frame bit for bit -- same rows, same row
    order, same kernels -- on each of four frames."""
    wl = synth.workload("so400m_448", rho=1.0)
    m = wl.model
    enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=1)
    fr = [torch.from_numpy(f).cuda() for f in wl.patch_frames(5)]
    bufa, ca = enc.new_caches(1)
    bufb, cb = enc.new_caches(1)
    enc.full_encode(fr[0], ca)
    for t in range(1, 5):
        idx, count, refreshed = enc.step(fr[t], ca, wl.tau, wl.caps)
        enc.full_encode(fr[t], cb)
        torch.cuda.synchronize()
        say(f"[448 rho 100%] frame {t}: count={count.tolist()}")
        assert count.tolist() == [m.n_tokens]
        assert idx[0].tolist() == list(range(m.n_tokens))
        assert torch.equal(_raw(enc, ca)[0], _raw(enc, cb)[0])
    enc.close()


def test_uninitialised_cache_and_nan_frame_are_no_ops():
    m, w, enc, fr = _setup()
    buf, c = enc.new_caches(2)           # zero-filled: never encoded
    assert enc.status(c[0]) == incvit.INCVIT_ERR_STATE
    idx, count, _ = enc.step(fr[1], c, 0.98, [m.n_tokens] * 2)
    torch.cuda.synchronize()
    assert count.tolist() == [0, 0]
    enc.full_encode(fr[0], c)
    assert enc.status(c[1]) == incvit.INCVIT_OK
    bad = fr[1].clone()
    bad[1, 3, 0] = float("nan")
    before = _raw(enc, c)
    idx, count, _ = enc.step(bad, c, 0.98, [m.n_tokens] * 2)
    torch.cuda.synchronize()
    assert int(count[1]) == 0 and int(count[0]) > 0
    assert enc.status(c[1]) == incvit.INCVIT_ERR_ARG
    assert enc.status(c[0]) == incvit.INCVIT_OK
    after = _raw(enc, c)                 # the export holds the data, not the header
    assert torch.equal(before[1], after[1])
    enc.full_encode(fr[1], c)           # a full encode re-arms the cache
    assert enc.status(c[1]) == incvit.INCVIT_OK


def test_argument_errors_are_reported_before_launch():
    m, w, enc, fr = _setup()
    buf, c = enc.new_caches(2)
    ws = enc.workspace(2).data_ptr()
    L = incvit
    assert L.incvit_step(enc.h, 3, fr[0].data_ptr(), c + [c[0]], 0.98, [1, 1, 1], 0, 0, 0, ws) == L.INCVIT_ERR_ARG
    assert L.incvit_step(enc.h, 2, fr[0].data_ptr(), c, float("nan"), [1, 1], fr[0].data_ptr(),
                         fr[0].data_ptr(), 0, ws) == L.INCVIT_ERR_ARG
    assert "NaN" in L.incvit_last_error(enc.h)
    assert L.incvit_full_encode(enc.h, 2, fr[0].data_ptr(), [c[0], 0], ws) == L.INCVIT_ERR_ARG
    assert L.incvit_full_encode(enc.h, 2, fr[0].data_ptr(), [c[0] + 8, c[1]], ws) == L.INCVIT_ERR_ARG
    assert L.incvit_set_tuning(enc.h, [3, 0, 0, 0]) == L.INCVIT_ERR_ARG
    assert L.incvit_set_tuning(enc.h, [0, 0, -1, 0]) == L.INCVIT_ERR_ARG
    assert L.incvit_set_tuning(enc.h, [0, 0, 0, 5]) == L.INCVIT_ERR_ARG
    assert L.incvit_set_tuning(enc.h, [1, 2, 0, 2]) == L.INCVIT_OK
    assert L.incvit_set_tuning(enc.h, [4, 4, 4, 4]) == L.INCVIT_OK
    assert L.incvit_set_tuning(enc.h, attn_waves=3) == L.INCVIT_ERR_ARG
    assert L.incvit_set_tuning(enc.h, None) == L.INCVIT_OK
