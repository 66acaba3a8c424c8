"""The allocation-free step (incvit_step_noalloc) against incvit_step, through
the C ABI: same frames on two copies of the same caches, results compared bit
for bit (same kernels, same order), on two calls in a row where the second is
smaller (three streams, then one).  (A call too large for the static scratch
is rejected on the host: tests/test_abi.py.)"""
import numpy as np
import pytest
import torch

from paper_2607_12287_amd import incvit, synth
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def _frames(m, B, count, seed):
    its = [synth.RefillRectStream(m, seed + v, v, 15, 19).frames(count) for v in range(B)]
    return [torch.from_numpy(np.stack([synth.patchify(next(it), m.patch) for it in its])).cuda()
            for _ in range(count)]


def _step_noalloc(enc, patches, caches, tau, caps):
    B = len(caches)
    idx = torch.full((B, enc.N), -7, dtype=torch.int32, device="cuda")
    count = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    refreshed = torch.zeros((B, enc.N, enc.D), dtype=enc.dtype, device="cuda")
    incvit._check(incvit.incvit_step_noalloc(enc.h, B, patches.data_ptr(), caches, tau, caps, idx.data_ptr(),
                                             count.data_ptr(), refreshed.data_ptr(), enc.stream_ptr()), enc.h)
    return idx, count, refreshed


def _same(enc, a, b, label):
    """count equal; idx[v][0..count) and refreshed rows 0..count equal (the
    entries past count are unspecified)."""
    assert torch.equal(a[1], b[1]), (label, "count")
    cnt = a[1].cpu().numpy()
    for v in range(len(cnt)):
        k = int(cnt[v])
        assert torch.equal(a[0][v, :k], b[0][v, :k]), (label, "idx", v)
        assert torch.equal(a[2][v, :k], b[2][v, :k]), (label, "refreshed", v)


@pytest.mark.parametrize("name", ["small_bf16", "so400m"])
def test_noalloc_step_equals_step(name):
    if name == "so400m":
        wl = synth.workload("so400m_x3")
        m, w, B = wl.model, wl.weights(), 3
        frames = [torch.from_numpy(f).cuda() for f in wl.patch_frames(3)]
        tau = wl.tau
    else:
        m = synth.small_model(dim=256, depth=2, heads=4, mlp=512, img=40, patch=4, dtype="bf16")
        w, B = synth.make_weights(m, 2401), 3
        frames = _frames(m, B, 3, 2410)
        tau = 0.98
    say(f"[noalloc {name}] N={m.n_tokens} D={m.dim} B={B}")
    enc = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=B)
    assert incvit.incvit_workspace_bytes(enc.h, B) <= incvit.NOALLOC_SCRATCH_BYTES
    buf_a, ca = enc.new_caches(B)
    buf_b, cb = enc.new_caches(B)
    enc.full_encode(frames[0], ca)
    enc.full_encode(frames[0], cb)
    torch.cuda.synchronize()
    assert torch.equal(buf_a, buf_b)
    # call 1: every stream; call 2: the first stream only (smaller input)
    for t, (views, caps) in enumerate([(list(range(B)), [m.n_tokens] * B), ([0], [m.n_tokens])], start=1):
        patches = frames[t][views].contiguous()
        ref = enc.step(patches, [ca[v] for v in views], tau, caps)
        got = _step_noalloc(enc, patches, [cb[v] for v in views], tau, caps)
        torch.cuda.synchronize()
        say(f"  call {t}: streams {views} count {got[1].tolist()}")
        assert int(got[1].sum()) > 0
        _same(enc, ref, got, f"call {t}")
        assert torch.equal(buf_a, buf_b), f"call {t}: caches differ"
    enc.close()


def test_noalloc_large_row_gemm():
    """The 448x448 frame (1024 tokens) top-k: 512 rows (the large-row GEMM,
    its down projection's partial sums in the static scratch), then 102 rows
    (the weight-streaming GEMM) -- both equal incvit_step bit for bit."""
    wl = synth.workload("so400m_448", rho=0.5)
    m = wl.model
    say(f"[noalloc 448] N={m.n_tokens} D={m.dim}")
    enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=1)
    assert incvit.incvit_workspace_bytes(enc.h, 1) <= incvit.NOALLOC_SCRATCH_BYTES
    frames = [torch.from_numpy(f).cuda() for f in wl.patch_frames(3)]
    buf_a, ca = enc.new_caches(1)
    buf_b, cb = enc.new_caches(1)
    enc.full_encode(frames[0], ca)
    enc.full_encode(frames[0], cb)
    torch.cuda.synchronize()
    for t, cap in enumerate([512, 102], start=1):
        ref = enc.step(frames[t], ca, wl.tau, [cap])
        got = _step_noalloc(enc, frames[t], cb, wl.tau, [cap])
        torch.cuda.synchronize()
        say(f"  call {t}: cap {cap} count {got[1].tolist()}")
        assert got[1].tolist() == [cap]
        _same(enc, ref, got, f"call {t}")
        assert torch.equal(buf_a, buf_b), f"call {t}: caches differ"
    enc.close()
