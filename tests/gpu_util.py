"""Helpers for the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them.

Bars:
* token indices and counts bit-exact; the fp32 reference rows (`ref`, each
  token's score vector -- embedding or first-layer key -- at its last refresh)
  and the layer-0 rows bit-exact, since the embedding and the key score are
  computed in the same fixed fp32 order on both sides;
* per layer, teacher-forced: the oracle's layer applied to the GPU's own cached
  inputs of that layer gives the GPU's outputs (X^{l+1}, K^l, V^l, and Y)
  within max|gpu - oracle| / max|oracle| <= 2e-2 (bf16 storage) or 1e-4 (fp32);
* free-running (GPU from the first frame vs the oracle from the first frame):
  within FREE_TOL.  With bf16 storage, roundings that sit at a tie flip when
  accumulation is fp32 instead of fp64 and the flips compound through the
  residual stream; a CPU implementation that only swaps fp64 for fp32
  accumulation drifts by the same amount (tests/test_precision_drift.py).
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import vit
from paper_2607_12287_amd import incvit, synth

TOL = {"bf16": 2e-2, "f32": 1e-4}
GUARD_BYTE = 0xA5
FREE_TOL = {"bf16": 5e-2, "f32": 1e-4}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(a: np.ndarray, b: np.ndarray) -> float:
    den = float(np.abs(b).max())
    return float(np.abs(a - b).max()) / (den if den > 0 else 1.0)


class Pair:
    """The HIP encoder and the oracle on the same model and weights."""

    def __init__(self, m: synth.ModelShape, w, B: int, oracle_views=None, score: str = "embed",
                 mlp: str = "reuse", guard: int = 0):
        self.m, self.w, self.B = m, w, B
        self.enc = incvit.Encoder(m, synth.flatten_weights(m, w), max_streams=B, score=score, mlp=mlp)
        self.model = vit.Model(m, w, score=score, mlp=mlp)
        self.guard = guard
        if guard:
            self._guarded_buffers(B, guard)
        else:
            self.buf, self.caches = self.enc.new_caches(B)
        # each sampled stream once (the oracle steps every listed stream's cache)
        self.views = list(range(B)) if oracle_views is None else sorted(set(oracle_views))
        self.ora = {}

    def _guarded_buffers(self, B: int, guard: int):
        """Caches and workspace with `guard` bytes of a fixed pattern before the
        first cache, between consecutive caches and around the workspace; every
        byte the library may write lies inside its caches and workspace."""
        assert guard % 256 == 0
        enc = self.enc
        self.stride = enc.cache_stride + guard
        self.buf = torch.full((guard + B * self.stride,), GUARD_BYTE, dtype=torch.uint8, device="cuda")
        base = self.buf.data_ptr() + guard
        self.caches = [base + v * self.stride for v in range(B)]
        for v in range(B):
            o = guard + v * self.stride
            self.buf[o:o + enc.cache_bytes].zero_()
        n = incvit.incvit_workspace_bytes(enc.h, B)
        self.ws_n = n
        self.wsbuf = torch.full((guard + n + guard,), GUARD_BYTE, dtype=torch.uint8, device="cuda")
        enc._ws[B] = self.wsbuf[guard:guard + n]

    def check_guards(self, label=""):
        """Every guard byte still holds the pattern."""
        if not self.guard:
            return
        torch.cuda.synchronize()
        g, cb = self.guard, self.enc.cache_bytes
        buf = self.buf.cpu().numpy()
        spans = [(0, g)] + [(g + v * self.stride + cb, g + (v + 1) * self.stride) for v in range(self.B)]
        for a, b in spans:
            bad = np.nonzero(buf[a:b] != GUARD_BYTE)[0]
            assert bad.size == 0, (label, "cache guard", a, int(bad[0]))
        ws = self.wsbuf.cpu().numpy()
        for a, b in ((0, g), (g + self.ws_n, ws.size)):
            bad = np.nonzero(ws[a:b] != GUARD_BYTE)[0]
            assert bad.size == 0, (label, "workspace guard", a, int(bad[0]))

    def full_encode(self, batch: np.ndarray):
        self.enc.full_encode(torch.from_numpy(batch).cuda(), self.caches)
        torch.cuda.synchronize()
        self.ora = {v: vit.full_encode(self.model, batch[v]) for v in self.views}

    def step(self, batch: np.ndarray, tau: float, caps):
        idx, count, refreshed = self.enc.step(torch.from_numpy(batch).cuda(), self.caches, tau, caps)
        torch.cuda.synchronize()
        res = {v: vit.step(self.model, batch[v], self.ora[v], tau, caps[v]) for v in self.views}
        return idx.cpu().numpy(), count.cpu().numpy(), refreshed.float().cpu().numpy(), res

    def check_step(self, idx, count, refreshed, res, label="", free_y=True):
        """Indices and counts bit-exact, refreshed == Y[idx]; with free_y the
        refreshed rows also within the free-running bar of the oracle's."""
        tol = FREE_TOL[self.m.dtype]
        for v in self.views:
            r = res[v]
            assert int(count[v]) == r.count, (label, v, int(count[v]), r.count)
            assert np.array_equal(idx[v, :r.count], r.idx), (label, v)
            if r.count:
                g = self.enc.export(self.caches[v])
                assert np.array_equal(refreshed[v, :r.count], g["Y"][r.idx]), (label, v, "refreshed != Y[idx]")
                if free_y:
                    e = rel_err(refreshed[v, :r.count], r.refreshed)
                    assert e <= tol, (label, v, "refreshed", e)

    def check_layers(self, U_of=None, label=""):
        """Teacher-forced parity of every layer; U_of(v) = refreshed rows
        (None: all rows, after a full encode).  Returns the worst error."""
        m, tol, dt = self.m, TOL[self.m.dtype], self.m.dtype
        worst = 0.0
        for v in self.views:
            g = self.enc.export(self.caches[v])
            U = np.arange(m.n_tokens) if U_of is None else np.asarray(U_of(v))
            assert np.array_equal(g["ref"], self.ora[v].ref), (label, v, "ref")
            assert np.array_equal(g["X"][0][U], self.ora[v].X[0][U]), (label, v, "X0")
            if self.model.score == "embed":
                assert np.array_equal(g["X"][0][U], vit.S(g["ref"][U].astype(np.float64), dt)), (label, v, "X0")
            if self.model.mlp == "all":
                worst = max(worst, self._check_layers_all(g, v, U, label))
                continue
            if U.size == 0:
                continue
            for l in range(m.depth):
                K, V = g["K"][l].copy(), g["V"][l].copy()
                Z = vit.layer_rows(self.model, l, g["X"][l][U], U, K, V)
                for name, a, b in (("X", g["X"][l + 1][U], Z), ("K", g["K"][l][U], K[U]), ("V", g["V"][l][U], V[U])):
                    e = rel_err(a, b)
                    worst = max(worst, e)
                    assert e <= tol, (label, v, "layer", l, name, e)
            e = rel_err(g["Y"][U], vit.final_rows(self.model, g["X"][m.depth][U]))
            worst = max(worst, e)
            assert e <= tol, (label, v, "Y", e)
        return worst

    def _check_layers_all(self, g, v, U, label):
        """Teacher-forced parity of the all-rows MLP reading: every row of every
        layer from the GPU's own inputs and cached K, V and attention branch."""
        m, tol = self.m, TOL[self.m.dtype]
        assert np.array_equal(g["X"][0], self.ora[v].X[0]), (label, v, "X0 all rows")
        worst = 0.0
        for l in range(m.depth):
            K, V, A = g["K"][l].copy(), g["V"][l].copy(), g["A"][l].copy()
            Z = vit.layer_all(self.model, l, g["X"][l], U, K, V, A)
            pairs = [("X", g["X"][l + 1], Z)]
            if U.size:
                pairs += [("K", g["K"][l][U], K[U]), ("V", g["V"][l][U], V[U]), ("A", g["A"][l][U], A[U])]
            for name, a, b in pairs:
                e = rel_err(a, b)
                worst = max(worst, e)
                assert e <= tol, (label, v, "layer", l, name, e)
        e = rel_err(g["Y"], vit.final_rows(self.model, g["X"][m.depth]))
        assert e <= tol, (label, v, "Y", e)
        return max(worst, e)

    def check_caches(self, label="", tensors=("X", "K", "V", "A", "Y")):
        tol = FREE_TOL[self.m.dtype]
        worst = 0.0
        for v in self.views:
            g = self.enc.export(self.caches[v])
            o = self.ora[v]
            assert np.array_equal(g["ref"], o.ref), (label, v, "ref")
            names = [("X", self.m.depth + 1), ("K", self.m.depth), ("V", self.m.depth)]
            if self.model.mlp == "all":
                names.append(("A", self.m.depth))
            for name, depth in [nd for nd in names if nd[0] in tensors]:
                for l in range(depth):
                    e = rel_err(g[name][l], getattr(o, name)[l])
                    worst = max(worst, e)
                    assert e <= tol, (label, v, name, l, e)
            if "Y" in tensors:
                e = rel_err(g["Y"], o.Y)
                worst = max(worst, e)
                assert e <= tol, (label, v, "Y", e)
        return worst


def workspace_arrays(enc, B: int):
    """The per-token fp32 arrays of the last call, read from the library's
    workspace through a mirror of its layout (256-byte aligned parts: meta,
    row map, counts, idx, sim, T0, then in key mode the LayerNorm rows and the
    keys).  Tests check T0 against the oracle first, which validates the mirror."""
    N, D = enc.N, enc.D
    M = B * N
    mpad = (max(M, 1) + 63) // 64 * 64
    offs, off = {}, 0
    sizes = [("meta", 4 + 65 * 4), ("rows", mpad * 16), ("count", 64 * 4), ("idx", M * 4), ("sim", M * 4),
             ("t0", M * D * 4)]
    if enc.score == "key":
        sizes += [("kn", M * D * 4), ("key", M * D * 4)]
    for name, n in sizes:
        offs[name] = off
        off = (off + n + 255) // 256 * 256
    ws = enc.workspace(B)
    torch.cuda.synchronize()

    def f32(name, shape):
        o = offs[name]
        return ws[o:o + int(np.prod(shape)) * 4].view(torch.float32).reshape(shape).cpu().numpy()

    out = {"sim": f32("sim", (B, N)), "t0": f32("t0", (B, N, D))}
    if enc.score == "key":
        out["key"] = f32("key", (B, N, D))
    return out
