"""Python binding of libincvit.so: the C ABI functions under the same names
(argument marshalling only) and a small wrapper, :class:`Encoder`, that uses
torch for device memory and streams.  Every step of the encoder runs in the
library's HIP kernels; there is no fallback: without the built library or a GPU
the calls raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# INCVIT_LIB may name another build of the same library (the tests' sanitizer
# build of the host code); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("INCVIT_LIB") or os.path.join(_HERE, "libincvit.so")

INCVIT_OK, INCVIT_ERR_ARG, INCVIT_ERR_SHAPE, INCVIT_ERR_UNSUPPORTED, INCVIT_ERR_STATE, INCVIT_ERR_HIP = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "INCVIT_OK", -1: "INCVIT_ERR_ARG", -2: "INCVIT_ERR_SHAPE", -3: "INCVIT_ERR_UNSUPPORTED",
                -4: "INCVIT_ERR_STATE", -5: "INCVIT_ERR_HIP"}
INCVIT_F32, INCVIT_BF16 = 0, 1
INCVIT_SCORE_EMBED, INCVIT_SCORE_KEY = 0, 1
SCORES = {"embed": INCVIT_SCORE_EMBED, "key": INCVIT_SCORE_KEY}
KERNEL_KINDS = ("embed", "sim", "select", "commit", "qkv", "attn", "oproj", "fc1", "fc2", "res_ln1",
                "key_ln", "key_proj", "hsum")
MLPS = {"reuse": 0, "all": 1}

# Exported symbols, as declared in include/incvit.h.
EXPORTS = ("incvit_canonical_weights_bytes", "incvit_packed_weights_bytes", "incvit_pack_weights",
           "incvit_create", "incvit_destroy", "incvit_cache_bytes", "incvit_cache_canonical_bytes",
           "incvit_workspace_bytes", "incvit_full_encode", "incvit_step", "incvit_cache_export",
           "incvit_cache_import", "incvit_cache_status", "incvit_last_error", "incvit_profile_enable",
           "incvit_profile_read", "incvit_step_graph_create", "incvit_full_graph_create",
           "incvit_graph_launch", "incvit_graph_destroy", "incvit_set_tuning", "incvit_encode_frame",
           "incvit_flow_two_anchor", "incvit_step_noalloc")
NOALLOC_SCRATCH_BYTES = 64 << 20


class incvit_config(ctypes.Structure):
    _fields_ = [("img_h", ctypes.c_int32), ("img_w", ctypes.c_int32), ("channels", ctypes.c_int32),
                ("patch", ctypes.c_int32), ("dim", ctypes.c_int32), ("depth", ctypes.c_int32),
                ("heads", ctypes.c_int32), ("mlp_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("max_streams", ctypes.c_int32), ("score", ctypes.c_int32),
                ("mlp_all", ctypes.c_int32)]


class incvit_tuning(ctypes.Structure):
    _fields_ = [("cols", ctypes.c_int32 * 4), ("attn_qtiles", ctypes.c_int32), ("row_groups", ctypes.c_int32),
                ("attn_waves", ctypes.c_int32), ("fc2_mode", ctypes.c_int32), ("tiled", ctypes.c_int32)]


class IncvitError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libincvit.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_12287_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, C, S, I32, F32 = ctypes.c_void_p, ctypes.POINTER(incvit_config), ctypes.c_size_t, ctypes.c_int32, ctypes.c_float
        sig = {
            "incvit_canonical_weights_bytes": (S, [C]),
            "incvit_packed_weights_bytes": (S, [C]),
            "incvit_pack_weights": (I32, [C, P, P, P]),
            "incvit_create": (I32, [C, P, ctypes.POINTER(P)]),
            "incvit_destroy": (None, [P]),
            "incvit_cache_bytes": (S, [P]),
            "incvit_cache_canonical_bytes": (S, [P]),
            "incvit_workspace_bytes": (S, [P, I32]),
            "incvit_full_encode": (I32, [P, I32, P, P, P, P]),
            "incvit_step": (I32, [P, I32, P, P, F32, P, P, P, P, P, P]),
            "incvit_cache_export": (I32, [P, P, P, P]),
            "incvit_cache_import": (I32, [P, P, P, P]),
            "incvit_cache_status": (I32, [P, P, P]),
            "incvit_last_error": (ctypes.c_char_p, [P]),
            "incvit_profile_enable": (I32, [P, I32]),
            "incvit_profile_read": (I32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), I32]),
            "incvit_step_graph_create": (I32, [P, I32, P, P, F32, P, P, P, P, P, ctypes.POINTER(P)]),
            "incvit_full_graph_create": (I32, [P, I32, P, P, P, ctypes.POINTER(P)]),
            "incvit_graph_launch": (I32, [P, P]),
            "incvit_graph_destroy": (None, [P]),
            "incvit_set_tuning": (I32, [P, ctypes.POINTER(incvit_tuning)]),
            "incvit_encode_frame": (I32, [P, I32, P, P, ctypes.c_int64, I32, F32, P, P, P, P, P, P]),
            "incvit_flow_two_anchor": (I32, [I32, ctypes.c_int64, P, P, P, P, P, P, P, P]),
            "incvit_step_noalloc": (I32, [P, I32, P, P, F32, P, P, P, P, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(status: int, handle=None):
    if status != INCVIT_OK:
        msg = lib().incvit_last_error(handle)
        raise IncvitError(status, msg.decode() if msg else "")


# --- C ABI, same names -------------------------------------------------------

def incvit_canonical_weights_bytes(cfg: incvit_config) -> int:
    return lib().incvit_canonical_weights_bytes(ctypes.byref(cfg))


def incvit_packed_weights_bytes(cfg: incvit_config) -> int:
    return lib().incvit_packed_weights_bytes(ctypes.byref(cfg))


def incvit_pack_weights(cfg, canonical: int, packed: int, stream: int = 0) -> int:
    return lib().incvit_pack_weights(ctypes.byref(cfg), canonical, packed, stream)


def incvit_create(cfg, packed: int):
    h = ctypes.c_void_p()
    st = lib().incvit_create(ctypes.byref(cfg), packed, ctypes.byref(h))
    return st, h


def incvit_destroy(h) -> None:
    lib().incvit_destroy(h)


def incvit_cache_bytes(h) -> int:
    return lib().incvit_cache_bytes(h)


def incvit_cache_canonical_bytes(h) -> int:
    return lib().incvit_cache_canonical_bytes(h)


def incvit_workspace_bytes(h, B: int) -> int:
    return lib().incvit_workspace_bytes(h, B)


def _ptr_array(ptrs: Sequence[int]):
    arr = (ctypes.c_void_p * len(ptrs))(*ptrs)
    return arr


def incvit_full_encode(h, B: int, patches: int, caches: Sequence[int], workspace: int, stream: int = 0) -> int:
    return lib().incvit_full_encode(h, B, patches, _ptr_array(caches), workspace, stream)


def incvit_step(h, B: int, patches: int, caches: Sequence[int], tau: float, cap: Sequence[int], idx: int,
                count: int, refreshed: int, workspace: int, stream: int = 0) -> int:
    caps = (ctypes.c_int32 * B)(*[int(c) for c in cap])
    return lib().incvit_step(h, B, patches, _ptr_array(caches), float(tau), caps, idx, count,
                             refreshed, workspace, stream)


def incvit_step_noalloc(h, B: int, patches: int, caches: Sequence[int], tau: float, cap: Sequence[int], idx: int,
                        count: int, refreshed: int, stream: int = 0) -> int:
    caps = (ctypes.c_int32 * B)(*[int(c) for c in cap])
    return lib().incvit_step_noalloc(h, B, patches, _ptr_array(caches), float(tau), caps, idx, count, refreshed,
                                     stream)


def incvit_encode_frame(h, B: int, patches: int, caches: Sequence[int], frame_index: int, period: int, tau: float,
                        cap: Sequence[int], idx: int, count: int, refreshed: int, workspace: int,
                        stream: int = 0) -> int:
    caps = (ctypes.c_int32 * B)(*[int(c) for c in cap])
    return lib().incvit_encode_frame(h, B, patches, _ptr_array(caches), int(frame_index), int(period), float(tau),
                                     caps, idx, count, refreshed, workspace, stream)


def incvit_flow_two_anchor(S: int, n: int, x0: int, v0: int, v7: int, alpha: int, beta: int, b: int, xT: int,
                           stream: int = 0) -> int:
    return lib().incvit_flow_two_anchor(int(S), int(n), x0, v0, v7, alpha, beta, b, xT, stream)


def flow_two_anchor(x0, v0, v7, alpha, beta, b, out=None):
    """x_T = x_0 + alpha v_0 + beta v_7 + b per sample on device fp32 tensors
    ([S][...] and [S]); returns out (a new tensor unless given)."""
    import torch
    S = x0.shape[0]
    n = x0.numel() // S
    for t in (x0, v0, v7, b):
        assert t.is_cuda and t.dtype == torch.float32 and t.is_contiguous() and t.numel() == S * n
    assert alpha.numel() == S and beta.numel() == S and alpha.is_contiguous() and beta.is_contiguous()
    if out is None:
        out = torch.empty_like(x0)
    _check(incvit_flow_two_anchor(S, n, x0.data_ptr(), v0.data_ptr(), v7.data_ptr(), alpha.data_ptr(),
                                  beta.data_ptr(), b.data_ptr(), out.data_ptr(),
                                  torch.cuda.current_stream(x0.device).cuda_stream))
    return out


def incvit_cache_export(h, cache: int, dst: int, stream: int = 0) -> int:
    return lib().incvit_cache_export(h, cache, dst, stream)


def incvit_cache_import(h, src: int, cache: int, stream: int = 0) -> int:
    return lib().incvit_cache_import(h, src, cache, stream)


def incvit_cache_status(h, cache: int, stream: int = 0) -> int:
    return lib().incvit_cache_status(h, cache, stream)


def incvit_last_error(h=None) -> str:
    m = lib().incvit_last_error(h)
    return m.decode() if m else ""


def incvit_profile_enable(h, enable: bool) -> int:
    return lib().incvit_profile_enable(h, 1 if enable else 0)


def incvit_profile_read(h, reset: bool = True):
    ms = (ctypes.c_double * len(KERNEL_KINDS))()
    n = (ctypes.c_int64 * len(KERNEL_KINDS))()
    _check(lib().incvit_profile_read(h, ms, n, 1 if reset else 0), h)
    return {k: (ms[i], n[i]) for i, k in enumerate(KERNEL_KINDS)}


def incvit_step_graph_create(h, B: int, patches: int, caches: Sequence[int], tau: float, cap: Sequence[int],
                             idx: int, count: int, refreshed: int, workspace: int):
    caps = (ctypes.c_int32 * B)(*[int(c) for c in cap])
    g = ctypes.c_void_p()
    st = lib().incvit_step_graph_create(h, B, patches, _ptr_array(caches), float(tau), caps, idx, count,
                                        refreshed, workspace, ctypes.byref(g))
    return st, g


def incvit_full_graph_create(h, B: int, patches: int, caches: Sequence[int], workspace: int):
    g = ctypes.c_void_p()
    st = lib().incvit_full_graph_create(h, B, patches, _ptr_array(caches), workspace, ctypes.byref(g))
    return st, g


def incvit_graph_launch(g, stream: int = 0) -> int:
    return lib().incvit_graph_launch(g, stream)


def incvit_graph_destroy(g) -> None:
    lib().incvit_graph_destroy(g)


def incvit_set_tuning(h, cols: Optional[Sequence[int]] = None, attn_qtiles: int = 0, row_groups: int = 0,
                      attn_waves: int = 0, fc2_mode: int = 0, tiled: int = 0) -> int:
    if cols is None and not attn_qtiles and not row_groups and not attn_waves and not fc2_mode and not tiled:
        return lib().incvit_set_tuning(h, None)
    t = incvit_tuning((ctypes.c_int32 * 4)(*[int(k) for k in (cols or (0, 0, 0, 0))]), int(attn_qtiles),
                      int(row_groups), int(attn_waves), int(fc2_mode), int(tiled))
    return lib().incvit_set_tuning(h, ctypes.byref(t))


# --- convenience wrapper -------------------------------------------------------

def make_config(shape, max_streams: int = 1, score: str = "embed", mlp: str = "reuse") -> incvit_config:
    """Config from a model shape with attributes img_h, img_w, channels, patch,
    dim, depth, heads, mlp_dim, dtype ('f32'/'bf16'), ln_eps; score is 'embed'
    or 'key' (what the cosine compares); mlp is 'reuse' (exact) or 'all' (every
    row through the MLP each frame)."""
    return incvit_config(shape.img_h, shape.img_w, shape.channels, shape.patch, shape.dim, shape.depth,
                         shape.heads, shape.mlp_dim, INCVIT_BF16 if shape.dtype == "bf16" else INCVIT_F32,
                         float(shape.ln_eps), int(max_streams), SCORES[score], MLPS[mlp])


class Encoder:
    """Device-resident encoder: packed weights, per-stream caches, workspace."""

    def __init__(self, shape, canonical_weights, max_streams: int = 1, device: str = "cuda",
                 score: str = "embed", mlp: str = "reuse"):
        import torch
        self.torch = torch
        self.shape = shape
        self.score = score
        self.mlp = mlp
        self.device = torch.device(device)
        self.cfg = make_config(shape, max_streams, score, mlp)
        self.dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.N = shape.n_tokens
        self.D = shape.dim
        nbytes = incvit_canonical_weights_bytes(self.cfg)
        if nbytes == 0:
            raise IncvitError(INCVIT_ERR_SHAPE, incvit_last_error())
        w = canonical_weights
        if not isinstance(w, torch.Tensor):
            w = torch.from_numpy(np.ascontiguousarray(w, dtype=np.float32))
        canon = w.to(self.device).to(self.dtype).contiguous()
        if canon.numel() * canon.element_size() != nbytes:
            raise IncvitError(INCVIT_ERR_ARG, f"canonical weights hold {canon.numel()} values, expected {nbytes}")
        self.packed = torch.empty(incvit_packed_weights_bytes(self.cfg), dtype=torch.uint8, device=self.device)
        stream = self.stream_ptr()
        _check(incvit_pack_weights(self.cfg, canon.data_ptr(), self.packed.data_ptr(), stream))
        torch.cuda.current_stream(self.device).synchronize()
        del canon
        st, h = incvit_create(self.cfg, self.packed.data_ptr())
        _check(st)
        self.h = h
        self.cache_bytes = incvit_cache_bytes(h)
        self.cache_stride = (self.cache_bytes + 255) // 256 * 256
        self._ws: Dict[int, object] = {}

    def stream_ptr(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    def close(self):
        if getattr(self, "h", None):
            incvit_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def new_caches(self, B: int):
        """One device buffer holding B caches; returns (buffer, [B base pointers])."""
        buf = self.torch.zeros(B * self.cache_stride, dtype=self.torch.uint8, device=self.device)
        base = buf.data_ptr()
        return buf, [base + v * self.cache_stride for v in range(B)]

    def workspace(self, B: int):
        ws = self._ws.get(B)
        if ws is None:
            ws = self.torch.empty(max(256, incvit_workspace_bytes(self.h, B)), dtype=self.torch.uint8,
                                  device=self.device)
            self._ws[B] = ws
        return ws

    def full_encode(self, patches, caches: Sequence[int]):
        B = len(caches)
        assert patches.is_cuda and patches.dtype == self.torch.float32 and patches.is_contiguous()
        assert tuple(patches.shape) == (B, self.N, self.shape.patch_dim)
        _check(incvit_full_encode(self.h, B, patches.data_ptr(), caches, self.workspace(B).data_ptr(),
                                  self.stream_ptr()), self.h)

    def step(self, patches, caches: Sequence[int], tau: float, cap: Sequence[int], out=None):
        """Returns (idx [B][N] int32, count [B] int32, refreshed [B][N][D]) device tensors."""
        B = len(caches)
        torch = self.torch
        assert patches.is_cuda and patches.dtype == torch.float32 and patches.is_contiguous()
        assert tuple(patches.shape) == (B, self.N, self.shape.patch_dim)
        if out is None:
            out = (torch.empty((B, self.N), dtype=torch.int32, device=self.device),
                   torch.empty((B,), dtype=torch.int32, device=self.device),
                   torch.empty((B, self.N, self.D), dtype=self.dtype, device=self.device))
        idx, count, refreshed = out
        _check(incvit_step(self.h, B, patches.data_ptr(), caches, tau, cap, idx.data_ptr(), count.data_ptr(),
                           refreshed.data_ptr() if refreshed is not None else 0, self.workspace(B).data_ptr(),
                           self.stream_ptr()), self.h)
        return idx, count, refreshed

    def encode_frame(self, patches, caches: Sequence[int], frame_index: int, period: int, tau: float,
                     cap: Sequence[int], out=None):
        """One frame under a refresh period (full encode when frame_index % period
        == 0, else a step); returns (idx, count, refreshed) like step."""
        B = len(caches)
        torch = self.torch
        assert patches.is_cuda and patches.dtype == torch.float32 and patches.is_contiguous()
        assert tuple(patches.shape) == (B, self.N, self.shape.patch_dim)
        if out is None:
            out = (torch.empty((B, self.N), dtype=torch.int32, device=self.device),
                   torch.empty((B,), dtype=torch.int32, device=self.device),
                   torch.empty((B, self.N, self.D), dtype=self.dtype, device=self.device))
        idx, count, refreshed = out
        _check(incvit_encode_frame(self.h, B, patches.data_ptr(), caches, frame_index, period, tau, cap,
                                   idx.data_ptr(), count.data_ptr(),
                                   refreshed.data_ptr() if refreshed is not None else 0,
                                   self.workspace(B).data_ptr(), self.stream_ptr()), self.h)
        return idx, count, refreshed

    def step_graph(self, patches, caches: Sequence[int], tau: float, cap: Sequence[int], out):
        """Capture one step with fixed buffers; replay with launch(graph) after
        writing the next frame into `patches`.  Destroy with drop_graph."""
        idx, count, refreshed = out
        st, g = incvit_step_graph_create(self.h, len(caches), patches.data_ptr(), caches, tau, cap, idx.data_ptr(),
                                         count.data_ptr(), refreshed.data_ptr() if refreshed is not None else 0,
                                         self.workspace(len(caches)).data_ptr())
        _check(st, self.h)
        return g

    def full_graph(self, patches, caches: Sequence[int]):
        st, g = incvit_full_graph_create(self.h, len(caches), patches.data_ptr(), caches,
                                         self.workspace(len(caches)).data_ptr())
        _check(st, self.h)
        return g

    def launch(self, graph):
        _check(incvit_graph_launch(graph, self.stream_ptr()))

    @staticmethod
    def drop_graph(graph):
        incvit_graph_destroy(graph)

    def export(self, cache: int) -> Dict[str, np.ndarray]:
        """Canonical copy of one cache as float64 numpy arrays: ref, X, K, V, Y
        (and A with mlp 'all')."""
        torch = self.torch
        nb = incvit_cache_canonical_bytes(self.h)
        dst = torch.empty(nb, dtype=torch.uint8, device=self.device)
        _check(incvit_cache_export(self.h, cache, dst.data_ptr(), self.stream_ptr()), self.h)
        torch.cuda.current_stream(self.device).synchronize()
        s = self.shape
        N, D, L = s.n_tokens, s.dim, s.depth
        nd = N * D
        ref = dst[: nd * 4].view(torch.float32).reshape(N, D)
        rest = dst[nd * 4:].view(self.dtype).float()
        o = 0
        X = rest[o:o + (L + 1) * nd].reshape(L + 1, N, D); o += (L + 1) * nd
        K = rest[o:o + L * nd].reshape(L, N, D); o += L * nd
        V = rest[o:o + L * nd].reshape(L, N, D); o += L * nd
        Y = rest[o:o + nd].reshape(N, D); o += nd
        parts = [("ref", ref), ("X", X), ("K", K), ("V", V), ("Y", Y)]
        if self.mlp == "all":
            parts.append(("A", rest[o:o + L * nd].reshape(L, N, D)))
        return {k: t.cpu().numpy().astype(np.float64 if k != "ref" else np.float32) for k, t in parts}

    def export_raw(self, cache: int):
        nb = incvit_cache_canonical_bytes(self.h)
        dst = self.torch.empty(nb, dtype=self.torch.uint8, device=self.device)
        _check(incvit_cache_export(self.h, cache, dst.data_ptr(), self.stream_ptr()), self.h)
        return dst

    def import_raw(self, canonical, cache: int):
        _check(incvit_cache_import(self.h, canonical.data_ptr(), cache, self.stream_ptr()), self.h)

    def status(self, cache: int) -> int:
        return incvit_cache_status(self.h, cache, self.stream_ptr())
