"""ctypes loader for the oracle's fixed-order fp32 routines (``pinned.c``).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pinned.c")
_LIB = os.path.join(_HERE, "_pinned.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile pinned.c with gcc (contraction off, so only the written fmaf fuse).
    ORACLE_PINNED_LIB names a prebuilt copy instead (the sanitizer build)."""
    if os.environ.get("ORACLE_PINNED_LIB"):
        return os.environ["ORACLE_PINNED_LIB"]
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O3", "-mavx2", "-mfma", "-ffp-contract=off", "-fno-fast-math",
                               "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            f = ctypes.POINTER(ctypes.c_float)
            i32 = ctypes.c_int32
            lib.oracle_embed_f32.argtypes = [f, f, f, f, i32, i32, i32, f]
            lib.oracle_embed_f32.restype = None
            lib.oracle_cosine_f32.argtypes = [f, f, i32, i32, f]
            lib.oracle_cosine_f32.restype = None
            lib.oracle_key_score_f32.argtypes = [f, f, f, f, f, i32, i32, ctypes.c_float, i32, f]
            lib.oracle_key_score_f32.restype = None
            _lib = lib
    return _lib


def _fp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def embed_f32(patches: np.ndarray, w_pe: np.ndarray, b_pe: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """T0 = patch embedding + Pos in the fixed fp32 fmaf order; [N][D] float32."""
    lib = _load()
    patches = np.ascontiguousarray(patches, dtype=np.float32)
    w_pe = np.ascontiguousarray(w_pe, dtype=np.float32)
    b_pe = np.ascontiguousarray(b_pe, dtype=np.float32)
    pos = np.ascontiguousarray(pos, dtype=np.float32)
    n, p = patches.shape
    d = w_pe.shape[1]
    assert w_pe.shape == (p, d) and b_pe.shape == (d,) and pos.shape == (n, d)
    out = np.empty((n, d), dtype=np.float32)
    lib.oracle_embed_f32(_fp(patches), _fp(w_pe), _fp(b_pe), _fp(pos), n, p, d, _fp(out))
    return out


def cosine_f32(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Row-wise cosine in the fixed fp32 order; [N] float32."""
    lib = _load()
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    assert a.shape == b.shape and a.ndim == 2
    out = np.empty((a.shape[0],), dtype=np.float32)
    lib.oracle_cosine_f32(_fp(a), _fp(b), a.shape[0], a.shape[1], _fp(out))
    return out


def key_score_f32(t0: np.ndarray, ln_g: np.ndarray, ln_b: np.ndarray, w_k: np.ndarray, b_k: np.ndarray,
                  eps: float, bf16: bool) -> np.ndarray:
    """First-layer keys of every token in the fixed fp32 order of pinned.c:
    LayerNorm 1 of layer 0 on S(t0), then the key projection; [N][D] float32."""
    lib = _load()
    t0 = np.ascontiguousarray(t0, dtype=np.float32)
    n, d = t0.shape
    assert d <= 4096
    ln_g = np.ascontiguousarray(ln_g, dtype=np.float32)
    ln_b = np.ascontiguousarray(ln_b, dtype=np.float32)
    w_k = np.ascontiguousarray(w_k, dtype=np.float32)
    b_k = np.ascontiguousarray(b_k, dtype=np.float32)
    assert ln_g.shape == (d,) and ln_b.shape == (d,) and w_k.shape == (d, d) and b_k.shape == (d,)
    out = np.empty((n, d), dtype=np.float32)
    lib.oracle_key_score_f32(_fp(t0), _fp(ln_g), _fp(ln_b), _fp(w_k), _fp(b_k), n, d, float(eps),
                             1 if bf16 else 0, _fp(out))
    return out
