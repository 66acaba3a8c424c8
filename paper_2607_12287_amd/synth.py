"""Seeded synthetic inputs: model shapes, weights and camera-frame streams.

This module produces *inputs only*.  It holds none of the incremental-encoding
arithmetic (no embedding, similarity, selection, normalisation or attention);
both the HIP path and the CPU oracle consume what it returns.

The model is a pre-LN ViT of the kind the paper's vision encoder is (§III-A:
a SigLIP/ViT that turns the image into spatial tokens).  The paper gives no
shapes for it; the shapes below are the SigLIP-So400m, ViT-L and a tiny ViT,
and the streams imitate the 224x224 camera observations of §IV-A (LIBERO /
RoboTwin) and the three-camera robot of §IV-A, none of which are available
here.

Randomness: every array is drawn from ``np.random.default_rng([seed, *tags])``
with integer tags, so any array can be regenerated on its own and the order of
generation never matters.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Iterator, List, Optional, Sequence

import numpy as np

# ----------------------------------------------------------------------------
# Model shapes
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Shape of a pre-LN ViT encoder with learned positions and no CLS token."""

    img_h: int
    img_w: int
    channels: int
    patch: int
    dim: int
    depth: int
    heads: int
    mlp_dim: int
    dtype: str  # "f32" or "bf16": storage of weights, caches and activations
    ln_eps: float = 1e-6

    @property
    def grid_h(self) -> int:
        return self.img_h // self.patch

    @property
    def grid_w(self) -> int:
        return self.img_w // self.patch

    @property
    def n_tokens(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def patch_dim(self) -> int:
        return self.channels * self.patch * self.patch

    @property
    def head_dim(self) -> int:
        return self.dim // self.heads


TINY = ModelShape(224, 224, 3, 16, 192, 12, 3, 768, "f32")
SO400M = ModelShape(224, 224, 3, 14, 1152, 27, 16, 4304, "bf16")
SO400M_448 = ModelShape(448, 448, 3, 14, 1152, 27, 16, 4304, "bf16")
VIT_L = ModelShape(224, 224, 3, 14, 1024, 24, 16, 4096, "bf16")


# ----------------------------------------------------------------------------
# Weights, canonical layout
# ----------------------------------------------------------------------------

LAYER_PARAMS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def param_shapes(m: ModelShape) -> List[tuple]:
    """Canonical parameter list: (name, shape) in storage order.

    Matrices are stored [in][out] (y = x @ W).  W_pe rows are indexed by the
    patch feature (c*p + dy)*p + dx.  W_qkv columns [0,D) are Q, [D,2D) K,
    [2D,3D) V; head j owns columns [j*dh, (j+1)*dh) of each block.
    """
    D, F, P, N = m.dim, m.mlp_dim, m.patch_dim, m.n_tokens
    out = [("w_pe", (P, D)), ("b_pe", (D,)), ("pos", (N, D))]
    per = {"ln1_g": (D,), "ln1_b": (D,), "w_qkv": (D, 3 * D), "b_qkv": (3 * D,),
           "w_o": (D, D), "b_o": (D,), "ln2_g": (D,), "ln2_b": (D,),
           "w_1": (D, F), "b_1": (F,), "w_2": (F, D), "b_2": (D,)}
    for l in range(m.depth):
        for name in LAYER_PARAMS:
            out.append((f"l{l}.{name}", per[name]))
    out += [("lnf_g", (D,)), ("lnf_b", (D,))]
    return out


def _round_to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round fp32 draws to the nearest bf16 value (ties to even); fp32 result.

    This is input preparation: the weights of a bf16 model are bf16 numbers.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def make_weights(m: ModelShape, seed: int, *, scale: float = 0.02,
                 overrides: Optional[Dict[str, np.ndarray]] = None,
                 names: Optional[Sequence[str]] = None) -> Dict[str, np.ndarray]:
    """Seeded weights: matrices, biases and Pos ~ scale*N(0,1); LN gamma 1+scale*N(0,1),
    LN beta scale*N(0,1).  Drawn in fp32 and stored at the model's precision
    (fp32 arrays whose values are bf16 numbers for a bf16 model).  `names`
    restricts the draw to those parameters (the others are not generated)."""
    out: Dict[str, np.ndarray] = {}
    for pid, (name, shape) in enumerate(param_shapes(m)):
        if names is not None and name not in names:
            continue
        rng = np.random.default_rng([seed, 7, pid])
        a = rng.standard_normal(shape, dtype=np.float32) * np.float32(scale)
        if name.endswith("_g"):
            a = a + np.float32(1.0)
        a = a.astype(np.float32)
        if overrides and name in overrides:
            a = np.asarray(overrides[name], dtype=np.float32).reshape(shape)
        if m.dtype == "bf16":
            a = _round_to_bf16_values(a)
        out[name] = a
    return out


def flatten_weights(m: ModelShape, w: Dict[str, np.ndarray]) -> np.ndarray:
    """Concatenate the weights in canonical order into one fp32 vector."""
    return np.concatenate([w[name].reshape(-1) for name, _ in param_shapes(m)]).astype(np.float32)


def canonical_weight_count(m: ModelShape) -> int:
    return int(sum(int(np.prod(s)) for _, s in param_shapes(m)))


# ----------------------------------------------------------------------------
# Frames
# ----------------------------------------------------------------------------


def smooth_noise(rng: np.random.Generator, c: int, h: int, w: int, cell: int = 8) -> np.ndarray:
    """U[0,1) lattice values every `cell` pixels, bilinearly interpolated.

    The lattice has sub-patch structure, so two independent patches are far
    apart in cosine (well below 0.98), unlike near-constant patches.
    """
    gh, gw = -(-h // cell) + 1, -(-w // cell) + 1
    lat = rng.random((c, gh, gw), dtype=np.float32)
    y = np.arange(h, dtype=np.float32) / cell
    x = np.arange(w, dtype=np.float32) / cell
    y0 = np.floor(y).astype(np.int64)
    x0 = np.floor(x).astype(np.int64)
    fy = (y - y0)[None, :, None]
    fx = (x - x0)[None, None, :]
    a = lat[:, y0][:, :, x0]
    b = lat[:, y0][:, :, x0 + 1]
    cc = lat[:, y0 + 1][:, :, x0]
    d = lat[:, y0 + 1][:, :, x0 + 1]
    top = a * (1 - fx) + b * fx
    bot = cc * (1 - fx) + d * fx
    return (top * (1 - fy) + bot * fy).astype(np.float32)


def add_pixel_noise(rng: np.random.Generator, clean: np.ndarray, sigma: float = 0.005) -> np.ndarray:
    """Fresh, non-cumulative sensor noise, clipped to [0, 1]."""
    return np.clip(clean + rng.normal(0.0, sigma, clean.shape).astype(np.float32), 0.0, 1.0).astype(np.float32)


def patchify(frame: np.ndarray, p: int) -> np.ndarray:
    """(C,H,W) -> [N][C*p*p]; tokens row-major over the patch grid, features (c, dy, dx)."""
    c, h, w = frame.shape
    gh, gw = h // p, w // p
    return np.ascontiguousarray(
        frame.reshape(c, gh, p, gw, p).transpose(1, 3, 0, 2, 4).reshape(gh * gw, c * p * p),
        dtype=np.float32)


def _reflect(pos: int, lo: int, hi: int, vel: int):
    """Advance a coordinate by vel inside [lo, hi], reflecting at the ends."""
    if hi <= lo:
        return lo, vel
    nxt = pos + vel
    if nxt > hi:
        nxt, vel = 2 * hi - nxt, -vel
    if nxt < lo:
        nxt, vel = 2 * lo - nxt, -vel
    return nxt, vel


class Stream:
    """A single camera stream: yields float32 frames (C,H,W) in [0,1]."""

    def frames(self, count: int) -> Iterator[np.ndarray]:  # pragma: no cover
        raise NotImplementedError


class RefillRectStream(Stream):
    """Each frame one h x w rectangle at a seeded position is refilled with fresh
    smooth noise; the change persists.  `align` snaps positions to the patch grid."""

    def __init__(self, m: ModelShape, seed: int, view: int, rect_h: int, rect_w: int,
                 align: bool = False):
        self.m, self.seed, self.view = m, seed, view
        self.rect_h, self.rect_w, self.align = rect_h, rect_w, align

    def frames(self, count: int) -> Iterator[np.ndarray]:
        m = self.m
        clean = smooth_noise(np.random.default_rng([self.seed, 11, self.view]),
                             m.channels, m.img_h, m.img_w)
        for t in range(count):
            if t > 0:
                rng = np.random.default_rng([self.seed, 12, self.view, t])
                if self.align:
                    p = m.patch
                    y = int(rng.integers(0, m.img_h // p - self.rect_h // p + 1)) * p
                    x = int(rng.integers(0, m.img_w // p - self.rect_w // p + 1)) * p
                else:
                    y = int(rng.integers(0, m.img_h - self.rect_h + 1))
                    x = int(rng.integers(0, m.img_w - self.rect_w + 1))
                clean = clean.copy()
                clean[:, y:y + self.rect_h, x:x + self.rect_w] = smooth_noise(
                    rng, m.channels, self.rect_h, self.rect_w)
            yield add_pixel_noise(np.random.default_rng([self.seed, 13, self.view, t]), clean)


class MovingRectStream(Stream):
    """A textured square moving horizontally at `speed` px/frame over a static
    background, reflecting at the borders.  With `refill` its texture is fresh
    smooth noise every frame (a "moving blob"); otherwise the texture is fixed.
    `flicker` single patches per frame are refilled with fresh noise (they
    revert next frame)."""

    def __init__(self, m: ModelShape, seed: int, view: int, side: int, speed: int = 4,
                 refill: bool = False, flicker: int = 0, tex_cell: int = 8):
        self.m, self.seed, self.view = m, seed, view
        self.side = min(side, m.img_h, m.img_w)
        self.speed, self.refill, self.flicker = speed, refill, flicker
        self.tex_cell = tex_cell

    def frames(self, count: int) -> Iterator[np.ndarray]:
        m, s = self.m, self.side
        bg = smooth_noise(np.random.default_rng([self.seed, 21, self.view]),
                          m.channels, m.img_h, m.img_w)
        tex = smooth_noise(np.random.default_rng([self.seed, 22, self.view]), m.channels, s, s,
                           cell=self.tex_cell)
        r0 = np.random.default_rng([self.seed, 23, self.view])
        y = int(r0.integers(0, m.img_h - s + 1))
        x = int(r0.integers(0, m.img_w - s + 1))
        vel = self.speed if r0.random() < 0.5 else -self.speed
        for t in range(count):
            if t > 0:
                x, vel = _reflect(x, 0, m.img_w - s, vel)
            clean = bg.copy()
            if self.refill:
                tex = smooth_noise(np.random.default_rng([self.seed, 24, self.view, t]), m.channels, s, s,
                                   cell=self.tex_cell)
            clean[:, y:y + s, x:x + s] = tex
            if self.flicker:
                rng = np.random.default_rng([self.seed, 25, self.view, t])
                p = m.patch
                cells = rng.choice(m.n_tokens, size=self.flicker, replace=False)
                for cell in cells:
                    gy, gx = divmod(int(cell), m.grid_w)
                    clean[:, gy * p:(gy + 1) * p, gx * p:(gx + 1) * p] = smooth_noise(rng, m.channels, p, p)
            yield add_pixel_noise(np.random.default_rng([self.seed, 26, self.view, t]), clean)


# ----------------------------------------------------------------------------
# The five workloads
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class Workload:
    name: str
    model: ModelShape
    views: int
    tau: float                 # +inf disables the threshold (pure top-k)
    caps: List[int]            # per view, clamped to N
    frames: int
    weight_seed: int
    scene_seed: int
    streams: List[Stream]
    rho: Optional[float] = None

    def patch_frames(self, count: Optional[int] = None) -> Iterator[np.ndarray]:
        """Yield [views][N][P] float32 patch batches, one per frame."""
        n = self.frames if count is None else count
        its = [s.frames(n) for s in self.streams]
        for _ in range(n):
            yield np.stack([patchify(next(it), self.model.patch) for it in its])

    def weights(self) -> Dict[str, np.ndarray]:
        return make_weights(self.model, self.weight_seed)


def _cap_top_k(rho: float, n: int) -> int:
    return int(math.floor(rho * n + 0.5))


def workload(name: str, rho: float = 0.10) -> Workload:
    """The five configurations: 'tiny', 'so400m', 'so400m_x3', 'so400m_448', 'vitl_x8'."""
    if name == "tiny":
        m = TINY
        return Workload(name, m, 1, 0.98, [20], 9, 1001, 2001,
                        [RefillRectStream(m, 2001, 0, 48, 48)])
    if name == "so400m":
        m = SO400M
        return Workload(name, m, 1, 0.98, [m.n_tokens], 64, 1002, 2002,
                        [MovingRectStream(m, 2002, 0, 56, tex_cell=4)])
    if name == "so400m_x3":
        m = SO400M
        p = m.patch
        rects = [(3 * p, 4 * p), (5 * p, 5 * p), (8 * p, 8 * p)]
        return Workload(name, m, 3, 0.98, [m.n_tokens] * 3, 128, 1003, 2003,
                        [RefillRectStream(m, 2003, v, h, w, align=True) for v, (h, w) in enumerate(rects)])
    if name == "so400m_448":
        m = SO400M_448
        n = m.n_tokens
        side = m.patch * math.ceil(math.sqrt(1.25 * rho * n))
        return Workload(name, m, 1, float("inf"), [_cap_top_k(rho, n)], 32, 1004, 2004,
                        [MovingRectStream(m, 2004, 0, side, refill=True)], rho=rho)
    if name == "vitl_x8":
        m = VIT_L
        return Workload(name, m, 8, 0.98, [m.n_tokens] * 8, 256, 1005, 2005,
                        [MovingRectStream(m, 2005, v, 42, flicker=5) for v in range(8)])
    raise KeyError(name)


WORKLOADS = ("tiny", "so400m", "so400m_x3", "so400m_448", "vitl_x8")
RHO_SWEEP = (0.02, 0.05, 0.10, 0.25, 0.50, 1.00)


def small_model(dim: int = 64, depth: int = 2, heads: int = 2, mlp: int = 96, img: int = 32,
                patch: int = 8, channels: int = 3, dtype: str = "f32") -> ModelShape:
    """A small model for tests that must run in seconds on a CPU."""
    return ModelShape(img, img, channels, patch, dim, depth, heads, mlp, dtype)


def random_patches(m: ModelShape, seed: int, views: int = 1) -> np.ndarray:
    """[views][N][P] patches from independent smooth-noise frames."""
    out = []
    for v in range(views):
        rng = np.random.default_rng([seed, 31, v])
        out.append(patchify(add_pixel_noise(rng, smooth_noise(rng, m.channels, m.img_h, m.img_w)), m.patch))
    return np.stack(out)
