"""CPU oracle of incremental ViT encoding with temporal token reuse.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package; the product path
never does, and this package imports nothing from the product.

What it computes (paper §III-B, "Temporal Token Reuse"):

* every frame is patch-embedded and each token is scored by the cosine of its
  current and cached representation (eq. 3); the least similar tokens are the
  updated set U, the rest R reuse their cache (the top-rho*N rule, here a
  threshold tau followed by a cap);
* the index set is chosen once, before the first layer, and reused by every
  layer;
* in every layer, Q, K and V are recomputed only for the rows in U (eq. 4);
  the new K/V rows are scattered into the cached full K/V (eq. 5);
* attention is computed only for the updated queries, over all N keys;
  reused tokens keep their cached outputs; the updated rows then go through the
  residual add and the MLP.

The model is a pre-LN ViT (the paper's vision encoder is a SigLIP/ViT, §III-A):
no CLS token, learned positions added after the patch embedding, biased
linear layers, LayerNorm with biased variance, tanh-form GELU, softmax
attention scaled by 1/sqrt(d_h), and a final LayerNorm.  These details are not
in the paper; they are the readings taken here.

What the cosine compares (``Model.score``): "embed" scores the layer-1 input
token (patch embedding + position) against its value at the token's last
refresh; "key" scores the first layer's key projection of that token, which is
what eq. 3 compares (the current key of a token against its cached key).
Either way the vector is kept per token as the reference for later frames.

The paper's odd/even chunk schedule (a full forward on odd chunks whose keys
become the reference, incremental encoding on even chunks) is
``run_schedule`` with period 2; other periods generalise it.

How the MLP sentence of §III-B is read (``Model.mlp``; the paper says every
token goes through the MLP): "reuse" (default) reads it exactly: a reused
row's MLP input is its cached state, so its MLP output is its cached output
and only the rows U need computing.  "all" is the non-exact reading: every
frame, every row starts from this frame's embedded token, reused rows add
their cached attention-branch output (attention + output projection, per
layer) to their current residual stream, and the MLP runs over all rows, so
reused rows follow the new frame without their attention being recomputed
(their K and V stay cached).

Arithmetic: everything is float64 except the patch embedding, the key score
and the cosine, which follow a fixed fp32 order (``pinned.c``) so that the
selection is reproducible bit for bit.

Storage rounding, one reading applied everywhere: the paper runs its encoder
in half precision under PyTorch (Appendix A, hardware table), where every
operation reads stored tensors, computes internally at higher precision and
stores its result in the storage type.  ``S(.)`` (round to nearest, ties to
even, to bf16 or fp32; nothing in the "f64" mode of the pins) is therefore
applied to the output of every operation of the layer and nowhere else:

    A  = S(LN1(X))            Q|K|V = S(A W_qkv + b_qkv)
    O  = S(Attn(Q, K, V))     B     = S(O W_o + b_o)       H = S(X + B)
    A2 = S(LN2(H))            F     = S(A2 W_1 + b_1)      G = S(GELU(F))
    M  = S(G W_2 + b_2)       X'    = S(H + M)             Y = S(LN_f(X^L))

and X^0 = S(T^0).  A linear layer with its bias is one operation, as is the
attention.  The two MLP readings share this block exactly (the "all" reading
caches B per layer), so their full encodes are identical.  The test
``tests/test_oracle_rounding.py`` pins these points against PyTorch's own
bf16 modules.

Parity: pinned (see tests/test_oracle_*.py) by library routines (torch fp64
functional ops), closed forms, brute-force selection, and the invariants the
method fixes.  No intermediate value printed in the paper exists to pin against.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import pinned

# ----------------------------------------------------------------------------
# Elementary operations
# ----------------------------------------------------------------------------


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 number (8 significant bits),
    ties to even, directly from float64.  Normal range only."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)              # x = m * 2**e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def S(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the storage precision; returns float64."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis with the biased variance."""
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps) * g + b


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """GELU, tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """Multi-head softmax attention of the rows of q over all rows of k, v.

    q: [m][D], k, v: [N][D]; head j uses columns [j*dh, (j+1)*dh)."""
    m, d = q.shape
    dh = d // heads
    out = np.empty((m, d), dtype=np.float64)
    for j in range(heads):
        c = slice(j * dh, (j + 1) * dh)
        s = q[:, c] @ k[:, c].T / math.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        out[:, c] = (p @ v[:, c]) / p.sum(axis=1, keepdims=True)
    return out


# ----------------------------------------------------------------------------
# Token selection (eq. 3 and the top-rho*N rule)
# ----------------------------------------------------------------------------


def select(sim: np.ndarray, tau: float, cap: int) -> np.ndarray:
    """U = {i : sim_i < tau} (fp32 compare); if |U| > cap keep the cap lowest
    similarities, equal similarities going to the lower index.  Ascending."""
    sim = np.asarray(sim, dtype=np.float32)
    if np.isnan(sim).any():
        raise ValueError("non-finite similarity: the frame holds NaN or Inf")
    n = sim.shape[0]
    cap = max(0, min(int(cap), n))
    cand = np.nonzero(sim < np.float32(tau))[0]
    if cand.size > cap:
        order = np.lexsort((cand, sim[cand]))   # by sim, then by index
        cand = np.sort(cand[order[:cap]])
    return cand.astype(np.int32)


# ----------------------------------------------------------------------------
# Model and per-view cache
# ----------------------------------------------------------------------------


SCORES = ("embed", "key")
MLPS = ("reuse", "all")


class Model:
    """Weights of the encoder as float64 arrays (values as stored).

    score: "embed" (cosine of the embedded tokens) or "key" (cosine of the
    first layer's keys, eq. 3); mlp: "reuse" or "all" (see the module text)."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], dtype: Optional[str] = None,
                 score: str = "embed", mlp: str = "reuse"):
        if score not in SCORES:
            raise ValueError(f"score must be one of {SCORES}")
        if mlp not in MLPS:
            raise ValueError(f"mlp must be one of {MLPS}")
        self.shape = shape
        self.dtype = dtype or shape.dtype
        self.score = score
        self.mlp = mlp
        self.eps = float(shape.ln_eps)
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.w32 = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in
                    (("w_pe", weights["w_pe"]), ("b_pe", weights["b_pe"]), ("pos", weights["pos"]))}
        if score == "key":
            D = shape.dim
            self.w32.update({
                "ln1_g": np.ascontiguousarray(weights["l0.ln1_g"], dtype=np.float32),
                "ln1_b": np.ascontiguousarray(weights["l0.ln1_b"], dtype=np.float32),
                "w_k": np.ascontiguousarray(np.asarray(weights["l0.w_qkv"])[:, D:2 * D], dtype=np.float32),
                "b_k": np.ascontiguousarray(np.asarray(weights["l0.b_qkv"])[D:2 * D], dtype=np.float32)})

    def p(self, l: int, name: str) -> np.ndarray:
        return self.w[f"l{l}.{name}"]


@dataclasses.dataclass
class ViewCache:
    """Everything one stream keeps between frames, canonical layout.

    ref: [N][D] fp32, each token's score vector (embedding or first-layer
    key, per Model.score) at its last refresh: the reference the cosine is
    taken against;
    X: [L+1][N][D] layer inputs (X[0] = embedded tokens, X[l+1] = layer l out);
    K, V: [L][N][D] per-layer keys and values;  Y: [N][D] final output;
    A: [L][N][D] attention-branch outputs S(O W_o + b_o) per layer (mlp "all"
    only, else None)."""

    ref: np.ndarray
    X: np.ndarray
    K: np.ndarray
    V: np.ndarray
    Y: np.ndarray
    A: Optional[np.ndarray] = None

    def copy(self) -> "ViewCache":
        return ViewCache(self.ref.copy(), self.X.copy(), self.K.copy(), self.V.copy(), self.Y.copy(),
                         None if self.A is None else self.A.copy())


@dataclasses.dataclass
class StepResult:
    idx: np.ndarray        # int32 [k], ascending
    sim: np.ndarray        # float32 [N], fixed-order cosine
    refreshed: np.ndarray  # [k][D] = Y[idx]
    t0: np.ndarray         # float32 [N][D] embedded tokens of this frame
    sv: Optional[np.ndarray] = None  # float32 [N][D] score vectors (t0 or first-layer keys)

    @property
    def count(self) -> int:
        return int(self.idx.shape[0])


def embed(model: Model, patches: np.ndarray) -> np.ndarray:
    """Patch embedding + Pos for all tokens, fixed fp32 order; [N][D] fp32."""
    w = model.w32
    return pinned.embed_f32(patches, w["w_pe"], w["b_pe"], w["pos"])


def key_score(model: Model, t0: np.ndarray) -> np.ndarray:
    """First-layer keys of every token, fixed fp32 order: LayerNorm 1 of layer
    0 on the stored layer input S(t0), then the key projection (eq. 3 compares
    these keys); [N][D] fp32."""
    w = model.w32
    return pinned.key_score_f32(t0, w["ln1_g"], w["ln1_b"], w["w_k"], w["b_k"], model.eps,
                                model.dtype == "bf16")


def score_vectors(model: Model, t0: np.ndarray) -> np.ndarray:
    """The per-token vectors the cosine of eq. 3 compares, [N][D] fp32."""
    if model.score == "key":
        return key_score(model, t0)
    return t0


def attn_branch(model: Model, l: int, Z: np.ndarray, U: np.ndarray, K: np.ndarray, V: np.ndarray,
                trace: Optional[dict] = None) -> np.ndarray:
    """Attention branch of layer l for the rows U (inputs Z, [|U|][D]):
    B = S(S(Attn(Q, K, V)) W_o + b_o).  The new K/V rows of U are written into
    the layer's full [N][D] caches K, V before the attention (eq. 5), so the
    updated queries see the new keys of U and the cached keys of the rest."""
    m, dt = model.shape, model.dtype
    D = m.dim
    A = S(layer_norm(Z, model.p(l, "ln1_g"), model.p(l, "ln1_b"), model.eps), dt)
    qkv = S(A @ model.p(l, "w_qkv") + model.p(l, "b_qkv"), dt)     # eq. 4
    K[U] = qkv[:, D:2 * D]
    V[U] = qkv[:, 2 * D:]
    O = S(attention(qkv[:, :D], K, V, m.heads), dt)
    if trace is not None:
        trace.setdefault("O", []).append(O)
    return S(O @ model.p(l, "w_o") + model.p(l, "b_o"), dt)


def mlp_block(model: Model, l: int, X: np.ndarray, Bo: np.ndarray, trace: Optional[dict] = None) -> np.ndarray:
    """Residual add of the attention branch, then the MLP with its residual:
    H = S(X + B), X' = S(H + S(S(GELU(S(S(LN2(H)) W_1 + b_1))) W_2 + b_2))."""
    dt = model.dtype
    Hres = S(X + Bo, dt)
    if trace is not None:
        trace.setdefault("H", []).append(Hres)
    A2 = S(layer_norm(Hres, model.p(l, "ln2_g"), model.p(l, "ln2_b"), model.eps), dt)
    F1 = S(A2 @ model.p(l, "w_1") + model.p(l, "b_1"), dt)
    G = S(gelu_tanh(F1), dt)
    M2 = S(G @ model.p(l, "w_2") + model.p(l, "b_2"), dt)
    return S(Hres + M2, dt)


def layer_rows(model: Model, l: int, Z: np.ndarray, U: np.ndarray, K: np.ndarray, V: np.ndarray,
               trace: Optional[dict] = None) -> np.ndarray:
    """Layer l for the rows U, whose inputs are Z ([|U|][D]); K, V are the
    layer's full [N][D] key/value caches (updated in place).  Returns the
    layer's output rows."""
    return mlp_block(model, l, Z, attn_branch(model, l, Z, U, K, V, trace), trace)


def layer_all(model: Model, l: int, X: np.ndarray, U: np.ndarray, K: np.ndarray, V: np.ndarray,
              A: np.ndarray, trace: Optional[dict] = None) -> np.ndarray:
    """Layer l in the "all" reading: the attention branch for the rows U only
    (new K/V rows scattered first) goes into the branch cache A; every row then
    adds its A row (new for U, cached for the rest) to its current input and
    goes through the MLP.  X: [N][D] inputs of all rows; returns the [N][D]
    outputs."""
    if U.size:
        A[U] = attn_branch(model, l, X[U], U, K, V, trace)
    return mlp_block(model, l, X, A, trace)


def final_rows(model: Model, Z: np.ndarray) -> np.ndarray:
    """Final LayerNorm of the last layer's output rows."""
    return S(layer_norm(Z, model.w["lnf_g"], model.w["lnf_b"], model.eps), model.dtype)


def _encode_rows(model: Model, cache: ViewCache, U: np.ndarray, t0: np.ndarray, sv: np.ndarray,
                 trace: Optional[dict] = None) -> None:
    """Recompute rows U through every layer against the cached rows R.

    The caller has already decided U; the same rows are recomputed in every
    layer, and their score vectors `sv` become their new references.  `trace`,
    if given, collects the per-layer attention outputs and residuals of the
    rows U (for tests)."""
    cache.ref[U] = sv[U]
    Z = S(t0[U].astype(np.float64), model.dtype)
    cache.X[0][U] = Z
    for l in range(model.shape.depth):
        Z = layer_rows(model, l, Z, U, cache.K[l], cache.V[l], trace)
        cache.X[l + 1][U] = Z
    cache.Y[U] = final_rows(model, Z)


def _encode_all(model: Model, cache: ViewCache, U: np.ndarray, t0: np.ndarray, sv: np.ndarray,
                trace: Optional[dict] = None) -> None:
    """The "all" reading of one frame: rows U are refreshed (new reference,
    new Q/K/V and attention); every row's layer-0 input is this frame's
    embedded token and every row goes through every MLP."""
    cache.ref[U] = sv[U]
    X = S(t0.astype(np.float64), model.dtype)
    cache.X[0] = X
    for l in range(model.shape.depth):
        X = layer_all(model, l, X, U, cache.K[l], cache.V[l], cache.A[l], trace)
        cache.X[l + 1] = X
    cache.Y = final_rows(model, X)


def empty_cache(model: Model) -> ViewCache:
    m = model.shape
    N, D, L = m.n_tokens, m.dim, m.depth
    return ViewCache(ref=np.zeros((N, D), np.float32), X=np.zeros((L + 1, N, D)),
                     K=np.zeros((L, N, D)), V=np.zeros((L, N, D)), Y=np.zeros((N, D)),
                     A=np.zeros((L, N, D)) if model.mlp == "all" else None)


def full_encode(model: Model, patches: np.ndarray) -> ViewCache:
    """Full forward of one frame; fills every cache row (the paper's odd chunk)."""
    cache = empty_cache(model)
    t0 = embed(model, patches)
    encode = _encode_all if model.mlp == "all" else _encode_rows
    encode(model, cache, np.arange(model.shape.n_tokens), t0, score_vectors(model, t0))
    return cache


def step(model: Model, patches: np.ndarray, cache: ViewCache, tau: float, cap: int,
         trace: Optional[dict] = None) -> StepResult:
    """Incremental encode of one frame; updates `cache` in place."""
    t0 = embed(model, patches)
    sv = score_vectors(model, t0)
    sim = pinned.cosine_f32(sv, cache.ref)
    U = select(sim, tau, cap)
    if model.mlp == "all":  # every row follows the new frame, even when U is empty
        _encode_all(model, cache, U, t0, sv, trace)
    elif U.size:
        _encode_rows(model, cache, U, t0, sv, trace)
    return StepResult(idx=U, sim=sim, refreshed=cache.Y[U].copy(), t0=t0, sv=sv)


def run_schedule(model: Model, frames: Sequence[np.ndarray], period: int, tau: float, cap: int,
                 cache: Optional[ViewCache] = None, first: int = 0):
    """Encode one stream frame by frame under a refresh period (§III-B): frame
    t (counted from `first`) is encoded in full when t % period == 0, which
    replaces every cached row and reference, and incrementally otherwise.
    Period 2 is the paper's odd/even chunk schedule: the incremental frames
    compare against the keys of the preceding full pass.  A full frame reports
    every token as refreshed.  Returns (cache, [StepResult per frame])."""
    if period < 1:
        raise ValueError("period must be >= 1")
    out = []
    for j, patches in enumerate(frames):
        t = first + j
        if t % period == 0 or cache is None:
            cache = full_encode(model, patches)
            n = model.shape.n_tokens
            t0 = embed(model, patches)
            out.append(StepResult(idx=np.arange(n, dtype=np.int32), sim=np.full(n, np.nan, np.float32),
                                  refreshed=cache.Y.copy(), t0=t0, sv=cache.ref.copy()))
        else:
            out.append(step(model, patches, cache, tau, cap))
    return cache, out


def full_forward_dense(model: Model, patches: np.ndarray) -> np.ndarray:
    """Y of a plain full forward (no cache); same as full_encode(...).Y."""
    return full_encode(model, patches).Y
