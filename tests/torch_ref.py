"""An independent float64 ViT written with torch functional ops.

Used only as a pin for the oracle: the patch embedding is F.conv2d over the
image (which also checks the patch/feature order), and every layer is built
from F.layer_norm, F.linear, F.scaled_dot_product_attention and
F.gelu(approximate='tanh').  It applies no storage rounding, so it is compared
with the oracle's "f64" mode.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def t64(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def conv_embed(m, w, frame: np.ndarray) -> torch.Tensor:
    """[N][D] = conv2d(frame, W_pe as a (D, C, p, p) kernel, stride p) + b_pe + Pos."""
    D, C, p = m.dim, m.channels, m.patch
    kernel = t64(w["w_pe"]).T.reshape(D, C, p, p)
    y = F.conv2d(t64(frame)[None], kernel, t64(w["b_pe"]), stride=p)  # (1, D, gh, gw)
    return y[0].reshape(D, -1).T + t64(w["pos"])


def layer(m, w, l: int, x: torch.Tensor) -> torch.Tensor:
    """One pre-LN encoder layer over all rows of x: [N][D] -> [N][D]."""
    D, h = m.dim, m.heads
    dh = D // h
    g = lambda n: t64(w[f"l{l}.{n}"])
    a = F.layer_norm(x, (D,), g("ln1_g"), g("ln1_b"), m.ln_eps)
    qkv = F.linear(a, g("w_qkv").T, g("b_qkv"))
    q, k, v = qkv.split(D, dim=-1)
    heads = lambda t: t.reshape(-1, h, dh).transpose(0, 1)  # (h, N, dh)
    o = F.scaled_dot_product_attention(heads(q)[None], heads(k)[None], heads(v)[None])[0]
    o = o.transpose(0, 1).reshape(-1, D)
    hres = x + F.linear(o, g("w_o").T, g("b_o"))
    a2 = F.layer_norm(hres, (D,), g("ln2_g"), g("ln2_b"), m.ln_eps)
    f = F.gelu(F.linear(a2, g("w_1").T, g("b_1")), approximate="tanh")
    return hres + F.linear(f, g("w_2").T, g("b_2"))


def kv_of(m, w, l: int, x: torch.Tensor):
    """K and V rows a layer computes from its input rows x."""
    D = m.dim
    a = F.layer_norm(x, (D,), t64(w[f"l{l}.ln1_g"]), t64(w[f"l{l}.ln1_b"]), m.ln_eps)
    qkv = F.linear(a, t64(w[f"l{l}.w_qkv"]).T, t64(w[f"l{l}.b_qkv"]))
    return qkv[:, D:2 * D], qkv[:, 2 * D:]


def forward_from_tokens(m, w, x0: torch.Tensor):
    """All layer inputs X[0..L] and the final output Y, from X[0] = x0."""
    xs = [x0]
    for l in range(m.depth):
        xs.append(layer(m, w, l, xs[-1]))
    y = F.layer_norm(xs[-1], (m.dim,), t64(w["lnf_g"]), t64(w["lnf_b"]), m.ln_eps)
    return xs, y
