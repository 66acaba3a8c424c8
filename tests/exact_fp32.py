"""Exact emulation of fp32 operations with Python rationals (tests only).

fmaf(a, b, c) is the exact value a*b + c rounded once to fp32 (nearest, ties
to even).  The other operations are taken in float64 and rounded to fp32: for
+, -, *, / and sqrt of fp32 operands that double rounding is exact, because
float64 carries more than 2*24+2 significand bits.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


def round_f32(x: Fraction) -> float:
    """Nearest fp32 to the exact rational x (ties to even); returns a Python float."""
    if x == 0:
        return 0.0
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length() - 24
    while a >= Fraction(2) ** (e + 24):
        e += 1
    while a < Fraction(2) ** (e + 23):
        e -= 1
    e = max(e, -149)  # fp32 subnormal spacing
    q = a / Fraction(2) ** e
    n = q.numerator // q.denominator
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return float(sign * n * Fraction(2) ** e)


def f32(x: float) -> float:
    return float(np.float32(x))


def fmaf(a: float, b: float, c: float) -> float:
    return round_f32(Fraction(a) * Fraction(b) + Fraction(c))


def add(a: float, b: float) -> float:
    return f32(a + b)


def mul(a: float, b: float) -> float:
    return f32(a * b)


def div(a: float, b: float) -> float:
    return f32(a / b)


def sqrt(a: float) -> float:
    return f32(math.sqrt(a))


def embed_token(x, w_pe, b_pe, pos_row):
    """One token of the fixed-order patch embedding, every fmaf exact."""
    P, D = w_pe.shape
    out = []
    for d in range(D):
        acc = float(b_pe[d])
        for k in range(P):
            acc = fmaf(float(x[k]), float(w_pe[k, d]), acc)
        out.append(add(acc, float(pos_row[d])))
    return np.array(out, dtype=np.float32)


def cosine(a, b):
    """Fixed-order cosine: 64 fmaf lane partials, then the halving tree."""
    D = len(a)

    def partials(u, v):
        s = []
        for j in range(64):
            acc = 0.0
            for d in range(j, D, 64):
                acc = fmaf(float(u[d]), float(v[d]), acc)
            s.append(acc)
        off = 32
        while off >= 1:
            for j in range(off):
                s[j] = add(s[j], s[j + off])
            off //= 2
        return s[0]

    dot, na, nb = partials(a, b), partials(a, a), partials(b, b)
    denom = mul(sqrt(na), sqrt(nb))
    return np.float32(div(dot, max(denom, f32(1e-8))))


def _tree64(s):
    s = list(s)
    off = 32
    while off >= 1:
        for j in range(off):
            s[j] = add(s[j], s[j + off])
        off //= 2
    return s[0]


def key_token(x, ln_g, ln_b, w_k, b_k, eps):
    """One token of the fixed-order first-layer key score, every fmaf exact.

    x: the stored layer-0 input (already rounded to the storage type);
    LayerNorm with 64 lane partials and the halving tree, then the key
    projection as one fmaf chain per output in increasing input index."""
    D = len(x)
    x = [float(v) for v in x]
    s = []
    for j in range(64):
        acc = 0.0
        for d in range(j, D, 64):
            acc = add(acc, x[d])
        s.append(acc)
    mean = div(_tree64(s), float(D))
    c = [add(v, -mean) for v in x]
    s = []
    for j in range(64):
        acc = 0.0
        for d in range(j, D, 64):
            acc = fmaf(c[d], c[d], acc)
        s.append(acc)
    var = div(_tree64(s), float(D))
    rstd = div(1.0, sqrt(add(var, f32(eps))))
    n = [fmaf(mul(c[d], rstd), float(ln_g[d]), float(ln_b[d])) for d in range(D)]
    out = []
    for e in range(D):
        acc = float(b_k[e])
        for d in range(D):
            acc = fmaf(n[d], float(w_k[d, e]), acc)
        out.append(acc)
    return np.array(out, dtype=np.float32)
