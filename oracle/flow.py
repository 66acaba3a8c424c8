"""CPU oracle of the compressed 2-step flow update (paper §III-C).

TEST INFRASTRUCTURE ONLY: imported by ``tests/`` and never by the product
path; it shares no code with the HIP library.

The paper writes the Euler solution of the flow ODE as the sum of the step
velocities, models each velocity as a combination of two anchor velocities
(the first one, v_0, and a mid-trajectory one, v_7) plus a residual, and so
reduces the final state to x_T = x_0 + alpha v_0 + beta v_7 + b, where alpha,
beta and b collect the per-step coefficients and residuals.  In the paper a
trained adaptor predicts (alpha, beta, b) from v_0; here they are inputs, or
are fitted from a known velocity sequence by least squares, which makes the
two-anchor formula reproduce the Euler sum by construction.

Everything is float64.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np


def euler_final(x0: np.ndarray, velocities: Sequence[np.ndarray], dt: float) -> np.ndarray:
    """x_T = x_0 + sum_t dt * v_t (the explicit Euler steps, summed)."""
    out = np.asarray(x0, dtype=np.float64).copy()
    for v in velocities:
        out = out + dt * np.asarray(v, dtype=np.float64)
    return out


def fit_anchors(velocities: Sequence[np.ndarray], dt: float, i0: int = 0, i1: int = 7
                ) -> Tuple[float, float, np.ndarray]:
    """Per step t, the least-squares (a_t, b_t) of v_t ~ a_t v_i0 + b_t v_i1 and
    its residual e_t; returns alpha = sum dt a_t, beta = sum dt b_t and
    b = sum dt e_t (the anchors' own coefficients are 1 and 0 exactly)."""
    v = [np.asarray(x, dtype=np.float64).ravel() for x in velocities]
    basis = np.stack([v[i0], v[i1]], axis=1)
    alpha, beta = 0.0, 0.0
    resid = np.zeros_like(v[0])
    for t, vt in enumerate(v):
        if t == i0:
            a, b = 1.0, 0.0
        elif t == i1:
            a, b = 0.0, 1.0
        else:
            (a, b), *_ = np.linalg.lstsq(basis, vt, rcond=None)
        alpha += dt * a
        beta += dt * b
        resid += dt * (vt - a * v[i0] - b * v[i1])
    return alpha, beta, resid.reshape(np.shape(velocities[0]))


def two_anchor_final(x0: np.ndarray, v0: np.ndarray, v7: np.ndarray, alpha, beta, b) -> np.ndarray:
    """x_T = x_0 + alpha v_0 + beta v_7 + b, per sample: x0, v0, v7, b are
    [S][...]; alpha, beta are [S]."""
    x0 = np.asarray(x0, dtype=np.float64)
    shape = (-1,) + (1,) * (x0.ndim - 1)
    al = np.asarray(alpha, dtype=np.float64).reshape(shape)
    be = np.asarray(beta, dtype=np.float64).reshape(shape)
    return x0 + al * np.asarray(v0, np.float64) + be * np.asarray(v7, np.float64) + np.asarray(b, np.float64)
