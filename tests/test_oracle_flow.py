"""Pins of the oracle's two-anchor flow update (paper §III-C).

* the Euler sum against a step-by-step loop written out here;
* velocities that lie exactly in the span of the two anchors: the fitted
  residual is zero and the two-anchor formula equals the Euler result;
* general velocities: with the fitted residual the formula reproduces the
  Euler result exactly (up to rounding), and without it the error is the
  residual;
* a constant velocity field: the two anchors coincide, the split between
  alpha and beta is not unique, but alpha + beta = T dt and the residual is 0.
"""
import numpy as np

from oracle import flow


def test_euler_final_is_the_step_loop():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 50, 32))
    vs = [rng.standard_normal((4, 50, 32)) for _ in range(10)]
    y = x.copy()
    for v in vs:
        y = y + 0.1 * v
    assert np.allclose(flow.euler_final(x, vs, 0.1), y, rtol=0, atol=1e-13)


def test_low_rank_velocities_are_reproduced_exactly():
    rng = np.random.default_rng(2)
    u0, u1 = rng.standard_normal(200), rng.standard_normal(200)
    coef = rng.standard_normal((10, 2))
    vs = [c0 * u0 + c1 * u1 for c0, c1 in coef]
    x0 = rng.standard_normal(200)
    alpha, beta, b = flow.fit_anchors(vs, 0.1)
    assert np.abs(b).max() < 1e-12
    y = flow.two_anchor_final(x0[None], vs[0][None], vs[7][None], [alpha], [beta], b[None])[0]
    assert np.allclose(y, flow.euler_final(x0, vs, 0.1), rtol=0, atol=1e-12)


def test_residual_closes_the_gap_for_general_velocities():
    rng = np.random.default_rng(3)
    vs = [rng.standard_normal(300) for _ in range(10)]
    x0 = rng.standard_normal(300)
    alpha, beta, b = flow.fit_anchors(vs, 0.1)
    exact = flow.euler_final(x0, vs, 0.1)
    y = flow.two_anchor_final(x0[None], vs[0][None], vs[7][None], [alpha], [beta], b[None])[0]
    assert np.allclose(y, exact, rtol=0, atol=1e-12)
    y0 = flow.two_anchor_final(x0[None], vs[0][None], vs[7][None], [alpha], [beta], np.zeros((1, 300)))[0]
    assert np.allclose(exact - y0, b, rtol=0, atol=1e-12) and np.abs(b).max() > 1e-2


def test_constant_velocity_closed_form():
    rng = np.random.default_rng(4)
    v = rng.standard_normal(64)
    alpha, beta, b = flow.fit_anchors([v] * 10, 0.1)
    assert abs(alpha + beta - 1.0) < 1e-12 and np.abs(b).max() < 1e-12
