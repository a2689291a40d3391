"""Pins of oracle.calibrate_ebar, the per-head mean absolute residual of the
per-element correction (Sec. 3.4, Eq. 7): hand-worked vectors whose
normalized coordinates and nearest levels are known exactly, invariance under
a rotation that the calibration undoes, and the expectation under the exact
law of a coordinate of an isotropic 64-vector (t^2 ~ Beta(1/2, 63/2), u = 8t),
computed by quadrature."""
import numpy as np
import pytest
from scipy import integrate, special

from oracle import oracle

# an asymmetric table (catches a sign or index slip): midpoints
# -2.5, -1.5, -0.75, -0.125, 0.625, 1.5, 2.5
LEVELS = np.array([-3.0, -2.0, -1.0, -0.5, 0.25, 1.0, 2.0, 3.0])


def test_one_hot_vector():
    # u = (8, 0, ..., 0): 8 -> level 3 (|8 - 3| = 5), 0 -> level 0.25 (the
    # midpoint -0.125 is below 0, 0.625 above), 63 of them
    x = np.zeros((1, 64))
    x[0, 0] = 1.0
    assert oracle.calibrate_ebar(x, None, LEVELS) == pytest.approx((5.0 + 63 * 0.25) / 64, abs=1e-15)
    # the norm is divided out
    assert oracle.calibrate_ebar(37.5 * x, None, LEVELS) == pytest.approx((5.0 + 63 * 0.25) / 64, abs=1e-15)


def test_worked_pair_of_vectors_and_zero_vector():
    # (3, 4, 0, ...): norm 5, u = (4.8, 6.4, 0, ...): residuals 1.8, 3.4 and 62 x 0.25
    a = np.zeros(64)
    a[:2] = (3.0, 4.0)
    b = np.zeros(64)
    b[5] = -2.0                       # u_5 = -8 -> level -3, residual 5
    z = np.zeros(64)                  # zero vector: every u = 0, residual 0.25
    x = np.stack([a, b, z])
    want = ((1.8 + 3.4 + 62 * 0.25) + (5.0 + 63 * 0.25) + 64 * 0.25) / (3 * 64)
    assert oracle.calibrate_ebar(x, None, LEVELS) == pytest.approx(want, abs=1e-14)


def test_coordinates_in_every_cell():
    # u = 8 x / ||x|| with ||x|| = 8: u equals x. One coordinate in each of the
    # eight cells (nearest levels by hand), one coordinate carrying the rest of
    # the norm, the other 55 zero (level 0.25).
    u = np.array([-2.9, -1.7, -0.9, -0.3, 0.1, 0.9, 1.6, 2.7])
    near = np.array([-3.0, -2.0, -1.0, -0.5, 0.25, 1.0, 2.0, 3.0])
    rest = np.sqrt(64.0 - np.sum(u * u))      # about 4.76 -> level 3
    x = np.zeros((1, 64))
    x[0, :8] = u
    x[0, 8] = rest
    want = (np.sum(np.abs(u - near)) + abs(rest - 3.0) + 55 * 0.25) / 64
    assert oracle.calibrate_ebar(x, None, LEVELS) == pytest.approx(want, abs=1e-12)


def test_rotation_is_applied_before_normalizing():
    g = np.random.default_rng(5)
    q, _ = np.linalg.qr(g.standard_normal((64, 64)))
    x = np.zeros((1, 64))
    x[0, 0] = 1.0
    # x = Q^T e_0 rotated by Pi = Q gives e_0 back
    assert oracle.calibrate_ebar(x @ q, q, LEVELS) == pytest.approx((5.0 + 63 * 0.25) / 64, abs=1e-12)
    # without Pi the same vector is spread over all coordinates: a different value
    assert abs(oracle.calibrate_ebar(x @ q, None, LEVELS) - (5.0 + 63 * 0.25) / 64) > 1e-3


def test_isotropic_vectors_follow_the_coordinate_law():
    # E|u - c(u)| for u = 8t, t a coordinate of a uniform unit 64-vector:
    # density of t is (1 - t^2)^(61/2) / B(1/2, 63/2) on [-1, 1]
    c = LEVELS
    t_mid = 0.5 * (c[:-1] + c[1:]) / 8.0
    norm = special.beta(0.5, 31.5)
    edges = np.concatenate(([-1.0], t_mid, [1.0]))
    exact = 0.0
    for k in range(8):
        f = lambda t, k=k: abs(8.0 * t - c[k]) * (1.0 - t * t) ** 30.5 / norm
        val, _ = integrate.quad(f, edges[k], edges[k + 1], points=[c[k] / 8.0] if edges[k] < c[k] / 8 < edges[k + 1] else None,
                                epsabs=1e-13, epsrel=1e-12, limit=200)
        exact += val
    g = np.random.default_rng(11)
    x = g.standard_normal((20000, 64))
    got = oracle.calibrate_ebar(x, None, LEVELS)
    # standard error from the per-vector means (coordinates of one vector are
    # not independent)
    u = oracle.normalized_coordinates(x, None)
    idx = oracle.assign_levels(u.reshape(-1), c).reshape(u.shape)
    per_vec = np.mean(np.abs(u - c[idx]), axis=1)
    se = per_vec.std(ddof=1) / np.sqrt(len(per_vec))
    assert abs(got - exact) < 4 * se, (got, exact, se)
    # a plausible slip (normalizing to unit norm instead of norm 8) is far off
    assert abs(got - exact) * 50 < abs(exact - np.mean(np.abs(u / 8 - c[oracle.assign_levels(u.reshape(-1) / 8, c)].reshape(u.shape))))
