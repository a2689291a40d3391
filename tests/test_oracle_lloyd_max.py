"""Pins of the oracle's Lloyd-Max levels (Sec. 3.3, Eq. 5) and 1-D k-means LUT
calibration (Sec. 4.1) against published values, quadrature and brute force."""
import os

import numpy as np
import pytest
from scipy import integrate
from scipy.stats import norm

from oracle import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lloyd_max_gauss_3bit.txt")


def _golden():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, idx, val, tol = line.split()
            rows.append((kind, int(idx), float(val), float(tol)))
    return rows


def test_gaussian_levels_match_published_table():
    c, t, mse = oracle.lloyd_max_gaussian(8)
    for kind, i, val, tol in _golden():
        got = {"level": c, "level4": c, "threshold": t}.get(kind)
        if kind == "mse":
            assert abs(mse - val) <= tol, (mse, val)
        else:
            assert abs(got[i] - val) <= tol, (kind, i, got[i], val)


def test_gaussian_levels_satisfy_centroid_condition_by_quadrature():
    # Each level is the conditional mean of N(0,1) over its cell, computed here
    # by adaptive quadrature instead of the closed form the oracle iterates.
    c, t, _ = oracle.lloyd_max_gaussian(8)
    edges = np.concatenate(([-np.inf], t, [np.inf]))
    for k in range(8):
        a, b = edges[k], edges[k + 1]
        num = integrate.quad(lambda x: x * norm.pdf(x), a, b, epsabs=1e-14)[0]
        den = integrate.quad(norm.pdf, a, b, epsabs=1e-14)[0]
        assert abs(num / den - c[k]) < 1e-9
    # thresholds are midpoints (nearest-level rule)
    np.testing.assert_allclose(t, 0.5 * (c[:-1] + c[1:]), atol=0)
    # symmetric distribution -> symmetric quantizer
    np.testing.assert_allclose(c, -c[::-1], atol=1e-12)


def test_gaussian_mse_matches_quadrature_and_sampling():
    c, t, mse = oracle.lloyd_max_gaussian(8)
    edges = np.concatenate(([-np.inf], t, [np.inf]))
    quad = sum(integrate.quad(lambda x, ck=c[k]: (x - ck) ** 2 * norm.pdf(x),
                              edges[k], edges[k + 1], epsabs=1e-14)[0] for k in range(8))
    assert abs(quad - mse) < 1e-10
    g = np.random.Generator(np.random.PCG64(7))
    x = g.standard_normal(1_000_000)
    err = (x - c[oracle.assign_levels(x, c)]) ** 2
    se = err.std() / np.sqrt(len(x))
    assert abs(err.mean() - mse) < 4 * se


def test_one_bit_case_is_textbook():
    # 2 levels for N(0,1): +-sqrt(2/pi), threshold 0, MSE 1 - 2/pi.
    c, t, mse = oracle.lloyd_max_gaussian(2)
    np.testing.assert_allclose(c, [-np.sqrt(2 / np.pi), np.sqrt(2 / np.pi)], atol=1e-12)
    assert abs(t[0]) < 1e-15
    assert abs(mse - (1 - 2 / np.pi)) < 1e-12


def test_assign_levels_is_nearest_with_ties_low():
    c = np.array([-3.0, -1.0, 0.0, 1.0, 2.0, 4.0, 5.0, 9.0])
    x = np.array([-5, -2.0, -1.9, -0.5, 0.5, 0.51, 1.5, 3.0, 3.01, 4.5, 7.0, 100.0])
    got = oracle.assign_levels(x, c)
    brute = []
    for v in x:
        d = np.abs(v - c)
        brute.append(int(np.flatnonzero(d == d.min())[0]))   # first (lower) on ties
    np.testing.assert_array_equal(got, brute)


def test_kmeans_recovers_atoms_exactly():
    atoms = np.array([-4.0, -2.5, -1.0, -0.25, 0.5, 1.5, 3.0, 6.0])
    g = np.random.Generator(np.random.PCG64(3))
    x = atoms[g.integers(0, 8, 20000)]
    init = np.linspace(-3, 3, 8)
    c = oracle.kmeans_1d(x, init, max_iter=200)
    np.testing.assert_allclose(c, atoms, atol=1e-12)


def test_kmeans_on_gaussian_samples_approaches_lloyd_max():
    g = np.random.Generator(np.random.PCG64(11))
    x = g.standard_normal(400_000)
    ref, _, _ = oracle.lloyd_max_gaussian(8)
    c = oracle.kmeans_1d(x, ref)
    assert np.max(np.abs(c - ref)) < 0.02


def test_kmeans_keeps_level_of_empty_cell():
    x = np.array([0.0, 0.1, 0.2, 5.0, 5.1])
    init = np.array([0.1, 2.0, 5.05])       # middle cell attracts nothing
    c = oracle.kmeans_1d(x, init)
    np.testing.assert_allclose(c, [0.1, 2.0, 5.05], atol=1e-12)


@pytest.mark.parametrize("levels", [4, 8, 16])
def test_lloyd_max_iteration_is_a_fixed_point(levels):
    c, t, _ = oracle.lloyd_max_gaussian(levels)
    edges = np.concatenate(([-np.inf], t, [np.inf]))
    mass = norm.cdf(edges[1:]) - norm.cdf(edges[:-1])
    cn = (norm.pdf(edges[:-1]) - norm.pdf(edges[1:])) / mass
    assert np.max(np.abs(cn - c)) < 1e-13
    assert np.all(np.diff(c) > 0)


# ---- calibrated tables: normalized coordinates and the per-head Lloyd fit
def test_normalized_coordinates_have_norm_8_and_the_rotated_direction():
    g = np.random.Generator(np.random.PCG64(21))
    x = g.standard_normal((50, 64)) * np.exp(g.standard_normal((50, 1)))
    q, _ = np.linalg.qr(g.standard_normal((64, 64)))
    u = oracle.normalized_coordinates(x, q)
    np.testing.assert_allclose(np.linalg.norm(u, axis=1), 8.0, rtol=1e-14)
    xh = x @ q.T
    cos = np.sum(u * xh, axis=1) / (8.0 * np.linalg.norm(xh, axis=1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-14)
    z = oracle.normalized_coordinates(np.zeros((2, 64)), q)
    assert np.all(z == 0.0)
    # no rotation: the unit vector of x itself, times 8
    np.testing.assert_allclose(oracle.normalized_coordinates(x, None),
                               8.0 * x / np.linalg.norm(x, axis=1, keepdims=True), rtol=1e-14)


def test_calibrated_table_of_isotropic_vectors_fits_the_exact_marginal():
    # For isotropic vectors in 64 dimensions (any rotation), a normalized
    # coordinate is u = 8 t with t the coordinate of a uniform unit vector:
    # t^2 ~ Beta(1/2, 63/2), symmetric sign. The table calibrated on the
    # vectors must match the Lloyd fit of samples drawn from that law directly
    # (a wrong scale, a missing rotation or a norm of the unrotated vector
    # would all move it).
    g = np.random.Generator(np.random.PCG64(22))
    x = g.standard_normal((20000, 64))
    q, _ = np.linalg.qr(g.standard_normal((64, 64)))
    ref, _, _ = oracle.lloyd_max_gaussian(8)
    c = oracle.calibrate_lut(x, q, ref)
    t = np.sqrt(g.beta(0.5, 31.5, 2_000_000)) * np.where(g.random(2_000_000) < 0.5, -1.0, 1.0)
    c_law = oracle.kmeans_1d(8.0 * t, ref)
    assert np.all(np.diff(c) > 0)
    assert np.max(np.abs(c - c_law)) < 0.01, np.abs(c - c_law)
    # lighter tails than N(0, 1): the outer levels sit inside the Gaussian ones
    assert c[-1] < ref[-1] and c[0] > ref[0]
