"""Pins of the oracle's RoPE (Sec. 2.1, Eq. 1-2) and the RoPE-first rotation
identity (Sec. 3.1, Eq. 4) by closed forms and invariants."""
import numpy as np
import pytest

from oracle import oracle
from paper_2603_26110_amd import synth


@pytest.fixture(scope="module")
def cs():
    return oracle.rope_table(4096, 10000.0)


def test_table_closed_forms(cs):
    assert cs.shape == (4096, 32, 2)
    # position 0 is the identity
    np.testing.assert_array_equal(cs[0, :, 0], 1.0)
    np.testing.assert_array_equal(cs[0, :, 1], 0.0)
    # theta_0 = 1: pair 0 turns by p radians
    p = np.arange(4096)
    np.testing.assert_array_equal(cs[:, 0, 0], np.cos(p).astype(np.float32))
    np.testing.assert_array_equal(cs[:, 0, 1], np.sin(p).astype(np.float32))
    # theta_16 = 10000^(-1/2) = 0.01 exactly in real arithmetic
    np.testing.assert_allclose(cs[:, 16, 0], np.cos(0.01 * p), atol=2e-7)
    np.testing.assert_allclose(cs[:, 16, 1], np.sin(0.01 * p), atol=2e-7)
    # theta_31 = 10000^(-62/64)
    th = 10000.0 ** (-62 / 64)
    np.testing.assert_allclose(cs[:, 31, 1], np.sin(th * p), atol=2e-7)
    # unit modulus up to fp32 rounding
    np.testing.assert_allclose(cs[..., 0].astype(np.float64) ** 2 + cs[..., 1].astype(np.float64) ** 2,
                               1.0, atol=1e-6)


def test_rope_matrix_matches_eq2(cs):
    # Build R_{theta,p} explicitly as the block-diagonal matrix of Eq. 2.
    g = synth.rng(1)
    x = g.standard_normal(64)
    for p in [0, 1, 7, 513, 4095]:
        R = np.zeros((64, 64))
        for m in range(32):
            c, s = float(cs[p, m, 0]), float(cs[p, m, 1])
            R[2 * m:2 * m + 2, 2 * m:2 * m + 2] = [[c, -s], [s, c]]
        np.testing.assert_allclose(oracle.rope_apply(x, p, cs), R @ x, rtol=0, atol=1e-13)


def test_half_pairing_rotates_m_with_m_plus_32(cs):
    g = synth.rng(2)
    x = g.standard_normal(64)
    p = 321
    y = oracle.rope_apply(x, p, cs, half=True)
    for m in range(32):
        c, s = float(cs[p, m, 0]), float(cs[p, m, 1])
        assert abs(y[m] - (x[m] * c - x[m + 32] * s)) < 1e-13
        assert abs(y[m + 32] - (x[m] * s + x[m + 32] * c)) < 1e-13


def test_relative_position_property(cs):
    # (R_{i+s} q)^T (R_{j+s} k) = (R_i q)^T (R_j k): only j - i matters (Sec. 2.1).
    g = synth.rng(3)
    for _ in range(20):
        q, k = g.standard_normal(64), g.standard_normal(64)
        i, j, s = (int(v) for v in g.integers(0, 1300, 3))
        a = oracle.rope_apply(q, i + s, cs) @ oracle.rope_apply(k, j + s, cs)
        b = oracle.rope_apply(q, i, cs) @ oracle.rope_apply(k, j, cs)
        assert abs(a - b) <= 2e-5 * (np.linalg.norm(q) * np.linalg.norm(k))


def test_rope_preserves_norm(cs):
    g = synth.rng(4)
    x = g.standard_normal(64)
    for p in [5, 999, 3000]:
        assert abs(np.linalg.norm(oracle.rope_apply(x, p, cs)) - np.linalg.norm(x)) < 1e-6


def test_rope_first_identity_eq4(cs):
    # (Pi R_i q)^T (Pi R_j k) = (R_i q)^T (R_j k) for orthogonal Pi (Eq. 4).
    g = synth.rng(5)
    pi = np.linalg.qr(g.standard_normal((64, 64)))[0]
    for _ in range(20):
        q, k = g.standard_normal(64), g.standard_normal(64)
        i, j = (int(v) for v in g.integers(0, 4096, 2))
        rq, rk = oracle.rope_apply(q, i, cs), oracle.rope_apply(k, j, cs)
        lhs = (pi @ rq) @ (pi @ rk)
        rhs = rq @ rk
        assert abs(lhs - rhs) <= 1e-12 * np.linalg.norm(q) * np.linalg.norm(k)


def test_rotation_before_rope_breaks_the_score(cs):
    # Pi applied before RoPE mixes the RoPE pairs (Sec. 3.1): the score no
    # longer equals the unrotated attention score, while Pi after RoPE does.
    g = synth.rng(6)
    pi = np.linalg.qr(g.standard_normal((64, 64)))[0]
    q, k = g.standard_normal(64), g.standard_normal(64)
    scale = np.linalg.norm(q) * np.linalg.norm(k)
    for i, j in [(10, 50), (300, 7), (1000, 1023)]:
        true = oracle.rope_apply(q, i, cs) @ oracle.rope_apply(k, j, cs)
        after = (pi @ oracle.rope_apply(q, i, cs)) @ (pi @ oracle.rope_apply(k, j, cs))
        before = oracle.rope_apply(pi @ q, i, cs) @ oracle.rope_apply(pi @ k, j, cs)
        assert abs(after - true) < 1e-10 * scale
        assert abs(before - true) > 1e-2 * scale


def test_rotated_input_matches_definition(cs):
    g = synth.rng(7)
    pi = synth.random_rotation(g)
    k = g.standard_normal(64).astype(np.float32)
    v = g.standard_normal(64).astype(np.float32)
    kh = oracle.rotated_input(k, True, 77, cs, pi)
    np.testing.assert_allclose(kh, pi.astype(np.float64) @ oracle.rope_apply(k, 77, cs), rtol=1e-6, atol=1e-6)
    vh = oracle.rotated_input(v, False, 77, cs, pi, rotate_v=True)
    np.testing.assert_allclose(vh, pi.astype(np.float64) @ v.astype(np.float64), rtol=1e-6, atol=1e-6)
    vu = oracle.rotated_input(v, False, 77, cs, pi, rotate_v=False)
    np.testing.assert_array_equal(vu, v)
