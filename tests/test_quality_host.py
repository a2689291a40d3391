"""Host-side pieces of the quality ablation: the fp64 exact-attention
reference against closed forms (no GPU)."""
import numpy as np

from paper_2603_26110_amd import quality


def test_rope_preserves_norm_and_relative_position():
    g = np.random.default_rng(3)
    x = g.standard_normal((5, 64))
    y = g.standard_normal((5, 64))
    pos = np.array([0, 1, 7, 100, 1023])
    rx = quality._rope(x, pos)
    assert np.allclose(np.linalg.norm(rx, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)
    assert np.allclose(rx[0], x[0])                       # position 0 is the identity
    # (R_{i+s} a) . (R_{j+s} b) = (R_i a) . (R_j b)
    a, b = x[1], y[2]
    d0 = quality._rope(a[None], np.array([3]))[0] @ quality._rope(b[None], np.array([10]))[0]
    d1 = quality._rope(a[None], np.array([50]))[0] @ quality._rope(b[None], np.array([57]))[0]
    assert abs(d0 - d1) < 1e-9 * (1 + abs(d0))


def test_exact_attention_special_cases():
    g = np.random.default_rng(4)
    H, T = 3, 9
    v = g.standard_normal((T, H, 64))
    q = np.zeros((H, 64))                                  # zero query: uniform weights
    k = g.standard_normal((T, H, 64))
    o = quality.exact_attention(q, k, v, T - 1)
    assert np.allclose(o, v.mean(axis=0), atol=1e-12)
    o1 = quality.exact_attention(g.standard_normal((H, 64)), k[:1], v[:1], 0)   # one token
    assert np.allclose(o1, v[0], atol=1e-12)
