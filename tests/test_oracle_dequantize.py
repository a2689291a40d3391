"""Pins of the oracle's dequantize (the first step of a dequantize-then-attend
path, the comparison of Sec. 5.3 / Table 6): textbook softmax attention over
the dequantized keys and values reproduces the oracle's decode, which is
pinned on its own; the table term alone has the textbook distortion of the
3-bit Lloyd-Max quantizer of N(0, 1); a hand-built slot gives the defined
vector."""
import numpy as np
import pytest

from oracle import oracle
from paper_2603_26110_amd import synth
from test_oracle_decode import LUT32, SCALE, build, exact_rope

# MSE of the 8-level Lloyd-Max quantizer of a unit Gaussian (Max 1960).
LLOYD_MAX_3BIT_MSE = 0.03455


@pytest.mark.parametrize("flags", [oracle.V_ROTATE, 0, oracle.V_ROTATE | oracle.V_QJL,
                                   oracle.QJL_PAPER | oracle.V_QJL | oracle.V_ROTATE,
                                   oracle.ROPE_HALF | oracle.V_ROTATE])
def test_attention_over_dequantized_rows_equals_decode(flags):
    g = synth.rng(31)
    L, H, n, max_len = 2, 3, 150, 160
    st = build(g, n, L, H, flags=flags, slots=192)
    q = g.standard_normal((L, 1, H, 64)).astype(np.float32)
    ebar = np.full((L, H, 2), 0.3, np.float32)
    qpos = n + 5
    ref = oracle.decode(st["cache"], flags, st["cs"], q, [qpos], [0], [n], st["pi"], st["luts"],
                        st["luts"], st["S"], ebar=ebar)
    kt, vt = oracle.dequantize(st["cache"], flags, [0], [n], max_len, st["luts"], st["luts"], st["S"],
                               ebar=ebar)
    assert np.all(np.isfinite(kt[:, :, :, :n])) and np.all(np.isnan(kt[:, :, :, n:]))
    for l in range(L):
        for h in range(H):
            qr = oracle.rope_apply(q[l, 0, h], qpos, st["cs"], half=bool(flags & oracle.ROPE_HALF))
            qhat = st["pi"][l, h].astype(np.float64) @ qr
            logits = SCALE * (kt[l, 0, h, :n] @ qhat)
            w = np.exp(logits - logits.max())
            oh = (w[:, None] * vt[l, 0, h, :n]).sum(0) / w.sum()
            out = st["pi"][l, h].astype(np.float64).T @ oh if flags & oracle.V_ROTATE else oh
            np.testing.assert_allclose(out, ref[l, 0, h], rtol=0, atol=1e-10)


def test_table_term_has_the_lloyd_max_distortion():
    # Per-element form with ebar = 0 leaves k~ = (n/8) c[idx]: for Gaussian
    # keys the relative error is the 3-bit Lloyd-Max distortion.
    g = synth.rng(32)
    n = 4096
    k = g.standard_normal((1, 1, n, 1, 64)).astype(np.float32)
    st = build(g, n, 1, 1, flags=oracle.QJL_PAPER | oracle.V_ROTATE, k=k, positions=n + 8)
    kt, _ = oracle.dequantize(st["cache"], oracle.QJL_PAPER | oracle.V_ROTATE, [0], [n], n,
                              st["luts"], st["luts"], st["S"], ebar=np.zeros((1, 1, 2), np.float32))
    P = st["pi"][0, 0].astype(np.float64)
    xh = np.stack([P @ exact_rope(k[0, 0, j, 0], j) for j in range(n)])
    rel = np.mean((kt[0, 0, 0, :n] - xh) ** 2) / np.mean(xh ** 2)
    assert abs(rel - LLOYD_MAX_3BIT_MSE) < 0.004, rel


def test_hand_built_slot():
    # One slot written by hand: indices i % 8, key signs alternate, n_k = 8,
    # g_k = 1 (exact in fp16); value nibble 5 everywhere with n_v = 16.
    g = synth.rng(33)
    S = g.standard_normal((64, 64)).astype(np.float32)
    lut = LUT32
    cache = oracle.Cache(1, 1, 64)
    kn = np.array([(i % 8) | ((i % 2) << 3) for i in range(64)], np.uint8)
    vn = np.full(64, 5, np.uint8)
    oracle.pack_slot(cache.region("k", 0, 0), 3, kn, "k")
    oracle.pack_slot(cache.region("v", 0, 0), 3, vn, "v")
    cache.scalars(0, 0)[3] = np.array([8.0, 1.0, 16.0, 0.0], np.float16).view(np.uint16)
    kt, vt = oracle.dequantize(cache, oracle.V_ROTATE, [0], [4], 4, lut[None, None], lut[None, None], S)
    s = np.where(np.arange(64) % 2 == 1, 1.0, -1.0)
    alpha = np.sqrt(np.pi / 2) / 64
    want_k = lut[np.arange(64) % 8].astype(np.float64) + alpha * (S.astype(np.float64).T @ s)
    np.testing.assert_allclose(kt[0, 0, 0, 3], want_k, rtol=0, atol=1e-12)
    np.testing.assert_allclose(vt[0, 0, 0, 3], 2.0 * float(lut[5]), rtol=0, atol=1e-12)
