"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Quantizer: bit-exact codes and fp16 scalars given identical rotated inputs
(TQ_INPUT_ROTATED), on both quantize kernels (T >= 64 one lane per token,
T < 64 one wave per vector), ragged and unaligned slots, every sign mode.
End to end (raw keys/values, GPU RoPE and rotation in binary32): codes may
differ only where the oracle's fp64 coordinate sits within rounding of a
decision threshold.
Decode: the GPU decodes an upload of the cache the oracle's quantizer wrote
and the oracle decodes that cache in fp64 (or, end to end, each side
quantizes the same inputs into a cache of its own), |err| <= 2e-3 (fp32
output), fp16 output within max(2e-3, 1 ulp).
"""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import (Case, GAUSS_LUT, assert_agree_up_to_threshold_rounding, device_bytes, fp16_ulp,
                       to_gpu)
from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu
TOL = 2e-3


def test_library_loaded_and_version():
    assert tq.version().startswith("turboesm-gfx950")
    import os
    maps = open(f"/proc/{os.getpid()}/maps").read()
    assert tq.lib_path in maps


def test_rope_table_matches_oracle():
    # fp64 cos/sin on the GPU and in libm may differ in the last fp64 bits;
    # after rounding to fp32 the tables agree to one fp32 ulp, except next to
    # zeros of sin/cos, where the absolute difference stays at fp64 noise.
    cs = tq.rope_table(8256).cpu().numpy()
    ref = oracle.rope_table(8256)
    ia = cs.view(np.int32).astype(np.int64)
    ib = ref.view(np.int32).astype(np.int64)
    same_sign = np.sign(cs) == np.sign(ref)
    ulps = np.where(same_sign, np.abs(ia - ib), np.abs(ia) + np.abs(ib))
    absdiff = np.abs(cs.astype(np.float64) - ref.astype(np.float64))
    assert np.all((ulps <= 1) | (absdiff <= 1e-10))
    assert np.mean(cs == ref) > 0.999


# ------------------------------------------------------------------ quantizer
def _rotated_inputs(seed, L, B, T, H):
    g = synth.rng(seed)
    scale = g.uniform(0.05, 40.0, (L, B, T, H, 1)).astype(np.float32)
    kh = (g.standard_normal((L, B, T, H, 64)) * scale).astype(np.float32)
    vh = (g.standard_t(4, (L, B, T, H, 64)) * scale).astype(np.float32)
    # special vectors: zero, constant, huge norm, coordinates on a threshold
    kh[0, 0, 0, 0] = 0.0
    kh[0, 0, min(1, T - 1), 0] = 0.75
    vh[0, 0, min(2, T - 1), 0] = 30000.0
    return kh, vh


@pytest.mark.parametrize("T,B,slot0,flags", [
    (256, 1, [0], tq.V_ROTATE),                       # whole tiles, tile kernel
    (200, 2, [64, 640], tq.V_ROTATE),                 # ragged tail
    (130, 2, [37, 300], tq.V_ROTATE),                 # unaligned slots
    (96, 1, [5], tq.V_QJL | tq.V_ROTATE),             # V sign bits
    (70, 1, [0], tq.QJL_PAPER),                       # per-element signs
    (70, 1, [3], tq.QJL_PAPER | tq.V_QJL),
    (1, 3, [0, 100, 1027], tq.V_ROTATE),              # appends: wave kernel
    (5, 2, [61, 200], tq.V_QJL | tq.V_ROTATE),
    (33, 1, [7], tq.QJL_PAPER | tq.V_QJL),
])
def test_quantize_bit_exact_on_rotated_inputs(T, B, slot0, flags):
    L, H = 2, 3
    flags |= tq.INPUT_ROTATED
    case = Case(11, L, H, B, T, io="f32", flags=flags, slots=1152, slot0=slot0, layer0=1, nl=1)
    kh, vh = _rotated_inputs(T * 7 + B, 1, B, T, H)
    cache = tq.Cache(L, H, 1152)
    case.gpu_quantize(cache, k=torch.from_numpy(kh).cuda(), v=torch.from_numpy(vh).cuda())
    torch.cuda.synchronize()
    oc = oracle.Cache(L, H, 1152)
    case.oracle_quantize(oc, k=kh, v=vh)
    got = device_bytes(cache)
    np.testing.assert_array_equal(got.s, oc.s)
    np.testing.assert_array_equal(got.k, oc.k)
    np.testing.assert_array_equal(got.v, oc.v)
    assert oc.s.any()


@pytest.mark.parametrize("T,flags", [
    (128, tq.V_ROTATE),                 # tile kernel
    (128, tq.QJL_PAPER | tq.V_QJL),
    (16, tq.V_ROTATE | tq.V_QJL),       # wave-per-vector kernel
])
def test_quantize_bit_exact_at_thresholds(T, flags):
    """Coordinates exactly on the decision thresholds. The levels are the
    half-integers -3.5 .. 3.5, so the thresholds are the integers -3 .. 3;
    each vector holds the values 0, +-1, +-2, +-3 with squares summing to
    64, times a power of two, so its norm is exactly 8 times that power and u
    equals the unscaled vector exactly. The index counts the thresholds
    strictly below u (Eq. 5 with ties to the lower level), so every such
    coordinate must land on the lower level, on both kernels."""
    L, H, B = 1, 2, 1
    lut = np.arange(-3.5, 4.0, 1.0, dtype=np.float32)
    case = Case(13, L, H, B, T, io="f32", flags=flags | tq.INPUT_ROTATED, slots=256, slot0=[64],
                lut_k=lut, lut_v=lut)
    g = np.random.default_rng(5)
    base = np.array([3, -3, 2, -2, 1, -1, 3, -3, 3, -3] + [0] * 54, np.float32)
    assert float(np.sum(base.astype(np.float64) ** 2)) == 64.0

    def vectors():
        out = np.empty((L, B, T, H, 64), np.float32)
        for idx in np.ndindex(L, B, T, H):
            sgn = np.where(g.random(64) < 0.5, -1.0, 1.0).astype(np.float32)
            out[idx] = g.permutation(base) * sgn * np.float32(2.0 ** int(g.integers(-4, 5)))
        return out

    kh, vh = vectors(), vectors()
    cache = tq.Cache(L, H, 256)
    case.gpu_quantize(cache, k=torch.from_numpy(kh).cuda(), v=torch.from_numpy(vh).cuda())
    torch.cuda.synchronize()
    oc = oracle.Cache(L, H, 256)
    case.oracle_quantize(oc, k=kh, v=vh)
    got = device_bytes(cache)
    np.testing.assert_array_equal(got.s, oc.s)
    np.testing.assert_array_equal(got.k, oc.k)
    np.testing.assert_array_equal(got.v, oc.v)
    assert oc.k.any() and oc.v.any()


@pytest.mark.parametrize("flags", [tq.V_ROTATE, tq.V_ROTATE | tq.V_QJL])
def test_projected_signs_inside_the_guard_band_are_exact(flags):
    # The tile kernel takes a projected sign from its matrix-core product only
    # where |p_i| > 2^-14 ||S_i|| ||r|| and runs the fixed-order chain
    # elsewhere. Rows of S built to land in that band: a zero row (p = 0,
    # sign +1), a row of tiny entries, rows with one nonzero entry (exact
    # products), and a row that cancels to a few ulps for most residuals.
    L, H, B, T = 2, 3, 1, 256
    flags |= tq.INPUT_ROTATED
    case = Case(14, L, H, B, T, io="f32", flags=flags, slots=256, slot0=[0], layer0=1, nl=1)
    g = synth.rng(15)
    S = g.standard_normal((64, 64)).astype(np.float32)
    S[0] = 0.0
    S[1] *= np.float32(2.0 ** -60)
    S[2] = 0.0
    S[2, 5] = 1.0
    S[3] = 0.0
    S[3, 9] = -3.0
    S[4] = np.float32(1.0) + (np.arange(64) % 2).astype(np.float32) * np.float32(2.0 ** -22)
    S[4, 32:] *= -1.0
    case.S = S
    kh, vh = _rotated_inputs(41, 1, B, T, H)
    cache = tq.Cache(L, H, 256)
    case.gpu_quantize(cache, k=torch.from_numpy(kh).cuda(), v=torch.from_numpy(vh).cuda())
    torch.cuda.synchronize()
    oc = oracle.Cache(L, H, 256)
    case.oracle_quantize(oc, k=kh, v=vh)
    got = device_bytes(cache)
    np.testing.assert_array_equal(got.s, oc.s)
    np.testing.assert_array_equal(got.k, oc.k)
    np.testing.assert_array_equal(got.v, oc.v)


def test_quantize_kernels_agree_on_raw_inputs():
    # The tile kernel (T >= 64, rotations on the matrix cores) and the wave
    # kernel (T < 64, fma chains) sum the rotations in different orders: the
    # codes they write for the same raw tokens agree up to threshold rounding.
    L, H, T = 1, 4, 128
    case = Case(12, L, H, 1, T, io="f16", slots=128)
    a = tq.Cache(L, H, 128)
    case.gpu_quantize(a)
    b = tq.Cache(L, H, 128)
    for j0 in range(0, T, 16):
        sl = slice(j0, j0 + 16)
        case.gpu_quantize(b, k=case.t("k")[:, :, sl].contiguous(), v=case.t("v")[:, :, sl].contiguous(),
                          pos0=[j0], slot0=[j0])
    torch.cuda.synchronize()
    assert_agree_up_to_threshold_rounding(case, device_bytes(a), device_bytes(b), 1, T, H)


@pytest.mark.parametrize("flags", [tq.V_ROTATE, tq.V_ROTATE | tq.ROPE_HALF, 0, tq.V_ROTATE | tq.V_QJL])
@pytest.mark.parametrize("T", [256, 3])
def test_quantize_end_to_end_matches_up_to_threshold_rounding(T, flags):
    L, H, B = 1, 8, 2
    case = Case(13, L, H, B, T, io="f16", flags=flags, slots=2 * 320, slot0=[0, 320], pos0=[0, 17])
    cache = tq.Cache(L, H, case.slots)
    case.gpu_quantize(cache)
    torch.cuda.synchronize()
    oc = oracle.Cache(L, H, case.slots)
    case.oracle_quantize(oc)
    assert_agree_up_to_threshold_rounding(case, device_bytes(cache), oc, B, T, H)


# --------------------------------------------------------------------- decode
# Decode parity takes the cache from the oracle's quantizer: the GPU decodes
# an upload of those bytes and the oracle decodes its own cache, so no GPU
# output ever reaches the oracle. test_decode_steps_append_then_attend runs
# both sides end to end instead (each quantizes the same inputs).
def _compare(case, got32, got16, ref):
    got = got32.astype(np.float64)
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got) == np.isfinite(ref))
    fin = np.isfinite(ref)
    assert np.max(err[fin], initial=0.0) <= TOL, np.max(err[fin])
    if got16 is not None:
        g16 = got16.astype(np.float64)
        r16 = ref.astype(np.float16).astype(np.float64)
        lim = np.maximum(TOL, fp16_ulp(r16))
        assert np.all(np.abs(g16 - r16)[fin] <= lim[fin])
    return got


def _decode_check(case, oc, q_pos, seq_slot0, seq_len, max_len, flags=None):
    flags = case.flags if flags is None else flags
    cache = to_gpu(oc)
    out32 = case.gpu_decode(cache, q_pos, seq_slot0, seq_len, max_len, flags=flags | tq.OUT_FP32)
    out16 = case.gpu_decode(cache, q_pos, seq_slot0, seq_len, max_len, flags=flags) if case.io == "f16" else None
    torch.cuda.synchronize()
    ref = case.oracle_decode(oc, q_pos, seq_slot0, seq_len, flags=flags)
    got = _compare(case, out32.cpu().numpy(), None if out16 is None else out16.cpu().numpy(), ref)
    return got, ref, cache


def _oracle_cache(case, L, H):
    oc = oracle.Cache(L, H, case.slots)
    case.oracle_quantize(oc)
    return oc


def test_decode_tiny_fp32_workload():
    # 1 layer, 1 head, 256 cached tokens, fp32 I/O, one query at position 256.
    case = Case(20260, 1, 1, 1, 256, io="f32", slots=320, slot0=[0])
    _decode_check(case, _oracle_cache(case, 1, 1), [256], [0], [256], 256)


@pytest.mark.parametrize("flags", [tq.V_ROTATE, 0, tq.V_ROTATE | tq.V_QJL, tq.QJL_PAPER,
                                   tq.QJL_PAPER | tq.V_QJL | tq.V_ROTATE,
                                   tq.ROPE_HALF | tq.V_ROTATE])
def test_decode_flags(flags):
    case = Case(21, 2, 4, 2, 300, io="f16", flags=flags, slots=2 * 384, slot0=[0, 384])
    _decode_check(case, _oracle_cache(case, 2, 4), [300, 310], [0, 384], [300, 257], 320)


@pytest.mark.parametrize("flags", [tq.V_ROTATE | tq.V_QJL, tq.QJL_PAPER | tq.V_QJL | tq.V_ROTATE, 0])
def test_decode_flags_split_k(flags):
    # max_len 2112 plans splits of 7 tiles for these 16 units; 1100 and 700
    # tokens span 3 and 2 of them, so the partials (with the V sign sums of
    # TQ_V_QJL) go through the workspace merge
    case = Case(24, 2, 4, 2, 1100, io="f16", flags=flags, slots=2 * 2112, slot0=[0, 2112])
    _decode_check(case, _oracle_cache(case, 2, 4), [1100, 1110], [0, 2112], [1100, 700], 2112)


@pytest.mark.parametrize("flags", [tq.V_ROTATE | tq.V_QJL, tq.QJL_PAPER | tq.V_QJL | tq.V_ROTATE, tq.V_ROTATE])
def test_decode_16_wave_blocks(flags):
    # Few units leave compute units free, so the plan takes 16-wave blocks:
    # 16 units of up to 1025 tokens, one block each (one tile per wave) ...
    case = Case(25, 2, 4, 2, 1025, io="f16", flags=flags, slots=2 * 1088, slot0=[0, 1088])
    _decode_check(case, _oracle_cache(case, 2, 4), [1025, 1030], [0, 1088], [1025, 700], 1025)
    # ... and 20 units with max_len 8193, split 17 tiles per block: 3000
    # tokens span three blocks, merged through the workspace
    case = Case(26, 1, 20, 1, 3000, io="f16", flags=flags, slots=8256, slot0=[0], positions=4096)
    _decode_check(case, _oracle_cache(case, 1, 20), [3000], [0], [3000], 8193)


@pytest.mark.parametrize("lens", [[1], [63], [64], [65], [0], [1024], [1025]])
def test_decode_lengths(lens):
    n = max(lens)
    case = Case(22, 1, 3, len(lens), max(n, 1), io="f16", slots=1088)
    got, ref, _ = _decode_check(case, _oracle_cache(case, 1, 3), [n], [0], lens, max(n, 1))
    if lens[0] == 0:
        assert np.all(got == 0)


def test_decode_ragged_batch_and_split_k():
    # lengths spread over [1, 1100]; max_len drives the split count
    g = synth.rng(23)
    B = 12
    lens = g.integers(1, 1100, B).astype(np.int32)
    offs, slots = synth.tile_aligned_offsets(lens)
    case = Case(23, 1, 5, B, int(lens.max()), io="f16", slots=slots, slot0=offs)
    oc = oracle.Cache(1, 5, slots)
    # each sequence's own tokens into its own range
    for b in range(B):
        n = int(lens[b])
        case.oracle_quantize(oc, k=case.k[:, b:b + 1, :n], v=case.v[:, b:b + 1, :n], pos0=[0],
                             slot0=[int(offs[b])])
    qpos = lens.copy()
    _, _, cache = _decode_check(case, oc, qpos, offs, lens, int(lens.max()))
    # a larger max_len bound (more splits) gives the same answer within rounding
    out_a = case.gpu_decode(cache, qpos, offs, lens, int(lens.max()), flags=case.flags | tq.OUT_FP32)
    out_b = case.gpu_decode(cache, qpos, offs, lens, int(slots), flags=case.flags | tq.OUT_FP32)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(out_a - out_b)).item() < 1e-5


def test_decode_invalid_sequences_give_nan():
    case = Case(24, 1, 2, 3, 64, io="f16", slots=256, slot0=[0, 64, 128])
    cache = tq.Cache(1, 2, 256)
    case.gpu_quantize(cache)
    # misaligned start, query position outside the table, length above max_len
    out = case.gpu_decode(cache, [64, 10 ** 6, 64], [1, 64, 128], [10, 10, 70], 64,
                          flags=case.flags | tq.OUT_FP32)
    o = out.cpu().numpy()
    assert np.all(np.isnan(o[:, 0])) and np.all(np.isnan(o[:, 1])) and np.all(np.isnan(o[:, 2]))


def test_decode_is_deterministic():
    case = Case(25, 2, 4, 1, 900, io="f16", slots=960)
    cache = tq.Cache(2, 4, 960)
    case.gpu_quantize(cache)
    a = case.gpu_decode(cache, [900], [0], [900], 900)
    b = case.gpu_decode(cache, [900], [0], [900], 900)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_decode_steps_append_then_attend():
    # one layer of 20 heads: prefill 1024 tokens, then 8 steps of
    # (quantize the new token at position len, attend over len + 1 tokens),
    # end to end on both sides: the GPU quantizes and attends on its cache,
    # the oracle on its own
    L, H, T, steps = 1, 20, 1024, 8
    case = Case(20261, L, H, 1, T + steps, io="f16", slots=1088, slot0=[0])
    cache = tq.Cache(L, H, 1088)
    oc = oracle.Cache(L, H, 1088)
    case.gpu_quantize(cache, k=case.t("k")[:, :, :T].contiguous(), v=case.t("v")[:, :, :T].contiguous())
    case.oracle_quantize(oc, k=case.k[:, :, :T], v=case.v[:, :, :T])
    for s in range(steps):
        n = T + s
        case.gpu_quantize(cache, k=case.t("k")[:, :, n:n + 1].contiguous(),
                          v=case.t("v")[:, :, n:n + 1].contiguous(), pos0=[n], slot0=[n])
        case.oracle_quantize(oc, k=case.k[:, :, n:n + 1], v=case.v[:, :, n:n + 1], pos0=[n], slot0=[n])
        out32 = case.gpu_decode(cache, [n], [0], [n + 1], 1088, flags=case.flags | tq.OUT_FP32)
        out16 = case.gpu_decode(cache, [n], [0], [n + 1], 1088)
        torch.cuda.synchronize()
        ref = case.oracle_decode(oc, [n], [0], [n + 1])
        _compare(case, out32.cpu().numpy(), out16.cpu().numpy(), ref)


# ---------------------------------------------------------------- calibration
def test_calibrate_rotation_matches_svd():
    g = synth.rng(30)
    nh, ncal = 6, 4096
    cs = oracle.rope_table(1024)
    ch = synth.outlier_channels(g, 1, nh)
    keys = synth.keys(g, 1, 1, ncal, nh, ch)[0, 0]          # [ncal][nh][64]
    pos = synth.calibration_positions(g, ncal, 1024)
    X = np.empty((nh, ncal, 64), np.float32)
    for h in range(nh):
        for i in range(ncal):
            X[h, i] = oracle.rope_apply(keys[i, h], int(pos[i]), cs)
    pi, sg = tq.calibrate_rotation(torch.from_numpy(X).cuda())
    pi = pi.cpu().numpy().astype(np.float64)
    sg = sg.cpu().numpy().astype(np.float64)
    for h in range(nh):
        P = pi[h]
        ref_pi, ref_s = oracle.calibrate_rotation(X[h])
        np.testing.assert_allclose(sg[h], ref_s, rtol=1e-5)
        np.testing.assert_allclose(P @ P.T, np.eye(64), atol=1e-6)
        G = X[h].astype(np.float64).T @ X[h].astype(np.float64)
        Dg = P @ G @ P.T
        assert np.max(np.abs(Dg - np.diag(np.diag(Dg)))) <= 1e-5 * ref_s[0] ** 2
        # rows with a well separated singular value match the oracle's row
        gap = np.minimum(np.abs(np.diff(np.concatenate(([np.inf], ref_s)))),
                         np.abs(np.diff(np.concatenate((ref_s, [-np.inf])))))
        sep = gap > 1e-3 * ref_s[0]
        np.testing.assert_allclose(P[sep], ref_pi[sep].astype(np.float64), atol=1e-4)


# ---------------------------------------------------------- table calibration
@pytest.mark.parametrize("kind,rotate", [("k", True), ("v", True), ("v", False)])
def test_calibrate_lut_matches_oracle(kind, rotate):
    g = synth.rng(41)
    H, ncal = 3, 1024
    ch = synth.outlier_channels(g, 1, H)
    if kind == "k":
        x = synth.keys(g, 1, 1, ncal, H, ch)[0, 0].transpose(1, 0, 2).copy()      # [H][ncal][64]
    else:
        x = synth.values(g, 1, 1, ncal, H)[0, 0].transpose(1, 0, 2).copy()
    x[0, 5] = 0.0                                                               # a zero vector
    pi = synth.rotations(g, 1, H)[0]
    init = GAUSS_LUT
    got = tq.calibrate_lut(torch.from_numpy(x).cuda(), torch.from_numpy(pi).cuda() if rotate else None,
                           init).cpu().numpy()
    for h in range(H):
        ref = oracle.calibrate_lut(x[h], pi[h] if rotate else None, init)
        np.testing.assert_allclose(got[h], ref, rtol=0, atol=2e-6)
        assert np.all(np.diff(got[h]) > 0)


def test_calibrate_lut_keeps_empty_cells_and_stops_at_max_iter():
    g = synth.rng(42)
    x = g.standard_normal((2, 256, 64)).astype(np.float32)
    init = np.array([-40.0, -1.3, -0.75, -0.25, 0.25, 0.75, 1.3, 40.0], np.float32)   # outer cells stay empty
    got = tq.calibrate_lut(torch.from_numpy(x).cuda(), None, init, max_iter=3).cpu().numpy()
    for h in range(2):
        ref = oracle.calibrate_lut(x[h], None, init, max_iter=3)
        np.testing.assert_allclose(got[h], ref, rtol=0, atol=2e-6)
        assert got[h][0] == -40.0 and got[h][-1] == 40.0
