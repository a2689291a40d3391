"""Failure handling at the boundary, on the GPU, through the C ABI:
device tables that are not strictly ascending (quantize does not write the
(layer, head), dequantize skips it, decode writes NaN), a decode step whose
bounded wait for its appends gives up (forced from the host with a wait limit
of 0: the unit's output is NaN, every kernel still exits normally), and one
split-K workspace reused across calls of different shapes (every completed
call leaves it zero). Also the ebar calibration against the oracle."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import Case, GAUSS_LUT, to_gpu
from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu


def _i32(x):
    return torch.tensor(np.asarray(x, np.int32), dtype=torch.int32).cuda()


def _i64(x):
    return torch.tensor(np.asarray(x, np.int64), dtype=torch.int64).cuda()


def _bad_tables(case, head_k, head_v):
    """lut_k with two levels of head_k swapped, lut_v with a NaN level at head_v."""
    lk, lv = case.lut_k.copy(), case.lut_v.copy()
    lk[0, head_k, [2, 3]] = lk[0, head_k, [3, 2]]
    lv[0, head_v, 5] = np.nan
    return torch.from_numpy(lk).cuda(), torch.from_numpy(lv).cuda()


@pytest.mark.parametrize("T", [200, 5])        # tile kernel, wave-per-vector kernel
def test_quantize_skips_heads_with_bad_tables(T):
    case = Case(51, 1, 4, 1, T, io="f16", slots=256)
    good = tq.Cache(1, 4, 256)
    case.gpu_quantize(good)
    lk, lv = _bad_tables(case, 1, 2)
    bad = tq.Cache(1, 4, 256)
    p = case.params()
    tq.quantize_pack(p, bad, case.t("k"), case.t("v"), case.t("pos0"), case.t("slot0"), case.t("pi"), lk, lv,
                     case.t("S"))
    torch.cuda.synchronize()
    n = 256 * 32
    for h in range(4):
        for plane in ("k_codes", "v_codes"):
            g, b = getattr(good, plane)[h * n:(h + 1) * n], getattr(bad, plane)[h * n:(h + 1) * n]
            if h in (1, 2):
                assert int(b.abs().sum()) == 0, (h, plane)      # never written
            else:
                assert torch.equal(g, b), (h, plane)
        sg, sb = good.scalars[h * 1024:(h + 1) * 1024], bad.scalars[h * 1024:(h + 1) * 1024]
        assert torch.equal(sg, sb) if h in (0, 3) else int(sb.abs().sum()) == 0


def test_decode_and_dequantize_with_bad_tables():
    case = Case(52, 1, 4, 2, 300, io="f16", slots=768, slot0=[0, 384])
    oc = oracle.Cache(1, 4, 768)
    case.oracle_quantize(oc)
    cache = to_gpu(oc)
    lk, lv = _bad_tables(case, 1, 2)
    p = case.params(case.flags | tq.OUT_FP32)
    args = (_i32([300, 300]), _i64([0, 384]), _i32([300, 250]), 300)
    good = tq.decode_attend(p, cache, case.t("q"), *args, case.t("pi"), case.t("lut_k"), case.t("lut_v"),
                            case.t("S")).cpu().numpy()
    bad = tq.decode_attend(p, cache, case.t("q"), *args, case.t("pi"), lk, lv, case.t("S")).cpu().numpy()
    assert np.all(np.isfinite(good))
    assert np.all(np.isnan(bad[:, :, 1])) and np.all(np.isnan(bad[:, :, 2]))
    assert np.array_equal(bad[:, :, 0], good[:, :, 0]) and np.array_equal(bad[:, :, 3], good[:, :, 3])
    # the step entry point: the unit is neither appended to nor finite
    k = case.t("k")[:, :, 250].contiguous()
    v = case.t("v")[:, :, 250].contiguous()
    before = (cache.k_codes.clone(), cache.v_codes.clone(), cache.scalars.clone())
    out = tq.decode_step(p, cache, case.t("q"), k, v, _i32([250, 250]), _i64([0, 384]), _i32([250, 250]), 300,
                         case.t("pi"), lk, lv, case.t("S")).cpu().numpy()
    assert np.all(np.isnan(out[:, :, 1])) and np.all(np.isnan(out[:, :, 2]))
    assert np.all(np.isfinite(out[:, :, 0])) and np.all(np.isfinite(out[:, :, 3]))
    n = 768 * 32
    for h in (1, 2):
        assert torch.equal(cache.k_codes[h * n:(h + 1) * n], before[0][h * n:(h + 1) * n])
        assert torch.equal(cache.v_codes[h * n:(h + 1) * n], before[1][h * n:(h + 1) * n])
    # dequantize skips the two heads (rows keep the fill value)
    ko = torch.full((1, 2, 4, 300, 64), 7.0, dtype=torch.float16, device="cuda")
    vo = torch.full((1, 2, 4, 300, 64), 7.0, dtype=torch.float16, device="cuda")
    tq.dequantize(case.params(), cache, _i64([0, 384]), _i32([250, 250]), 300, lk, lv, case.t("S"),
                  k_out=ko, v_out=vo)
    torch.cuda.synchronize()
    assert bool(torch.all(ko[:, :, 1:3] == 7.0)) and bool(torch.all(vo[:, :, 1:3] == 7.0))
    assert not bool(torch.all(ko[:, :, 0, :250] == 7.0))


@pytest.mark.parametrize("lens", [[100, 40], [3000, 40]])   # one block per unit; a split sequence
def test_step_wait_that_gives_up_marks_the_output(lens):
    lens = np.array(lens, np.int32)
    offs, slots = synth.tile_aligned_offsets(lens + 1)
    case = Case(53, 1, 2, 2, int(lens.max()) + 1, io="f16", slots=slots, slot0=offs, positions=4096)
    base = tq.Cache(1, 2, slots)
    for b in range(2):
        case.gpu_quantize(base, k=case.t("k")[:, b:b + 1, :int(lens[b])].contiguous(),
                          v=case.t("v")[:, b:b + 1, :int(lens[b])].contiguous(), pos0=[0], slot0=[int(offs[b])])
    k = torch.stack([case.t("k")[:, b, int(lens[b])] for b in range(2)], 1).contiguous()
    v = torch.stack([case.t("v")[:, b, int(lens[b])] for b in range(2)], 1).contiguous()
    p = case.params(case.flags | tq.OUT_FP32)

    def step(cache):
        return tq.decode_step(p, cache, case.t("q"), k, v, _i32(lens), _i64(offs), _i32(lens), slots,
                              case.t("pi"), case.t("lut_k"), case.t("lut_v"), case.t("S"))

    ok_cache = tq.Cache(1, 2, slots)
    ok_cache.k_codes.copy_(base.k_codes); ok_cache.v_codes.copy_(base.v_codes); ok_cache.scalars.copy_(base.scalars)
    ok = step(ok_cache)
    torch.cuda.synchronize()
    prev = tq.set_step_wait_limit(0)
    try:
        failed = step(base)
        torch.cuda.synchronize()
    finally:
        tq.set_step_wait_limit(prev)
    assert torch.all(torch.isfinite(ok))
    assert torch.all(torch.isnan(failed))
    # the appends themselves completed
    assert torch.equal(base.k_codes, ok_cache.k_codes) and torch.equal(base.v_codes, ok_cache.v_codes)
    assert torch.equal(base.scalars, ok_cache.scalars)
    # and with the default bound restored the same step succeeds again
    again = step(base)
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(again))


def test_one_workspace_serves_calls_of_different_shapes():
    shapes = [
        (1, 2, [3000]),             # 2 units, split over many blocks
        (2, 3, [1500, 700]),        # 12 units, fewer splits, different partial offsets
        (1, 1, [5000]),
    ]
    cases = []
    for i, (L, H, lens) in enumerate(shapes):
        lens = np.array(lens, np.int32)
        offs, slots = synth.tile_aligned_offsets(lens)
        case = Case(60 + i, L, H, len(lens), int(lens.max()), io="f16", slots=slots, slot0=offs, positions=8192)
        cache = tq.Cache(L, H, slots)
        for b in range(len(lens)):
            case.gpu_quantize(cache, k=case.t("k")[:, b:b + 1, :int(lens[b])].contiguous(),
                              v=case.t("v")[:, b:b + 1, :int(lens[b])].contiguous(), pos0=[0],
                              slot0=[int(offs[b])])
        cases.append((case, cache, lens, offs))
    need = max(tq.decode_workspace_bytes(c.params(), len(lens), c.L, int(lens.max())) for c, _, lens, _ in cases)
    assert need > 0
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")

    def run(i, workspace):
        case, cache, lens, offs = cases[i]
        p = case.params(case.flags | tq.OUT_FP32)
        return tq.decode_attend(p, cache, case.t("q"), _i32(lens), _i64(offs), _i32(lens), int(lens.max()),
                                case.t("pi"), case.t("lut_k"), case.t("lut_v"), case.t("S"), workspace=workspace)

    for i in (0, 1, 2, 0, 2, 1):
        shared = run(i, ws)
        fresh = run(i, None)
        torch.cuda.synchronize()
        assert torch.equal(shared, fresh), i
        assert int(ws.count_nonzero()) == 0, i


# ------------------------------------------------------------------ ebar
def test_calibrate_ebar_matches_oracle():
    g = synth.rng(70)
    H, ncal = 4, 2048
    ch = synth.outlier_channels(g, 1, H)
    xk = synth.keys(g, 1, 1, ncal, H, ch)[0, 0].transpose(1, 0, 2).copy()     # [H][ncal][64]
    xv = synth.values(g, 1, 1, ncal, H)[0, 0].transpose(1, 0, 2).copy()
    xk[1, 3] = 0.0                                                            # a zero vector
    pi = np.stack([oracle.calibrate_rotation(xk[h])[0] for h in range(H)])
    lut_k = np.stack([oracle.calibrate_lut(xk[h], pi[h], GAUSS_LUT) for h in range(H)]).astype(np.float32)
    lut_v = np.stack([oracle.calibrate_lut(xv[h], None, GAUSS_LUT) for h in range(H)]).astype(np.float32)
    lut_v[3, [0, 1]] = lut_v[3, [1, 0]]                                       # not ascending: NaN
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ebar = torch.full((1, H, 2), -1.0, dtype=torch.float32, device="cuda")
    tq.calibrate_ebar(d(xk), d(lut_k), d(pi), out=ebar.view(-1), stride=2)
    tq.calibrate_ebar(d(xv), d(lut_v), None, out=ebar.view(-1)[1:], stride=2)
    alone = tq.calibrate_ebar(d(xk), d(lut_k), d(pi))
    got = ebar.cpu().numpy()
    for h in range(H):
        ref_k = oracle.calibrate_ebar(xk[h], pi[h], lut_k[h])
        assert got[0, h, 0] == pytest.approx(ref_k, rel=1e-6)
        if h < 3:
            assert got[0, h, 1] == pytest.approx(oracle.calibrate_ebar(xv[h], None, lut_v[h]), rel=1e-6)
    assert np.isnan(got[0, 3, 1])
    assert torch.equal(alone.cpu(), ebar[0, :, 0].cpu())
