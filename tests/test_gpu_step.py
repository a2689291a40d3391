"""tq_decode_step (append the new token, then attend) against the two calls it
fuses, tq_quantize_pack with T = 1 followed by tq_decode_attend: the cache
bytes and the output must be identical, bit for bit, since the step runs the
same quantizer and attention arithmetic. Each step is also checked against
the oracle, which quantizes the same tokens into a cache of its own. Ragged batches, every flag combination, empty caches, split
sequences and invalid sequences are covered."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import Case, assert_agree_up_to_threshold_rounding, device_bytes
from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _i32(x):
    return torch.tensor(np.asarray(x, np.int32), dtype=torch.int32).cuda()


def _i64(x):
    return torch.tensor(np.asarray(x, np.int64), dtype=torch.int64).cuda()


def _clone(cache):
    c = tq.Cache(cache.num_layers, cache.num_heads, cache.slots)
    c.k_codes.copy_(cache.k_codes)
    c.v_codes.copy_(cache.v_codes)
    c.scalars.copy_(cache.scalars)
    return c


def _same_cache(a, b):
    return (torch.equal(a.k_codes, b.k_codes) and torch.equal(a.v_codes, b.v_codes)
            and torch.equal(a.scalars, b.scalars))


def _prefill(case, cache, lens, offs):
    for b in range(case.B):
        n = int(lens[b])
        if n == 0:
            continue
        case.gpu_quantize(cache, k=case.t("k")[:, b:b + 1, :n].contiguous(),
                          v=case.t("v")[:, b:b + 1, :n].contiguous(), pos0=[0], slot0=[int(offs[b])])


def _new_token(case, lens):
    """The token at index lens[b] of each sequence, [nl][B][H][64]."""
    k = torch.stack([case.t("k")[:, b, int(lens[b])] for b in range(case.B)], 1).contiguous()
    v = torch.stack([case.t("v")[:, b, int(lens[b])] for b in range(case.B)], 1).contiguous()
    return k, v


def _two_calls(case, cache, k, v, pos, offs, lens, max_len, flags):
    p = case.params(flags)
    tq.quantize_pack(p, cache, k.unsqueeze(2).contiguous(), v.unsqueeze(2).contiguous(), _i32(pos),
                     _i64(np.asarray(offs) + np.asarray(lens)), case.t("pi"), case.t("lut_k"),
                     case.t("lut_v"), case.t("S"), case.t("ebar"), layer0=case.layer0)
    return tq.decode_attend(p, cache, case.t("q"), _i32(pos), _i64(offs), _i32(np.asarray(lens) + 1),
                            max_len, case.t("pi"), case.t("lut_k"), case.t("lut_v"), case.t("S"),
                            case.t("ebar"), layer0=case.layer0)


def _step(case, cache, k, v, pos, offs, lens, max_len, flags):
    p = case.params(flags)
    return tq.decode_step(p, cache, case.t("q"), k, v, _i32(pos), _i64(offs), _i32(lens), max_len,
                          case.t("pi"), case.t("lut_k"), case.t("lut_v"), case.t("S"), case.t("ebar"),
                          layer0=case.layer0)


@pytest.mark.parametrize("flags,io", [
    (tq.V_ROTATE, "f16"), (0, "f16"), (tq.V_ROTATE | tq.V_QJL, "f16"),
    (tq.QJL_PAPER | tq.V_QJL | tq.V_ROTATE, "f16"), (tq.ROPE_HALF | tq.V_ROTATE, "f16"),
    (tq.V_ROTATE | tq.OUT_FP32, "f16"), (tq.V_ROTATE, "f32"),
])
def test_step_equals_append_then_attend(flags, io):
    # three sequences: an empty cache, a tile minus one token, a ragged length
    lens = np.array([0, 63, 200], np.int32)
    offs, slots = synth.tile_aligned_offsets(lens + 1)
    case = Case(31, 2, 3, 3, int(lens.max()) + 1, io=io, flags=flags, slots=slots, slot0=offs)
    base = tq.Cache(2, 3, slots)
    _prefill(case, base, lens, offs)
    k, v = _new_token(case, lens)
    pos = lens + 5                                   # positions need not equal lengths
    a, b = _clone(base), _clone(base)
    out_a = _two_calls(case, a, k, v, pos, offs, lens, int(lens.max()) + 1, flags)
    out_b = _step(case, b, k, v, pos, offs, lens, int(lens.max()) + 1, flags)
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(out_b))
    assert _same_cache(a, b)
    assert not _same_cache(a, base)
    assert torch.equal(out_a, out_b)


def test_step_equals_append_then_attend_split_sequence():
    # one long sequence split across blocks, plus a short one in the same call
    lens = np.array([3000, 40], np.int32)
    offs, slots = synth.tile_aligned_offsets(lens + 1)
    case = Case(32, 1, 2, 2, int(lens.max()) + 1, io="f16", slots=slots, slot0=offs, positions=4096)
    base = tq.Cache(1, 2, slots)
    _prefill(case, base, lens, offs)
    k, v = _new_token(case, lens)
    a, b = _clone(base), _clone(base)
    out_a = _two_calls(case, a, k, v, lens, offs, lens, slots, case.flags)
    out_b = _step(case, b, k, v, lens, offs, lens, slots, case.flags)
    torch.cuda.synchronize()
    assert _same_cache(a, b)
    assert torch.all(torch.isfinite(out_b))
    assert torch.equal(out_a, out_b)


@pytest.mark.parametrize("flags", [tq.V_ROTATE, tq.V_ROTATE | tq.V_QJL, tq.QJL_PAPER | tq.V_QJL | tq.V_ROTATE])
def test_steps_match_oracle(flags):
    # one layer of 20 heads: prefill 1024 tokens, then 6 decode steps, end to
    # end on both sides: the GPU steps on its cache, the oracle quantizes the
    # same tokens into its own cache and attends there (20 units leave
    # compute units free: 16-wave blocks)
    L, H, T, steps = 1, 20, 1024, 6
    case = Case(20262, L, H, 1, T + steps, io="f16", flags=flags, slots=1088, slot0=[0])
    cache = tq.Cache(L, H, 1088)
    _prefill(case, cache, [T], [0])
    oc = oracle.Cache(L, H, 1088)
    case.oracle_quantize(oc, k=case.k[:, :, :T], v=case.v[:, :, :T])
    flags = case.flags | tq.OUT_FP32
    for s in range(steps):
        n = T + s
        k = case.t("k")[:, :, n].contiguous()
        v = case.t("v")[:, :, n].contiguous()
        out = _step(case, cache, k, v, [n], [0], [n], 1088, flags)
        torch.cuda.synchronize()
        case.oracle_quantize(oc, k=case.k[:, :, n:n + 1], v=case.v[:, :, n:n + 1], pos0=[n], slot0=[n])
        ref = case.oracle_decode(oc, [n], [0], [n + 1])
        err = np.abs(out.cpu().numpy().astype(np.float64) - ref)
        assert np.max(err) <= TOL, (s, np.max(err))
    # the prefill quantizer on all T + steps tokens writes the same bytes for
    # the T prefilled ones, and the appended ones agree with its codes up to
    # threshold rounding (the append rotates with fma chains, the prefill on
    # the matrix cores)
    full = tq.Cache(L, H, 1088)
    case.gpu_quantize(full, k=case.t("k")[:, :, :T + steps].contiguous(),
                      v=case.t("v")[:, :, :T + steps].contiguous())
    torch.cuda.synchronize()
    got, ref = device_bytes(cache), device_bytes(full)
    for h in range(H):
        for which in ("k", "v"):
            assert np.array_equal(got.region(which, 0, h)[:T * 32], ref.region(which, 0, h)[:T * 32])
        assert np.array_equal(got.scalars(0, h)[:T], ref.scalars(0, h)[:T])
    assert_agree_up_to_threshold_rounding(case, got, ref, 1, T + steps, H, tokens=range(T, T + steps))


@pytest.mark.parametrize("T", [1088, 1087, 0])
def test_step_new_token_alone_in_its_split(T):
    # 20 units with max_len 8193 split the tiles 17 per block (0-16, 17-33,
    # ...). With 1088 cached tokens the new token (index 1088) starts tile
    # 17: the second split holds no cached token, only the new one, which its
    # block scores apart from the tiles. With 1087 the new token shares tile
    # 16 with cached ones; with 0 it is the only token.
    L, H, slots = 1, 20, 8256
    case = Case(20263, L, H, 1, T + 1, io="f16", slots=slots, slot0=[0])
    assert tq.decode_workspace_bytes(case.params(), 1, L, 8193) > 0     # the plan splits
    cache = tq.Cache(L, H, slots)
    _prefill(case, cache, [T], [0])
    oc = oracle.Cache(L, H, slots)
    if T:
        case.oracle_quantize(oc, k=case.k[:, :, :T], v=case.v[:, :, :T])
    flags = case.flags | tq.OUT_FP32
    k = case.t("k")[:, :, T].contiguous()
    v = case.t("v")[:, :, T].contiguous()
    two = _clone(cache)
    out = _step(case, cache, k, v, [T], [0], [T], 8193, flags)
    out_two = _two_calls(case, two, k, v, [T], [0], [T], 8193, flags)
    torch.cuda.synchronize()
    assert _same_cache(cache, two)
    assert torch.equal(out, out_two)
    case.oracle_quantize(oc, k=case.k[:, :, T:T + 1], v=case.v[:, :, T:T + 1], pos0=[T], slot0=[T])
    ref = case.oracle_decode(oc, [T], [0], [T + 1])
    err = np.abs(out.cpu().numpy().astype(np.float64) - ref)
    assert np.max(err) <= TOL, np.max(err)


def test_step_invalid_sequences_are_not_appended():
    # over max_len, misaligned start, position outside the RoPE table
    lens = np.array([64, 10, 10], np.int32)
    offs = np.array([0, 129, 256], np.int64)
    case = Case(33, 1, 2, 3, 70, io="f16", slots=384, slot0=[0, 128, 256])
    base = tq.Cache(1, 2, 384)
    _prefill(case, base, lens, [0, 128, 256])
    k, v = _new_token(case, lens)
    c = _clone(base)
    out = _step(case, c, k, v, [64, 10, 10 ** 6], offs, lens, 64, case.flags | tq.OUT_FP32)
    torch.cuda.synchronize()
    assert _same_cache(c, base)
    assert torch.all(torch.isnan(out))
