"""tq_decode_attend_noalloc (the decode entry point that allocates nothing,
for callers that cannot call hipMalloc) against tq_decode_attend, through the
C ABI: identical output on two calls in a row, the second with a smaller
input, both on sizes that need the split-K workspace (the fixed device array
then serves in its place); sizes without a split; and every workspace the
decode planner asks for fits the fixed array (its size check stays as a
guard that no planned size reaches)."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import Case
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu


def _i32(x):
    return torch.tensor(np.asarray(x, np.int32), dtype=torch.int32).cuda()


def _i64(x):
    return torch.tensor(np.asarray(x, np.int64), dtype=torch.int64).cuda()


def _setup(seed, L, H, lens, flags=tq.V_ROTATE):
    lens = np.asarray(lens, np.int32)
    offs, slots = synth.tile_aligned_offsets(lens)
    case = Case(seed, L, H, len(lens), int(lens.max()), io="f16", flags=flags, slots=slots, slot0=offs,
                positions=8192)
    cache = tq.Cache(L, H, slots)
    for b in range(len(lens)):
        case.gpu_quantize(cache, k=case.t("k")[:, b:b + 1, :int(lens[b])].contiguous(),
                          v=case.t("v")[:, b:b + 1, :int(lens[b])].contiguous(), pos0=[0], slot0=[int(offs[b])])
    return case, cache, lens, offs


def _both(case, cache, lens, offs, flags):
    p = case.params(flags)
    args = (case.t("q"), _i32(lens), _i64(offs), _i32(lens), int(lens.max()), case.t("pi"), case.t("lut_k"),
            case.t("lut_v"), case.t("S"), case.t("ebar"))
    ref = tq.decode_attend(p, cache, *args)
    got = tq.decode_attend_noalloc(p, cache, *args)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("flags", [tq.V_ROTATE | tq.OUT_FP32, tq.V_ROTATE | tq.V_QJL])
def test_noalloc_equals_decode_attend_on_two_calls(flags):
    first = _setup(81, 1, 2, [3000, 500], flags)        # 4 units, long sequence split over many blocks
    second = _setup(82, 1, 1, [700], flags)             # 1 unit, fewer splits
    for case, cache, lens, offs in (first, second):
        assert tq.decode_workspace_bytes(case.params(flags), len(lens), case.L, int(lens.max())) > 0
        ref, got = _both(case, cache, lens, offs, flags)
        assert torch.all(torch.isfinite(ref))
        assert torch.equal(ref, got)


def test_noalloc_without_a_split_uses_no_scratch():
    case, cache, lens, offs = _setup(83, 13, 20, [1024])   # 260 units of 16 tiles: one block each, no split
    flags = tq.V_ROTATE
    assert tq.decode_workspace_bytes(case.params(flags), 1, 13, 1024) == 0
    ref, got = _both(case, cache, lens, offs, flags)
    assert torch.equal(ref, got)


def test_noalloc_scratch_holds_every_planned_workspace():
    # The planner splits a unit's tiles only while the blocks of all splits
    # fit one pass over the 256 compute units, so a workspace holds at most
    # 256 partials of 528 bytes (plus counters): always within the 256 KiB
    # fixed array.
    cs = tq.rope_table(64)
    worst = 0
    for H in (1, 2, 20, 40):
        for B in (1, 2, 7, 64):
            for L in (1, 2, 13, 33, 36):
                p = tq.Params(L, H, cs)
                for max_len in (1, 64, 65, 700, 1025, 2049, 3000, 8193, 65536):
                    worst = max(worst, tq.decode_workspace_bytes(p, B, L, max_len))
    assert 0 < worst <= 262144
