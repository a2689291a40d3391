"""tq_quantize_pack_ragged: one call for sequences of different lengths gives
every token the bytes that a call per sequence gives it (Sec. 3.1 prefill
steps 1, 3, 4), and writes nothing for the padding rows."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import Case

pytestmark = pytest.mark.gpu


def _cache_bytes(c):
    torch.cuda.synchronize()
    return c.k_codes.cpu().numpy(), c.v_codes.cpu().numpy(), c.scalars.cpu().numpy()


@pytest.mark.parametrize("T,lens,flags", [
    (300, [300, 70, 129, 0], tq.V_ROTATE),          # the tile kernel (every length >= 64 or 0)
    (300, [64, 257, 0, 128], tq.V_ROTATE | tq.V_QJL | tq.ROPE_HALF),
    (40, [40, 7, 0, 33], tq.V_ROTATE),              # the per-vector kernel (T < 64)
])
def test_ragged_pack_equals_one_call_per_sequence(T, lens, flags):
    B, H = len(lens), 4
    cap = ((T + 63) // 64) * 64
    slot0 = [b * cap for b in range(B)]
    pos0 = [3 * b for b in range(B)]
    case = Case(61, 1, H, B, T, io="f16", flags=flags, slots=B * cap, slot0=slot0, pos0=pos0)
    k = case.t("k").clone()
    v = case.t("v").clone()
    for b, n in enumerate(lens):            # padding rows hold NaN: they must not be read
        k[:, b, n:] = float("nan")
        v[:, b, n:] = float("nan")
    p = case.params()
    tokens = torch.tensor(lens, dtype=torch.int32, device="cuda")
    ragged = tq.Cache(1, H, B * cap)
    tq.quantize_pack(p, ragged, k, v, case.t("pos0"), case.t("slot0"), case.t("pi"), case.t("lut_k"),
                     case.t("lut_v"), case.t("S"), seq_tokens=tokens)
    each = tq.Cache(1, H, B * cap)
    for b, n in enumerate(lens):
        if n == 0:
            continue
        tq.quantize_pack(p, each, case.t("k")[:, b:b + 1, :n].contiguous(), case.t("v")[:, b:b + 1, :n].contiguous(),
                         torch.tensor([pos0[b]], dtype=torch.int32, device="cuda"),
                         torch.tensor([slot0[b]], dtype=torch.int64, device="cuda"),
                         case.t("pi"), case.t("lut_k"), case.t("lut_v"), case.t("S"))
    for got, ref in zip(_cache_bytes(ragged), _cache_bytes(each)):
        np.testing.assert_array_equal(got, ref)
    # a sequence of 0 tokens, and the slots past each sequence, are untouched
    kc = ragged.k_codes.view(1, H, B * cap * 32).cpu().numpy()
    for b, n in enumerate(lens):
        first_unused_tile = (n + 63) // 64
        lo = (slot0[b] + first_unused_tile * 64) * 32
        assert not np.any(kc[:, :, lo:(slot0[b] + cap) * 32])


def test_ragged_pack_clamps_counts_to_T():
    T, H = 128, 2
    lens = [500, -3]                         # read as T and 0
    case = Case(62, 1, H, 2, T, io="f16", slots=2 * T, slot0=[0, T])
    p = case.params()
    ragged = tq.Cache(1, H, 2 * T)
    tq.quantize_pack(p, ragged, case.t("k"), case.t("v"), case.t("pos0"), case.t("slot0"), case.t("pi"),
                     case.t("lut_k"), case.t("lut_v"), case.t("S"),
                     seq_tokens=torch.tensor(lens, dtype=torch.int32, device="cuda"))
    full = tq.Cache(1, H, 2 * T)
    tq.quantize_pack(p, full, case.t("k")[:, :1].contiguous(), case.t("v")[:, :1].contiguous(),
                     case.t("pos0")[:1], case.t("slot0")[:1], case.t("pi"), case.t("lut_k"), case.t("lut_v"),
                     case.t("S"))
    for got, ref in zip(_cache_bytes(ragged), _cache_bytes(full)):
        np.testing.assert_array_equal(got, ref)
