"""GPU dequantize (the first step of the dequantize-then-attend baseline)
against the oracle's dequantize, through the C ABI: the GPU dequantizes an
upload of the cache the oracle's quantizer wrote, and every fp16 row element
must be the fp16 rounding of the oracle's fp64 value to within one fp16 ulp
plus the fp32 error of its terms: the GPU sums the 64 terms of the residual
estimate in fp32 (at most 63 u of their absolute sum, u = 2^-24) and scales
in fp32, so an element that nearly cancels (c + coef e close to 0) carries
an absolute error up to 2^-16 (n/8)(max|c| + coef sum_i |S_ic|) (coef
sum_i|S_ic| -> ebar for the per-element form). Rows past a sequence's
length, and the rows of an invalid sequence, are not written. Attention over the GPU rows reproduces the fused
decode to within the bound that the fp16 rounding of the rows implies."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import Case, fp16_ulp, to_gpu
from oracle import oracle

pytestmark = pytest.mark.gpu
SENTINEL = -4096.0  # fp16-exact marker of rows that must stay untouched


def _run(case, oc, flags, slot0, lens, max_len):
    cache = to_gpu(oc)
    shape = (case.nl, len(lens), case.H, max_len, 64)
    ko = torch.full(shape, SENTINEL, dtype=torch.float16, device="cuda")
    vo = torch.full(shape, SENTINEL, dtype=torch.float16, device="cuda")
    p = case.params(flags)
    tq.dequantize(p, cache, torch.tensor(slot0, dtype=torch.int64).cuda(),
                  torch.tensor(lens, dtype=torch.int32).cuda(), max_len, case.t("lut_k"), case.t("lut_v"),
                  case.t("S"), case.t("ebar"), layer0=case.layer0, nlayers=case.nl, k_out=ko, v_out=vo)
    torch.cuda.synchronize()
    rk, rv = oracle.dequantize(oc, flags, slot0, lens, max_len, case.lut_k, case.lut_v, case.S,
                               ebar=case.ebar, layer0=case.layer0, nl=case.nl)
    return ko.cpu().numpy().astype(np.float64), vo.cpu().numpy().astype(np.float64), rk, rv


ALPHA = np.sqrt(np.pi / 2) / 64


def _term_scale(case, oc, flags, slot0, lens, max_len, which):
    """(n/8)(max|c| + coef sum_i |S_ic|) per row element, the scale of the
    fp32 error of a dequantized element ([nl][B][H][max_len][64])."""
    col = np.abs(case.S.astype(np.float64)).sum(0)
    out = np.zeros((case.nl, len(lens), case.H, max_len, 64))
    qjl = which == "k" or (flags & tq.V_QJL)
    for li in range(case.nl):
        l = case.layer0 + li
        for h in range(case.H):
            lut = (case.lut_k if which == "k" else case.lut_v)[l, h].astype(np.float64)
            sc = oc.scalars(l, h).view(np.float16).astype(np.float64)
            for b, n in enumerate(lens):
                if n <= 0:
                    continue
                rows = sc[slot0[b]:slot0[b] + n]
                nrm, g = (rows[:, 0], rows[:, 1]) if which == "k" else (rows[:, 2], rows[:, 3])
                if not qjl:
                    e = np.zeros((n, 64))
                elif flags & tq.QJL_PAPER:
                    e = np.full((n, 64), float(case.ebar[l, h, 0 if which == "k" else 1]))
                else:
                    e = ALPHA * g[:, None] * col[None, :]
                out[li, b, h, :n] = nrm[:, None] / 8 * (np.abs(lut).max() + e)
    return out


def _check(got, ref, lens, scale):
    for b, n in enumerate(lens):
        g, r = got[:, b], ref[:, b]
        if n > 0:
            r16 = r[:, :, :n].astype(np.float16).astype(np.float64)
            err = np.abs(g[:, :, :n] - r16)
            lim = fp16_ulp(r16) + 2.0 ** -16 * scale[:, b, :, :n]
            assert np.all(err <= lim), (b, (err - lim).max())
        assert np.all(g[:, :, max(n, 0):] == SENTINEL)


@pytest.mark.parametrize("flags", [tq.V_ROTATE, 0, tq.V_ROTATE | tq.V_QJL,
                                   tq.V_ROTATE | tq.QJL_PAPER | tq.V_QJL, tq.V_ROTATE | tq.QJL_PAPER])
def test_dequantize_matches_oracle(flags):
    L, H, B, T = 2, 3, 2, 300
    case = Case(41, L, H, B, T, io="f16", flags=flags, slots=2 * 320, slot0=[0, 320], pos0=[0, 9])
    oc = oracle.Cache(L, H, case.slots)
    case.oracle_quantize(oc)
    lens = [T, 131]        # several tiles with a ragged tail; a 3-token last tile
    max_len = 320
    gk, gv, rk, rv = _run(case, oc, flags, [0, 320], lens, max_len)
    _check(gk, rk, lens, _term_scale(case, oc, flags, [0, 320], lens, max_len, "k"))
    _check(gv, rv, lens, _term_scale(case, oc, flags, [0, 320], lens, max_len, "v"))


def test_dequantize_edge_lengths_and_invalid_sequences():
    L, H, B, T = 1, 2, 6, 64
    slots = 6 * 128
    slot0 = [0, 128, 256, 384, 512, 130]          # the last is misaligned: skipped
    case = Case(42, L, H, B, T, io="f16", slots=slots, slot0=[0, 128, 256, 384, 512, 640])
    oc = oracle.Cache(L, H, slots)
    case.oracle_quantize(oc)
    lens = [1, 0, 64, 63, 65 - 1, 10]
    gk, gv, rk, rv = _run(case, oc, tq.V_ROTATE, slot0, lens, 128)
    valid = lens[:5] + [0]
    _check(gk, rk, valid, _term_scale(case, oc, tq.V_ROTATE, slot0, valid, 128, "k"))
    _check(gv, rv, valid, _term_scale(case, oc, tq.V_ROTATE, slot0, valid, 128, "v"))


def test_attention_over_dequantized_rows_reproduces_the_fused_decode():
    # fp32 softmax attention of q^ = Pi RoPE(q) over the GPU's fp16 rows, then
    # Pi^T, against tq_decode_attend on the same cache. Row rounding moves a
    # logit by at most d_j = scale * sum_i |q^_i| ulp(k~_ji) / 2, which moves a
    # softmax weight by a factor within exp(+-2 max d) and the output by at
    # most (exp(2 max d) - 1) max_j |v~_j| plus the value rounding.
    L, H, T = 2, 4, 700
    case = Case(43, L, H, 1, T, io="f16", slots=768)
    oc = oracle.Cache(L, H, case.slots)
    case.oracle_quantize(oc)
    cache = to_gpu(oc)
    p = case.params(tq.V_ROTATE)
    s0 = torch.zeros(1, dtype=torch.int64, device="cuda")
    sl = torch.tensor([T], dtype=torch.int32, device="cuda")
    ko, vo = tq.dequantize(p, cache, s0, sl, T, case.t("lut_k"), case.t("lut_v"), case.t("S"))
    fused = case.gpu_decode(cache, [T - 1], [0], [T], T, flags=tq.V_ROTATE | tq.OUT_FP32)
    torch.cuda.synchronize()
    kf, vf = ko.float().cpu().numpy()[:, 0], vo.float().cpu().numpy()[:, 0]
    out = fused.cpu().numpy()[:, 0]
    for l in range(L):
        for h in range(H):
            qr = oracle.rope_apply(case.q[l, 0, h].astype(np.float32), T - 1, case.cs_host)
            P = case.pi[l, h].astype(np.float64)
            qh = P @ qr
            kk, vv = kf[l, h].astype(np.float64), vf[l, h].astype(np.float64)
            logits = 0.125 * (kk @ qh)
            w = np.exp(logits - logits.max())
            o = P.T @ ((w[:, None] * vv).sum(0) / w.sum())
            d = 0.125 * np.abs(qh) @ (fp16_ulp(kk).T / 2)
            bound = (np.exp(2 * d.max()) - 1) * np.abs(vv).max() + fp16_ulp(np.abs(vv).max()) + 2e-3
            assert np.max(np.abs(o - out[l, h])) <= bound, (l, h, np.max(np.abs(o - out[l, h])), bound)
