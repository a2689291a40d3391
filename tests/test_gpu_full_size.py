"""Parity at the full sizes of the workloads, in the launch configuration the
bench times: one tq_decode_step over every layer, sequence and head (the
prologue kernel appends the new token and rotates the query, the attention
kernel reads the whole packed cache).

  ESM-2 650M full cache   33 layers x 20 heads, batch 1, 1024 cached tokens
  ragged batch            33 x 20, 64 sequences of lengths uniform in [50, 1024],
                          tile-aligned packed offsets
  ESM-2 3B shape          36 layers x 40 heads, batch 16, 8192 cached tokens

At the ESM-2 650M shape every unit is compared: the oracle quantizes all the
raw tokens into a cache of its own and decodes every unit there in fp64. At
the ragged and 3B shapes, for a sample of (layer, sequence, head) units the
oracle quantizes that unit's raw tokens (the cached ones and the new one)
into a cache of its own and decodes there in fp64: 2e-3 on the fp32 output and max(2e-3, 1 fp16 ulp)
on the fp16 output. The GPU's codes of sampled tokens, including the appended
one, are checked against the oracle's quantizer of the same inputs: equal, or
one level apart where the rotated coordinate lies within rounding of a
threshold; its norms of every token of a sampled unit within one fp16 ulp of
the oracle's."""
import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import DeviceBytes, GAUSS_LUT, assert_region_agrees, device_bytes, fp16_ulp, unpack_slot
from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu
TOL = 2e-3
# a second, distinct ascending table for the values (separate K and V tables)
V_LUT = (GAUSS_LUT * np.float32(1.07) + np.float32(0.01)).astype(np.float32)


def _i32(x):
    return torch.tensor(np.asarray(x, np.int32), dtype=torch.int32).cuda()


def _i64(x):
    return torch.tensor(np.asarray(x, np.int64), dtype=torch.int64).cuda()


def _gpu_region(cache, l, h, s0, n):
    """The GPU's bytes of slots [s0, s0 + cap) of one (layer, head) region as
    a one-head layout, cap = n rounded up to a tile (s0 is tile-aligned, so
    tile layouts are unchanged by the shift). Compared with the oracle's
    bytes, never given to the oracle."""
    cap = (n + 63) // 64 * 64
    base = (l * cache.num_heads + h) * cache.slots + s0
    return DeviceBytes(1, 1, cap, cache.k_codes[base * 32:(base + cap) * 32].cpu().numpy(),
                       cache.v_codes[base * 32:(base + cap) * 32].cpu().numpy(),
                       cache.scalars[base * 4:(base + cap) * 4].cpu().numpy().view(np.uint16))


def _oracle_unit_cache(krows, vrows, l, h, pi, lut_k, lut_v, S, flags, cs_host):
    """The oracle's own cache of one unit: its raw tokens krows/vrows [n][64]
    (token j at position j) quantized into slots 0 .. n-1."""
    n = krows.shape[0]
    oc = oracle.Cache(1, 1, (n + 63) // 64 * 64)
    oracle.quantize_pack(oc, flags, cs_host, krows.reshape(1, 1, n, 1, 64), vrows.reshape(1, 1, n, 1, 64),
                         [0], [0], pi[l, h][None, None], lut_k[l, h][None, None], lut_v[l, h][None, None], S)
    return oc


def _check_units(cache, units, raw, out16, out32, q, pos, offs, n_att, pi, lut_k, lut_v, S, flags, cs_host):
    """units: (l, b, h) triples; raw[(l, b, h)] = (k rows, v rows) [n_att[b]][64]
    host float32; q [L][B][H][64] host float32; n_att[b] tokens attended."""
    worst = 0.0
    for (l, b, h) in units:
        n = int(n_att[b])
        krows, vrows = raw[(l, b, h)]
        assert krows.shape[0] == n
        oc = _oracle_unit_cache(krows, vrows, l, h, pi, lut_k, lut_v, S, flags, cs_host)
        # the GPU wrote every attended token (a skipped append or prefill
        # leaves zero norms), and its norms agree with the oracle's
        gs = _gpu_region(cache, l, h, int(offs[b]), n).scalars(0, 0)[:n]
        os_ = oc.scalars(0, 0)[:n]
        assert np.all(gs[:, 0] != 0) and np.all(gs[:, 2] != 0), (l, b, h)
        for col in (0, 2):
            ng = gs[:, col].view(np.float16).astype(np.float64)
            no = os_[:, col].view(np.float16).astype(np.float64)
            assert np.all(np.abs(ng - no) <= fp16_ulp(no) + 1e-12), (l, b, h, col)
        ref = oracle.decode(oc, flags, cs_host, q[l, b, h].reshape(1, 1, 1, 64), [int(pos[b])], [0], [n],
                            pi[l, h][None, None], lut_k[l, h][None, None], lut_v[l, h][None, None],
                            S)[0, 0, 0]
        g32 = out32[l, b, h].astype(np.float64)
        err = np.abs(g32 - ref)
        assert np.all(np.isfinite(g32)) and np.max(err) <= TOL, ((l, b, h), np.max(err))
        r16 = ref.astype(np.float16).astype(np.float64)
        g16 = out16[l, b, h].astype(np.float64)
        assert np.all(np.abs(g16 - r16) <= np.maximum(TOL, fp16_ulp(r16))), (l, b, h)
        worst = max(worst, float(np.max(err)))
    return worst


def _check_codes(cache, samples, cs_host, pi, lut_k, lut_v, S, flags):
    """samples: (l, h, slot, pos, k_row, v_row) with the raw fp16 inputs of the
    token; compares the GPU's key and value codes and norms with the oracle's
    quantizer of the same inputs."""
    for (l, h, slot, pos, krow, vrow) in samples:
        oc = _gpu_region(cache, l, h, slot - slot % 64, slot % 64 + 1)
        r = slot % 64
        for is_key, which, x, lut, col in ((True, "k", krow, lut_k, 0), (False, "v", vrow, lut_v, 2)):
            xh = oracle.rotated_input(np.asarray(x, np.float32), is_key, pos, cs_host, pi[l, h],
                                      rotate_v=bool(flags & tq.V_ROTATE))
            nib, n16, _ = oracle.quantize_vector(xh, lut[l, h], S, oracle.SIGN_PROJECTED if is_key else 0)
            got = unpack_slot(oc.region(which, 0, 0), r, which)
            bad = (got & 7) != (nib & 7)
            if bad.any():
                xd = xh.astype(np.float64)
                u = xd * 8.0 / np.linalg.norm(xd)
                t = 0.5 * (lut[l, h][:-1].astype(np.float64) + lut[l, h][1:])
                dist = np.min(np.abs(u[:, None] - t[None, :]), axis=1)
                assert np.all(dist[bad] < 1e-4), (l, h, slot, which)
                assert np.all(np.abs((got[bad] & 7).astype(int) - (nib[bad] & 7)) == 1)
            ng = float(np.array([oc.scalars(0, 0)[r, col]], np.uint16).view(np.float16)[0])
            no = float(np.array([n16], np.uint16).view(np.float16)[0])
            assert abs(ng - no) <= fp16_ulp(no) + 1e-12, (l, h, slot, which)


def _step_both_outputs(params, cache, q_d, k_d, v_d, pos, offs, lens, max_len, pi_d, lk_d, lv_d, S_d):
    """The bench's launch (fp16 output), then the same step again with fp32
    output (appending the same token to the same slot writes the same bytes)."""
    ws = torch.zeros(max(tq.decode_workspace_bytes(params, q_d.shape[1], q_d.shape[0], max_len), 16),
                     dtype=torch.uint8, device="cuda")
    out16 = tq.decode_step(params, cache, q_d, k_d, v_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d,
                           lk_d, lv_d, S_d, workspace=ws)
    p32 = tq.Params(params.num_layers, params.num_heads, params.rope_cs, io_dtype=params.io_dtype,
                    flags=params.flags | tq.OUT_FP32)
    out32 = tq.decode_step(p32, cache, q_d, k_d, v_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d,
                           lk_d, lv_d, S_d, workspace=ws)
    torch.cuda.synchronize()
    return out16.cpu().numpy(), out32.cpu().numpy()


def _sample_units(g, L, B, H, n):
    picks = {(0, 0, 0), (L - 1, B - 1, H - 1)}
    while len(picks) < n:
        picks.add((int(g.integers(L)), int(g.integers(B)), int(g.integers(H))))
    return sorted(picks)


def test_full_650m_33layer_step():
    # the bench's workload and inputs (same seed and draw order); every one of
    # the 660 (layer, head) units is compared with the oracle
    wl = synth.WORKLOADS["esm2-650m-33layer-seq1024"]
    L, H, T = wl.layers, wl.heads, wl.seq
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    k = synth.as_io(synth.keys(g, L, 1, T + 1, H, ch), "f16")
    v = synth.as_io(synth.values(g, L, 1, T + 1, H), "f16")
    q = synth.as_io(synth.queries(g, L, 1, H), "f16")
    pi = synth.rotations(g, L, H)
    S = synth.qjl_matrix(g)
    lut_k = np.broadcast_to(GAUSS_LUT, (L, H, 8)).copy()
    lut_v = np.broadcast_to(V_LUT, (L, H, 8)).copy()
    slots = 1088
    cs = tq.rope_table(slots + 64)
    cs_host = oracle.rope_table(slots + 64)
    params = tq.Params(L, H, cs, io_dtype=torch.float16, flags=tq.V_ROTATE)
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    pi_d, S_d, lk_d, lv_d = t_(pi), t_(S), t_(lut_k), t_(lut_v)
    cache = tq.Cache(L, H, slots)
    tq.quantize_pack(params, cache, t_(k[:, :, :T]), t_(v[:, :, :T]), _i32([0]), _i64([0]), pi_d, lk_d, lv_d,
                     S_d)
    out16, out32 = _step_both_outputs(params, cache, t_(q), t_(k[:, :, T]), t_(v[:, :, T]), [T], [0], [T],
                                      T + 1, pi_d, lk_d, lv_d, S_d)
    assert np.all(np.isfinite(out32))
    # the oracle quantizes the same T + 1 raw tokens of every unit (the T
    # prefilled and the appended one) into a cache of its own and decodes
    # every unit there in fp64
    oc = oracle.Cache(L, H, slots)
    oracle.quantize_pack(oc, tq.V_ROTATE, cs_host, k.astype(np.float32), v.astype(np.float32), [0], [0], pi,
                         lut_k, lut_v, S)
    ref = oracle.decode(oc, tq.V_ROTATE, cs_host, q.astype(np.float32), [T], [0], [T + 1], pi, lut_k, lut_v, S)
    err = np.abs(out32.astype(np.float64) - ref)
    assert np.max(err) <= TOL, np.unravel_index(np.argmax(err), err.shape)
    r16 = ref.astype(np.float16).astype(np.float64)
    assert np.all(np.abs(out16.astype(np.float64) - r16) <= np.maximum(TOL, fp16_ulp(r16)))
    # every unit's codes and norms, the appended token's included
    got = device_bytes(cache)
    total = diff = 0
    for l in range(L):
        for h in range(H):
            def rotated_of(s, is_key, l=l, h=h):
                x = (k if is_key else v)[l, 0, s, h].astype(np.float32)
                return (oracle.rotated_input(x, is_key, s, cs_host, pi[l, h]), (lut_k if is_key else lut_v)[l, h])
            t, d = assert_region_agrees(got.region("k", l, h), got.region("v", l, h), got.scalars(l, h),
                                        oc.region("k", l, h), oc.region("v", l, h), oc.scalars(l, h), T + 1,
                                        rotated_of)
            total += t
            diff += d
    print(f"650M step: max |err| {np.max(err):.3e} over 660 units; {diff} of {total} codes one level apart")
    # the two-step baseline at this size: fp32 softmax attention over the
    # dequantized fp16 rows reproduces the fused step's output to within the
    # bound the rows' fp16 rounding implies (see tests/test_gpu_dequant.py)
    units = _sample_units(synth.rng(1), L, 1, H, 12)
    ko, vo = tq.dequantize(params, cache, _i64([0]), _i32([T + 1]), T + 1, lk_d, lv_d, S_d)
    torch.cuda.synchronize()
    for (l, b, h) in units:
        kk = ko[l, b, h].float().cpu().numpy().astype(np.float64)
        vv = vo[l, b, h].float().cpu().numpy().astype(np.float64)
        qr = oracle.rope_apply(q[l, b, h].astype(np.float32), T, cs_host)
        P = pi[l, h].astype(np.float64)
        qh = P @ qr
        logits = 0.125 * (kk @ qh)
        w = np.exp(logits - logits.max())
        o = P.T @ ((w[:, None] * vv).sum(0) / w.sum())
        d = 0.125 * np.abs(qh) @ (fp16_ulp(kk).T / 2)
        bound = (np.exp(2 * d.max()) - 1) * np.abs(vv).max() + fp16_ulp(np.abs(vv).max()) + TOL
        assert np.max(np.abs(o - out32[l, b, h])) <= bound, ((l, b, h), np.max(np.abs(o - out32[l, b, h])))


def test_full_ragged_b64_step():
    wl = synth.WORKLOADS["esm2-650m-ragged-b64"]
    L, H, B = wl.layers, wl.heads, wl.batch
    g = synth.rng(wl.seed)
    lens = synth.ragged_lengths(g, B, *wl.ragged)
    ch = synth.outlier_channels(g, L, H)
    pi = synth.rotations(g, L, H)
    S = synth.qjl_matrix(g)
    lut_k = np.broadcast_to(GAUSS_LUT, (L, H, 8)).copy()
    lut_v = np.broadcast_to(V_LUT, (L, H, 8)).copy()
    offs, slots = synth.tile_aligned_offsets(lens, extra=1)
    positions = int(lens.max()) + 64
    cs = tq.rope_table(positions)
    cs_host = oracle.rope_table(positions)
    params = tq.Params(L, H, cs, io_dtype=torch.float16, flags=tq.V_ROTATE)
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    pi_d, S_d, lk_d, lv_d = t_(pi), t_(S), t_(lut_k), t_(lut_v)
    cache = tq.Cache(L, H, slots)
    units = _sample_units(synth.rng(2), L, B, H, 24)
    q_d = torch.empty((L, B, H, 64), dtype=torch.float16, device="cuda")
    k_new = torch.empty_like(q_d)
    v_new = torch.empty_like(q_d)
    samples = []
    raw = {}
    for l in range(L):
        gen = synth.device_generator(wl.seed, l, "cuda")
        kl = synth.keys_on(gen, B, int(lens.max()) + 1, H, ch[l], torch.float16, "cuda")
        vl = synth.values_on(gen, B, int(lens.max()) + 1, H, torch.float16, "cuda")
        q_d[l] = synth.queries_on(gen, B, H, torch.float16, "cuda")
        for b in range(B):
            n = int(lens[b])
            # each sequence's own tokens into its own packed range
            tq.quantize_pack(params, cache, kl[None, b:b + 1, :n].contiguous(), vl[None, b:b + 1, :n].contiguous(),
                             _i32([0]), _i64([int(offs[b])]), pi_d, lk_d, lv_d, S_d, layer0=l)
            k_new[l, b] = kl[b, n]
            v_new[l, b] = vl[b, n]
        for (ul, ub, uh) in units:
            if ul == l:
                n = int(lens[ub]) + 1
                raw[(ul, ub, uh)] = (kl[ub, :n, uh].float().cpu().numpy(), vl[ub, :n, uh].float().cpu().numpy())
                for j in (0, int(lens[ub]) - 1):
                    samples.append((l, uh, int(offs[ub]) + j, j, kl[ub, j, uh].float().cpu().numpy(),
                                    vl[ub, j, uh].float().cpu().numpy()))
        del kl, vl
    out16, out32 = _step_both_outputs(params, cache, q_d, k_new, v_new, lens, offs, lens, int(lens.max()) + 1,
                                      pi_d, lk_d, lv_d, S_d)
    assert np.all(np.isfinite(out32))
    q_host = q_d.float().cpu().numpy()
    _check_units(cache, units, raw, out16, out32, q_host, lens, offs, lens + 1, pi, lut_k, lut_v, S,
                 tq.V_ROTATE, cs_host)
    kn, vn = k_new.float().cpu().numpy(), v_new.float().cpu().numpy()
    samples += [(l, h, int(offs[b]) + int(lens[b]), int(lens[b]), kn[l, b, h], vn[l, b, h])
                for (l, b, h) in units[:8]]
    _check_codes(cache, samples, cs_host, pi, lut_k, lut_v, S, tq.V_ROTATE)


def test_full_3b_step():
    wl = synth.WORKLOADS["esm2-3b-36layer-b16-seq8192"]
    L, H, B, T = wl.layers, wl.heads, wl.batch, wl.seq
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    pi = synth.rotations(g, L, H)
    S = synth.qjl_matrix(g)
    lut_k = np.broadcast_to(GAUSS_LUT, (L, H, 8)).copy()
    lut_v = np.broadcast_to(V_LUT, (L, H, 8)).copy()
    cap = T + 64
    offs = np.arange(B, dtype=np.int64) * cap
    slots = B * cap
    cs = tq.rope_table(T + 64)
    cs_host = oracle.rope_table(T + 64)
    params = tq.Params(L, H, cs, io_dtype=torch.float16, flags=tq.V_ROTATE)
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    pi_d, S_d, lk_d, lv_d = t_(pi), t_(S), t_(lut_k), t_(lut_v)
    cache = tq.Cache(L, H, slots)            # 13.7 GB
    units = _sample_units(synth.rng(3), L, B, H, 12)
    q_d = torch.empty((L, B, H, 64), dtype=torch.float16, device="cuda")
    k_new = torch.empty_like(q_d)
    v_new = torch.empty_like(q_d)
    zeros = _i32(np.zeros(B))
    offs_d = _i64(offs)
    samples = []
    raw = {}
    for l in range(L):
        gen = synth.device_generator(wl.seed, l, "cuda")
        kl = synth.keys_on(gen, B, T + 1, H, ch[l], torch.float16, "cuda")
        vl = synth.values_on(gen, B, T + 1, H, torch.float16, "cuda")
        q_d[l] = synth.queries_on(gen, B, H, torch.float16, "cuda")
        tq.quantize_pack(params, cache, kl[None, :, :T].contiguous(), vl[None, :, :T].contiguous(), zeros,
                         offs_d, pi_d, lk_d, lv_d, S_d, layer0=l)
        k_new[l] = kl[:, T]
        v_new[l] = vl[:, T]
        for (ul, ub, uh) in units:
            if ul == l:
                raw[(ul, ub, uh)] = (kl[ub, :T + 1, uh].float().cpu().numpy(),
                                     vl[ub, :T + 1, uh].float().cpu().numpy())
                for j in (0, 4095, T - 1):
                    samples.append((l, uh, int(offs[ub]) + j, j, kl[ub, j, uh].float().cpu().numpy(),
                                    vl[ub, j, uh].float().cpu().numpy()))
        del kl, vl
    lens = np.full(B, T, np.int32)
    out16, out32 = _step_both_outputs(params, cache, q_d, k_new, v_new, lens, offs, lens, T + 1, pi_d, lk_d,
                                      lv_d, S_d)
    assert np.all(np.isfinite(out32))
    q_host = q_d.float().cpu().numpy()
    _check_units(cache, units, raw, out16, out32, q_host, lens, offs, lens + 1, pi, lut_k, lut_v, S,
                 tq.V_ROTATE, cs_host)
    kn, vn = k_new.float().cpu().numpy(), v_new.float().cpu().numpy()
    samples += [(l, h, int(offs[b]) + T, T, kn[l, b, h], vn[l, b, h]) for (l, b, h) in units]
    _check_codes(cache, samples, cs_host, pi, lut_k, lut_v, S, tq.V_ROTATE)
