"""Two workloads run as stated, end to end, against the oracle.

ESM-2 650M one layer (20 heads x 64, batch 1, fp16): per-head Pi from the SVD
of 4096 post-RoPE calibration keys (Sec. 3.2) and calibrated, separate K and V
tables (Sec. 3.3), both computed by the oracle and given to both sides (Pi
entries inside near-degenerate singular subspaces are not pinned, so the two
sides share one Pi); the GPU's own calibration of the same data is checked
against the oracle's. Prefill of 1024 tokens, then 64 tq_decode_step steps.

ESM-2 3B shape (36 layers x 40 heads, batch 16, 8192 tokens, fp16): Pi and
tables calibrated per head (the GPU calibrates every head; the sampled heads
take the oracle's calibration, on both sides), prefill, then 32 steps,
checked on sampled (layer, sequence, head) units.

Two claims are checked separately. The quantizer: the GPU's own prefill and
appends agree with the oracle's quantizer of the same raw tokens, codes equal
or one level apart where the exact coordinate lies within rounding of a
threshold (the two rotate in different arithmetic). Decode: on identical
caches (the GPU steps on an upload of the oracle's prefill; after each step
the appended token's bytes are compared, and where a code differs at a
threshold the oracle's bytes are uploaded and tq_decode_attend gives the
step's output), 2e-3 max-abs on the fp32 output and max(2e-3, 1 fp16 ulp) on
the fp16 output against the oracle rounded to fp16. With calibrated tables on
the SVD basis one threshold flip on a dominant key can move the output far
more than 2e-3, which is why decode is compared on the same codes."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import paper_2603_26110_amd as tq
from gpu_cases import GAUSS_LUT, assert_region_agrees, device_bytes, fp16_ulp, to_gpu, unpack_planes
from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _i32(x):
    return torch.tensor(np.asarray(x, np.int32), dtype=torch.int32).cuda()


def _i64(x):
    return torch.tensor(np.asarray(x, np.int64), dtype=torch.int64).cuda()


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _oracle_calibration(xk, xv, threads=16):
    """Per head: Pi from the SVD of the post-RoPE keys xk[h] [ncal][64], the K
    table fitted to Pi xk[h], the V table to Pi xv[h] (values are stored
    rotated). Returns float32 arrays [nh][64][64], [nh][8], [nh][8], sigma."""
    def one(h):
        pi, sg = oracle.calibrate_rotation(xk[h])
        lk = oracle.calibrate_lut(xk[h], pi, GAUSS_LUT).astype(np.float32)
        lv = oracle.calibrate_lut(xv[h], pi, GAUSS_LUT).astype(np.float32)
        assert np.all(np.diff(lk) > 0) and np.all(np.diff(lv) > 0)
        return pi, lk, lv, sg
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(one, range(len(xk))))
    return (np.stack([r[0] for r in res]), np.stack([r[1] for r in res]), np.stack([r[2] for r in res]),
            np.stack([r[3] for r in res]))


def _steps_both(params, cache, q_d, k_d, v_d, pos, offs, lens, max_len, pi_d, lk_d, lv_d, S_d, ws):
    """One step with fp16 output, then again with fp32 output (the same token
    appended to the same slot writes the same bytes)."""
    out16 = tq.decode_step(params, cache, q_d, k_d, v_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d,
                           lk_d, lv_d, S_d, workspace=ws)
    p32 = tq.Params(params.num_layers, params.num_heads, params.rope_cs, io_dtype=params.io_dtype,
                    flags=params.flags | tq.OUT_FP32)
    out32 = tq.decode_step(p32, cache, q_d, k_d, v_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d,
                           lk_d, lv_d, S_d, workspace=ws)
    torch.cuda.synchronize()
    return out16.cpu().numpy().astype(np.float64), out32.cpu().numpy().astype(np.float64)


def _attend_both(params, cache, q_d, pos, offs, lens, max_len, pi_d, lk_d, lv_d, S_d, ws):
    """tq_decode_attend with fp16, then fp32 output."""
    o16 = tq.decode_attend(params, cache, q_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d, lk_d, lv_d,
                           S_d, workspace=ws)
    p32 = tq.Params(params.num_layers, params.num_heads, params.rope_cs, io_dtype=params.io_dtype,
                    flags=params.flags | tq.OUT_FP32)
    o32 = tq.decode_attend(p32, cache, q_d, _i32(pos), _i64(offs), _i32(lens), max_len, pi_d, lk_d, lv_d, S_d,
                           workspace=ws)
    torch.cuda.synchronize()
    return o16.cpu().numpy().astype(np.float64), o32.cpu().numpy().astype(np.float64)


def _tile_bytes(cache, l, h, slot):
    """The GPU's K, V and scalar bytes of the tile holding `slot` of region
    (l, h) (for comparison with the oracle's; never an oracle input)."""
    t0 = ((l * cache.num_heads + h) * cache.slots + slot // 64 * 64)
    return (cache.k_codes[t0 * 32:(t0 + 64) * 32].cpu().numpy(), cache.v_codes[t0 * 32:(t0 + 64) * 32].cpu().numpy(),
            cache.scalars[t0 * 4:(t0 + 64) * 4].cpu().numpy().view(np.uint16))


def _slot_matches(got, ref, r, rotated_of):
    """Tile bytes (k, v, scalars) of the GPU and of the oracle: True if slot r
    is identical; otherwise its codes must differ only at threshold
    coordinates, by one level, and its norms by at most one fp16 ulp (False)."""
    gk, gv = unpack_planes(got[0], got[1])
    rk, rv = unpack_planes(ref[0], ref[1])
    gs, rs = got[2].reshape(64, 4)[r], ref[2].reshape(64, 4)[r]
    if np.array_equal(gk[r], rk[r]) and np.array_equal(gv[r], rv[r]) and np.array_equal(gs, rs):
        return True
    for col in (0, 2):
        a = np.array([gs[col]], np.uint16).view(np.float16).astype(np.float64)
        b = np.array([rs[col]], np.uint16).view(np.float16).astype(np.float64)
        assert np.all(np.abs(a - b) <= fp16_ulp(b) + 1e-12)
    for is_key, g_, r_ in ((True, gk[r], rk[r]), (False, gv[r], rv[r])):
        bad = (g_ & 7) != (r_ & 7)
        if bad.any():
            xh, lut = rotated_of(is_key)
            xd = xh.astype(np.float64)
            u = xd * 8.0 / np.linalg.norm(xd)
            t = 0.5 * (lut[:-1].astype(np.float64) + lut[1:])
            dist = np.min(np.abs(u[:, None] - t[None, :]), axis=1)
            assert np.all(dist[bad] < 1e-4), (is_key, dist[bad])
            assert np.all(np.abs((g_[bad] & 7).astype(int) - (r_[bad] & 7)) == 1)
    return False


def _compare(out16, out32, ref):
    assert np.all(np.isfinite(out32))
    err = np.abs(out32 - ref)
    assert np.max(err) <= TOL, np.max(err)
    r16 = ref.astype(np.float16).astype(np.float64)
    assert np.all(np.abs(out16 - r16) <= np.maximum(TOL, fp16_ulp(r16)))
    return float(np.max(err))


def test_esm2_650m_one_layer_svd_calibrated_64_steps():
    wl = synth.WORKLOADS["esm2-650m-1layer-seq1024"]
    L, H, T, steps, ncal = wl.layers, wl.heads, wl.seq, wl.decode_steps, wl.calib_vectors
    assert (L, H, T, steps, ncal, wl.rotation) == (1, 20, 1024, 64, 4096, "svd")
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    k = synth.as_io(synth.keys(g, L, 1, T + steps, H, ch), "f16")
    v = synth.as_io(synth.values(g, L, 1, T + steps, H), "f16")
    q_all = synth.as_io(synth.queries(g, steps * L, 1, H), "f16").reshape(steps, L, 1, H, 64)
    S = synth.qjl_matrix(g)
    # calibration set: 4096 keys per head, RoPE'd at seeded positions in [0, T), and 4096 values
    ck = synth.as_io(synth.keys(g, 1, 1, ncal, H, ch), "f16")[0, 0].astype(np.float32)     # [ncal][H][64]
    cv = synth.as_io(synth.values(g, 1, 1, ncal, H), "f16")[0, 0].astype(np.float32)
    cpos = synth.calibration_positions(g, ncal, T)
    slots = 1088
    cs_host = oracle.rope_table(slots + 64)
    xk = np.empty((H, ncal, 64), np.float32)
    for h in range(H):
        for i in range(ncal):
            xk[h, i] = oracle.rope_apply(ck[i, h], int(cpos[i]), cs_host)
    xv = np.ascontiguousarray(cv.transpose(1, 0, 2))
    pi1, lk1, lv1, sg = _oracle_calibration(xk, xv)
    # the GPU's calibration of the same data agrees with the oracle's
    gpi, gsg = tq.calibrate_rotation(_t(xk))
    glk = tq.calibrate_lut(_t(xk), _t(pi1), GAUSS_LUT)
    glv = tq.calibrate_lut(_t(xv), _t(pi1), GAUSS_LUT)
    np.testing.assert_allclose(gsg.cpu().numpy(), sg, rtol=1e-5)
    np.testing.assert_allclose(glk.cpu().numpy(), lk1, rtol=0, atol=2e-6)
    np.testing.assert_allclose(glv.cpu().numpy(), lv1, rtol=0, atol=2e-6)
    gp = gpi.cpu().numpy().astype(np.float64)
    for h in range(H):
        np.testing.assert_allclose(gp[h] @ gp[h].T, np.eye(64), atol=1e-6)
    pi, lut_k, lut_v = pi1[None], lk1[None], lv1[None]

    cs = tq.rope_table(slots + 64)
    params = tq.Params(L, H, cs, io_dtype=torch.float16, flags=tq.V_ROTATE)
    pi_d, S_d, lk_d, lv_d = _t(pi), _t(S), _t(lut_k), _t(lut_v)
    # the quantizer, end to end: the GPU's own prefill and appends of every
    # token against the oracle's
    own = tq.Cache(L, H, slots)
    tq.quantize_pack(params, own, _t(k[:, :, :T]), _t(v[:, :, :T]), _i32([0]), _i64([0]), pi_d, lk_d, lv_d, S_d)
    oc = oracle.Cache(L, H, slots)
    oracle.quantize_pack(oc, tq.V_ROTATE, cs_host, k[:, :, :T].astype(np.float32), v[:, :, :T].astype(np.float32),
                         [0], [0], pi, lut_k, lut_v, S)
    got = device_bytes(own)
    flips = 0
    for h in range(H):
        def rotated_of(sl, is_key, h=h):
            x = (k if is_key else v)[0, 0, sl, h].astype(np.float32)
            return oracle.rotated_input(x, is_key, sl, cs_host, pi[0, h]), (lut_k if is_key else lut_v)[0, h]
        flips += assert_region_agrees(got.region("k", 0, h), got.region("v", 0, h), got.scalars(0, h),
                                      oc.region("k", 0, h), oc.region("v", 0, h), oc.scalars(0, h), T,
                                      rotated_of)[1]
    # decode, on the oracle's prefill: 64 steps
    cache = to_gpu(oc)
    ws = torch.zeros(max(tq.decode_workspace_bytes(params, 1, L, T + steps), 16), dtype=torch.uint8, device="cuda")
    worst = 0.0
    patched = 0
    for s in range(steps):
        n = T + s
        q_d = _t(q_all[s])
        out16, out32 = _steps_both(params, cache, q_d, _t(k[:, :, n]), _t(v[:, :, n]), [n], [0], [n],
                                   T + steps, pi_d, lk_d, lv_d, S_d, ws)
        oracle.quantize_pack(oc, tq.V_ROTATE, cs_host, k[:, :, n:n + 1].astype(np.float32),
                             v[:, :, n:n + 1].astype(np.float32), [n], [n], pi, lut_k, lut_v, S)
        same = True
        for h in range(H):
            ref_tile = tuple(a[(h * slots + n // 64 * 64) * w:(h * slots + n // 64 * 64 + 64) * w]
                             for a, w in ((oc.k, 32), (oc.v, 32), (oc.s, 4)))

            def rotated_of(is_key, h=h):
                x = (k if is_key else v)[0, 0, n, h].astype(np.float32)
                return oracle.rotated_input(x, is_key, n, cs_host, pi[0, h]), (lut_k if is_key else lut_v)[0, h]
            same &= _slot_matches(_tile_bytes(cache, 0, h, n), ref_tile, n % 64, rotated_of)
        if not same:
            # an appended code differs at a threshold: decode the oracle's bytes
            cache = to_gpu(oc)
            out16, out32 = _attend_both(params, cache, q_d, [n], [0], [n + 1], T + steps, pi_d, lk_d, lv_d, S_d, ws)
            patched += 1
        ref = oracle.decode(oc, tq.V_ROTATE, cs_host, q_all[s].astype(np.float32), [n], [0], [n + 1], pi, lut_k,
                            lut_v, S)
        worst = max(worst, _compare(out16, out32, ref))
    print(f"650M one layer, SVD Pi + calibrated tables: prefill {flips} codes one level apart; 64 steps "
          f"({patched} with a threshold flip in the appended token) max |err| {worst:.3e}")


def _rope_torch(x, pos, cs):
    """RoPE (pairs (2m, 2m + 1)) of x [n][H][64] at positions pos [n], with the
    library's (cos, sin) table: test-side preparation of post-RoPE calibration
    keys for the GPU's own calibration."""
    c = cs[pos.long(), :, 0][:, None, :]
    s_ = cs[pos.long(), :, 1][:, None, :]
    x0, x1 = x[..., 0::2], x[..., 1::2]
    return torch.stack((x0 * c - x1 * s_, x0 * s_ + x1 * c), dim=-1).reshape(x.shape)


def test_esm2_3b_svd_calibrated_32_steps():
    wl = synth.WORKLOADS["esm2-3b-36layer-b16-seq8192"]
    L, H, B, T, steps, ncal = wl.layers, wl.heads, wl.batch, wl.seq, wl.decode_steps, wl.calib_vectors
    assert (L, H, B, T, steps, ncal, wl.rotation) == (36, 40, 16, 8192, 32, 4096, "svd")
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    S = synth.qjl_matrix(g)
    cap = T + steps + 64 - (T + steps) % 64 if (T + steps) % 64 else T + steps
    offs = np.arange(B, dtype=np.int64) * cap
    slots = B * cap
    positions = T + steps + 64
    cs = tq.rope_table(positions)
    cs_host = oracle.rope_table(positions)
    units = []
    gu = synth.rng(4)
    picks = {(0, 0, 0), (L - 1, B - 1, H - 1)}
    while len(picks) < 12:
        picks.add((int(gu.integers(L)), int(gu.integers(B)), int(gu.integers(H))))
    units = sorted(picks)
    heads = sorted({(l, h) for (l, _, h) in units})

    # ---- calibration: the GPU calibrates every head on calibration keys and
    # values drawn on the device; the sampled heads take the oracle's
    # calibration of host-drawn sets, on both sides
    pi_d = torch.empty((L, H, 64, 64), dtype=torch.float32, device="cuda")
    lk_d = torch.empty((L, H, 8), dtype=torch.float32, device="cuda")
    lv_d = torch.empty((L, H, 8), dtype=torch.float32, device="cuda")
    for l in range(L):
        gen = synth.device_generator(wl.seed + 7919, l, "cuda")
        ckl = synth.keys_on(gen, 1, ncal, H, ch[l], torch.float16, "cuda")[0].float()    # [ncal][H][64]
        cvl = synth.values_on(gen, 1, ncal, H, torch.float16, "cuda")[0].float()
        cpos = torch.randint(0, T, (ncal,), generator=gen, device="cuda")
        xk = _rope_torch(ckl, cpos, cs).transpose(0, 1).contiguous()                  # [H][ncal][64]
        xv = cvl.transpose(0, 1).contiguous()
        p, _ = tq.calibrate_rotation(xk)
        pi_d[l] = p
        lk_d[l] = tq.calibrate_lut(xk, p)
        lv_d[l] = tq.calibrate_lut(xv, p)
    torch.cuda.synchronize()
    print(f"  3B: GPU calibration of {L * H} heads done", flush=True)
    pi = np.zeros((L, H, 64, 64), np.float32)
    lut_k = np.zeros((L, H, 8), np.float32)
    lut_v = np.zeros((L, H, 8), np.float32)
    gh = synth.rng(wl.seed + 1)
    xk_h = np.empty((len(heads), ncal, 64), np.float32)
    xv_h = np.empty((len(heads), ncal, 64), np.float32)
    for i, (l, h) in enumerate(heads):
        kk = synth.as_io(synth.keys(gh, 1, 1, ncal, 1, ch[l:l + 1, h:h + 1]), "f16")[0, 0, :, 0].astype(np.float32)
        vv = synth.as_io(synth.values(gh, 1, 1, ncal, 1), "f16")[0, 0, :, 0].astype(np.float32)
        cp = synth.calibration_positions(gh, ncal, T)
        xk_h[i] = np.stack([oracle.rope_apply(kk[j], int(cp[j]), cs_host) for j in range(ncal)])
        xv_h[i] = vv
    opi, olk, olv, _ = _oracle_calibration(xk_h, xv_h)
    for i, (l, h) in enumerate(heads):
        pi[l, h], lut_k[l, h], lut_v[l, h] = opi[i], olk[i], olv[i]
        pi_d[l, h] = _t(opi[i])
        lk_d[l, h] = _t(olk[i])
        lv_d[l, h] = _t(olv[i])
    assert bool(torch.all(lk_d[..., 1:] > lk_d[..., :-1])) and bool(torch.all(lv_d[..., 1:] > lv_d[..., :-1]))

    # ---- prefill, the per-step tokens and queries, the oracle's unit caches
    params = tq.Params(L, H, cs, io_dtype=torch.float16, flags=tq.V_ROTATE)
    S_d = _t(S)
    cache = tq.Cache(L, H, slots)            # 13.7 GB
    q_all = torch.empty((steps, L, B, H, 64), dtype=torch.float16, device="cuda")
    k_all = torch.empty_like(q_all)
    v_all = torch.empty_like(q_all)
    zeros = _i32(np.zeros(B))
    offs_d = _i64(offs)
    raw = {}
    for l in range(L):
        gen = synth.device_generator(wl.seed, l, "cuda")
        kl = synth.keys_on(gen, B, T + steps, H, ch[l], torch.float16, "cuda")
        vl = synth.values_on(gen, B, T + steps, H, torch.float16, "cuda")
        for s in range(steps):
            q_all[s, l] = synth.queries_on(gen, B, H, torch.float16, "cuda")
        tq.quantize_pack(params, cache, kl[None, :, :T].contiguous(), vl[None, :, :T].contiguous(), zeros, offs_d,
                         pi_d, lk_d, lv_d, S_d, layer0=l)
        k_all[:, l] = kl[:, T:T + steps].transpose(0, 1)
        v_all[:, l] = vl[:, T:T + steps].transpose(0, 1)
        for (ul, ub, uh) in units:
            if ul == l:
                raw[(ul, ub, uh)] = (kl[ub, :, uh].float().cpu().numpy(), vl[ub, :, uh].float().cpu().numpy())
        del kl, vl
        if l % 6 == 5:
            print(f"  3B prefill: {l + 1} of {L} layers", flush=True)
    # the quantizer, end to end: the GPU's prefill of each sampled unit
    # against the oracle's quantizer of the same raw tokens; then the decode
    # cache of each sampled unit becomes the oracle's bytes
    ocs = {}
    flips = 0

    def region_slice(l, h, b):
        base = (l * H + h) * slots + int(offs[b])
        return base, base + cap

    def upload(u, first_slot=0, count=None):
        l, b, h = u
        base, _ = region_slice(l, h, b)
        oc = ocs[u]
        n = cap - first_slot if count is None else count
        lo, hi = base + first_slot, base + first_slot + n
        cache.k_codes[lo * 32:hi * 32].copy_(torch.from_numpy(oc.k[first_slot * 32:(first_slot + n) * 32]))
        cache.v_codes[lo * 32:hi * 32].copy_(torch.from_numpy(oc.v[first_slot * 32:(first_slot + n) * 32]))
        cache.scalars[lo * 4:hi * 4].copy_(torch.from_numpy(oc.s[first_slot * 4:(first_slot + n) * 4].view(np.int16)))

    for u in units:
        l, b, h = u
        kr, vr = raw[u]
        oc = oracle.Cache(1, 1, cap)
        oracle.quantize_pack(oc, tq.V_ROTATE, cs_host, kr[:T].reshape(1, 1, T, 1, 64), vr[:T].reshape(1, 1, T, 1, 64),
                             [0], [0], pi[l, h][None, None], lut_k[l, h][None, None], lut_v[l, h][None, None], S)
        ocs[u] = oc
        lo, hi = region_slice(l, h, b)
        gk = cache.k_codes[lo * 32:hi * 32].cpu().numpy()
        gv = cache.v_codes[lo * 32:hi * 32].cpu().numpy()
        gs = cache.scalars[lo * 4:hi * 4].cpu().numpy().view(np.uint16)

        def rotated_of(sl, is_key, l=l, h=h, kr=kr, vr=vr):
            x = (kr if is_key else vr)[sl]
            return oracle.rotated_input(x, is_key, sl, cs_host, pi[l, h]), (lut_k if is_key else lut_v)[l, h]
        flips += assert_region_agrees(gk, gv, gs, oc.k, oc.v, oc.s, T, rotated_of)[1]
        upload(u)
    print(f"  3B prefill: {flips} codes of the sampled units one level apart from the oracle's", flush=True)

    ws = torch.zeros(max(tq.decode_workspace_bytes(params, B, L, T + steps), 16), dtype=torch.uint8, device="cuda")
    lens = np.full(B, T, np.int32)
    worst = 0.0
    patched = 0
    for s in range(steps):
        n = T + s
        out16, out32 = _steps_both(params, cache, q_all[s], k_all[s].contiguous(), v_all[s].contiguous(), lens + s,
                                   offs, lens + s, T + steps, pi_d, lk_d, lv_d, S_d, ws)
        assert np.all(np.isfinite(out32))
        same = True
        for u in units:
            l, b, h = u
            kr, vr = raw[u]
            oc = ocs[u]
            oracle.quantize_pack(oc, tq.V_ROTATE, cs_host, kr[n:n + 1].reshape(1, 1, 1, 1, 64),
                                 vr[n:n + 1].reshape(1, 1, 1, 1, 64), [n], [n], pi[l, h][None, None],
                                 lut_k[l, h][None, None], lut_v[l, h][None, None], S)
            t0 = n // 64 * 64
            ref_tile = (oc.k[t0 * 32:(t0 + 64) * 32], oc.v[t0 * 32:(t0 + 64) * 32], oc.s[t0 * 4:(t0 + 64) * 4])
            lo, _ = region_slice(l, h, b)
            got_tile = (cache.k_codes[(lo + t0) * 32:(lo + t0 + 64) * 32].cpu().numpy(),
                        cache.v_codes[(lo + t0) * 32:(lo + t0 + 64) * 32].cpu().numpy(),
                        cache.scalars[(lo + t0) * 4:(lo + t0 + 64) * 4].cpu().numpy().view(np.uint16))

            def rotated_of(is_key, l=l, h=h, kr=kr, vr=vr):
                x = (kr if is_key else vr)[n]
                return oracle.rotated_input(x, is_key, n, cs_host, pi[l, h]), (lut_k if is_key else lut_v)[l, h]
            if not _slot_matches(got_tile, ref_tile, n % 64, rotated_of):
                upload(u, t0, 64)
                same = False
        if not same:
            out16, out32 = _attend_both(params, cache, q_all[s], lens + s, offs, lens + s + 1, T + steps, pi_d, lk_d,
                                        lv_d, S_d, ws)
            patched += 1
        qh = q_all[s].float().cpu().numpy()
        for u in units:
            l, b, h = u
            ref = oracle.decode(ocs[u], tq.V_ROTATE, cs_host, qh[l, b, h].reshape(1, 1, 1, 64), [n], [0], [n + 1],
                                pi[l, h][None, None], lut_k[l, h][None, None], lut_v[l, h][None, None], S)[0, 0, 0]
            worst = max(worst, _compare(out16[l, b, h], out32[l, b, h], ref))
        if s % 8 == 7:
            print(f"  3B: {s + 1} of {steps} steps, max |err| {worst:.3e}", flush=True)
    print(f"3B shape, calibrated, 32 steps ({patched} with a threshold flip in an appended token): max |err| "
          f"{worst:.3e} on {len(units)} sampled units")
