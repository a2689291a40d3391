"""Shared helpers of the GPU parity tests: seeded inputs for both sides,
running the library through its C ABI, moving the oracle's cache to the
device, and reading the device cache back for comparison with the oracle's
(never as an oracle input; GPU bytes are decoded by this module's own
unpacker)."""
from __future__ import annotations

import numpy as np
import torch

import paper_2603_26110_amd as tq
from oracle import oracle
from paper_2603_26110_amd import synth

GAUSS_LUT = oracle.lloyd_max_gaussian(8)[0].astype(np.float32)


class Case:
    """Inputs of one quantize + decode run, as numpy (oracle) and torch (GPU)."""

    def __init__(self, seed, L, H, B, T, io="f16", flags=tq.V_ROTATE, slots=None, slot0=None,
                 pos0=None, positions=2048, lut_k=None, lut_v=None, layer0=0, nl=None):
        g = synth.rng(seed)
        self.L, self.H, self.B, self.T = L, H, B, T
        self.nl = L if nl is None else nl
        self.layer0 = layer0
        self.io = io
        self.flags = flags
        ch = synth.outlier_channels(g, L, H)
        k = synth.keys(g, self.nl, B, T, H, ch[layer0:layer0 + self.nl])
        v = synth.values(g, self.nl, B, T, H)
        q = synth.queries(g, self.nl, B, H)
        self.k = synth.as_io(k, io)
        self.v = synth.as_io(v, io)
        self.q = synth.as_io(q, io)
        self.pi = synth.rotations(g, L, H)
        self.S = synth.qjl_matrix(g)
        self.lut_k = np.broadcast_to(GAUSS_LUT if lut_k is None else lut_k, (L, H, 8)).copy()
        self.lut_v = np.broadcast_to(GAUSS_LUT if lut_v is None else lut_v, (L, H, 8)).copy()
        self.ebar = (0.1 + 0.2 * g.random((L, H, 2))).astype(np.float32)
        self.slots = slots or ((T + 63) // 64 + 1) * 64 * B
        self.slot0 = np.arange(B, dtype=np.int64) * (self.slots // B) if slot0 is None \
            else np.asarray(slot0, np.int64)
        self.pos0 = np.zeros(B, np.int32) if pos0 is None else np.asarray(pos0, np.int32)
        self.positions = positions
        self.cs_host = oracle.rope_table(positions)
        self.dev = {}

    # ---------------------------------------------------------------- GPU side
    def params(self, flags=None, io=None) -> tq.Params:
        if "cs" not in self.dev:
            self.dev["cs"] = tq.rope_table(self.positions)
        io = io or self.io
        return tq.Params(self.L, self.H, self.dev["cs"],
                         io_dtype=torch.float16 if io == "f16" else torch.float32,
                         flags=self.flags if flags is None else flags)

    def t(self, name, arr=None):
        if name not in self.dev:
            a = getattr(self, name) if arr is None else arr
            self.dev[name] = torch.from_numpy(np.ascontiguousarray(a)).cuda()
        return self.dev[name]

    def gpu_quantize(self, cache, k=None, v=None, flags=None, pos0=None, slot0=None):
        p = self.params(flags)
        k = self.t("k") if k is None else k
        v = self.t("v") if v is None else v
        p0 = self.t("pos0") if pos0 is None else torch.from_numpy(np.asarray(pos0, np.int32)).cuda()
        s0 = self.t("slot0") if slot0 is None else torch.from_numpy(np.asarray(slot0, np.int64)).cuda()
        tq.quantize_pack(p, cache, k, v, p0, s0, self.t("pi"), self.t("lut_k"), self.t("lut_v"),
                         self.t("S"), self.t("ebar"), layer0=self.layer0)

    def gpu_decode(self, cache, q_pos, seq_slot0, seq_len, max_len, flags=None, io=None, q=None):
        p = self.params(flags, io)
        qq = self.t("q") if q is None else q
        return tq.decode_attend(p, cache, qq, torch.tensor(q_pos, dtype=torch.int32).cuda(),
                                torch.tensor(seq_slot0, dtype=torch.int64).cuda(),
                                torch.tensor(seq_len, dtype=torch.int32).cuda(), max_len,
                                self.t("pi"), self.t("lut_k"), self.t("lut_v"), self.t("S"),
                                self.t("ebar"), layer0=self.layer0)

    # ------------------------------------------------------------- oracle side
    def oracle_quantize(self, ocache, k=None, v=None, flags=None, pos0=None, slot0=None):
        k = self.k if k is None else k
        v = self.v if v is None else v
        oracle.quantize_pack(ocache, self.flags if flags is None else flags, self.cs_host,
                             np.asarray(k, np.float32), np.asarray(v, np.float32),
                             self.pos0 if pos0 is None else pos0,
                             self.slot0 if slot0 is None else slot0,
                             self.pi, self.lut_k, self.lut_v, self.S, layer0=self.layer0)

    def oracle_decode(self, ocache, q_pos, seq_slot0, seq_len, flags=None, units=None):
        return oracle.decode(ocache, self.flags if flags is None else flags, self.cs_host,
                             np.asarray(self.q, np.float32), q_pos, seq_slot0, seq_len, self.pi,
                             self.lut_k, self.lut_v, self.S, ebar=self.ebar, layer0=self.layer0,
                             units=units)


def to_gpu(oc: oracle.Cache) -> tq.Cache:
    """A device cache holding the bytes the oracle's quantizer wrote (so that
    decode parity never feeds GPU output to the oracle)."""
    cache = tq.Cache(oc.L, oc.H, oc.slots)
    cache.k_codes.copy_(torch.from_numpy(oc.k))
    cache.v_codes.copy_(torch.from_numpy(oc.v))
    cache.scalars.copy_(torch.from_numpy(oc.s.view(np.int16)))
    return cache


class DeviceBytes:
    """The bytes a GPU call wrote into a cache, copied to the host for
    comparison with the oracle's (never handed to the oracle): k and v code
    planes (uint8) and scalars (uint16), laid out per (layer, head) region."""

    def __init__(self, L, H, slots, k, v, s):
        self.L, self.H, self.slots = L, H, slots
        self.k, self.v, self.s = k, v, s

    def region(self, which: str, l: int, h: int) -> np.ndarray:
        plane = self.k if which == "k" else self.v
        base = (l * self.H + h) * self.slots * 32
        return plane[base:base + self.slots * 32]

    def scalars(self, l: int, h: int) -> np.ndarray:
        base = (l * self.H + h) * self.slots * 4
        return self.s[base:base + self.slots * 4].reshape(self.slots, 4)


def device_bytes(cache: tq.Cache) -> DeviceBytes:
    return DeviceBytes(cache.num_layers, cache.num_heads, cache.slots, cache.k_codes.cpu().numpy(),
                       cache.v_codes.cpu().numpy(), cache.scalars.cpu().numpy().view(np.uint16))


def unpack_slot(region: np.ndarray, s: int, plane: str = "k") -> np.ndarray:
    """The 64 nibbles (idx | sign << 3) of slot s of one (layer, head) region,
    decoded from the layout include/turboesm.h documents: K token-major (16-byte
    half c of slot r of tile t at t*2048 + (c*64 + r)*16, word w = dims
    8w..8w+7, index of dim 8w+j at bits 3j.., sign at bit 24+j); V
    dimension-major (half c of dimension i at t*2048 + (c*64 + i)*16, slot r
    is nibble r % 8 of word (r % 32) / 8)."""
    t, r = divmod(int(s), 64)
    out = np.empty(64, np.uint8)
    if plane == "k":
        for c in range(2):
            off = t * 2048 + (c * 64 + r) * 16
            words = region[off:off + 16].view(np.uint32)
            for wi in range(4):
                w = int(words[wi])
                for j in range(8):
                    out[8 * (4 * c + wi) + j] = ((w >> (3 * j)) & 7) | (((w >> (24 + j)) & 1) << 3)
    else:
        c, wi, nib = r // 32, (r % 32) // 8, r % 8
        for i in range(64):
            off = t * 2048 + (c * 64 + i) * 16 + wi * 4
            w = int(region[off:off + 4].view(np.uint32)[0])
            out[i] = (w >> (4 * nib)) & 15
    return out


def fp16_ulp(x):
    """Spacing of binary16 at |x| (subnormal spacing near 0)."""
    a = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -14)
    return 2.0 ** (np.floor(np.log2(a)) - 10)


def threshold_distance(case, oc_flags, li, b, j, h, is_key):
    x = (case.k if is_key else case.v)[li, b, j, h].astype(np.float32)
    l = case.layer0 + li
    xh = oracle.rotated_input(x, is_key, int(case.pos0[b]) + j, case.cs_host, case.pi[l, h],
                              half=bool(oc_flags & tq.ROPE_HALF), rotate_v=bool(oc_flags & tq.V_ROTATE))
    xd = xh.astype(np.float64)
    u = xd * 8.0 / np.linalg.norm(xd)
    lut = (case.lut_k if is_key else case.lut_v)[l, h].astype(np.float64)
    t = 0.5 * (lut[:-1] + lut[1:])
    return np.min(np.abs(u[:, None] - t[None, :]), axis=1)


def assert_agree_up_to_threshold_rounding(case, got, ref, B, T, H, tokens=None):
    """Two caches quantized from the same raw inputs by two binary32 paths
    (RoPE and rotation summed in different orders): the fp16 norms agree to
    one ulp and a code differs only where the exact coordinate sits within
    rounding of a decision threshold, by one level."""
    ng = got.s.view(np.float16).astype(np.float64)
    no = ref.s.view(np.float16).astype(np.float64)
    assert np.all(np.abs(ng - no) <= fp16_ulp(no) + 1e-12)
    code_diff = sign_diff = total = 0
    for b in range(B):
        for j in (range(T) if tokens is None else tokens):
            s = int(case.slot0[b]) + j
            for h in range(H):
                for is_key, which in ((True, "k"), (False, "v")):
                    ng_ = unpack_slot(got.region(which, 0, h), s, which)
                    no_ = unpack_slot(ref.region(which, 0, h), s, which)
                    total += 64
                    bad = (ng_ & 7) != (no_ & 7)
                    sign_diff += int(((ng_ >> 3) != (no_ >> 3)).sum())
                    if bad.any():
                        code_diff += int(bad.sum())
                        dist = threshold_distance(case, case.flags, 0, b, j, h, is_key)
                        assert np.all(dist[bad] < 1e-4), (b, j, h, which, dist[bad])
                        assert np.all(np.abs((ng_[bad] & 7).astype(int) - (no_[bad] & 7)) == 1)
    assert code_diff <= 1e-3 * total
    # a sign bit follows the residual: it may flip with a code, or where its
    # projection is within rounding of zero
    assert sign_diff <= 64 * code_diff + 1e-4 * total


def unpack_planes(k_region: np.ndarray, v_region: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """All nibbles (idx | sign << 3) of one (layer, head) region, [slots][64]
    for keys and values, decoded with NumPy from the documented layout (see
    unpack_slot)."""
    kw = np.ascontiguousarray(k_region).view(np.uint32).reshape(-1, 2, 64, 4)      # [tile][c][r][wi]
    nt = kw.shape[0]
    j = np.arange(8, dtype=np.uint32)
    # key word w = 4c + wi of slot (tile, r): dims 8w + j
    kw = kw.transpose(0, 2, 1, 3).reshape(nt, 64, 8)                                # [tile][r][w]
    idx = (kw[..., None] >> (3 * j)) & 7
    sgn = (kw[..., None] >> (24 + j)) & 1
    knib = (idx | (sgn << 3)).reshape(nt * 64, 64).astype(np.uint8)
    vw = np.ascontiguousarray(v_region).view(np.uint32).reshape(-1, 2, 64, 4)       # [tile][c][i][wi]
    nib = (vw[..., None] >> (4 * j)) & 15                                           # [tile][c][i][wi][n]
    # slot r = 32c + 8wi + n of dimension i
    vnib = nib.transpose(0, 1, 3, 4, 2).reshape(nt * 64, 64).astype(np.uint8)
    return knib, vnib


def assert_region_agrees(got_k, got_v, got_s, ref_k, ref_v, ref_s, n, rotated_of):
    """The first n slots of one (layer, head) region written by the GPU and by
    the oracle from the same raw tokens: fp16 norms within one ulp; codes
    equal, or one level apart where the oracle's fp64 coordinate lies within
    rounding of a threshold (rotated_of(slot, is_key) -> (x^ fp32, table));
    sign bits differ only with a code or within rounding of zero.
    Returns (codes compared, codes differing)."""
    gs = got_s.reshape(-1, 4)[:n].view(np.float16).astype(np.float64)
    os_ = ref_s.reshape(-1, 4)[:n].view(np.float16).astype(np.float64)
    for col in (0, 2):
        assert np.all(np.abs(gs[:, col] - os_[:, col]) <= fp16_ulp(os_[:, col]) + 1e-12), col
    gk, gv = unpack_planes(got_k, got_v)
    rk, rv = unpack_planes(ref_k, ref_v)
    total = diff = sdiff = 0
    for is_key, g_, r_ in ((True, gk[:n], rk[:n]), (False, gv[:n], rv[:n])):
        total += g_.size
        bad = (g_ & 7) != (r_ & 7)
        sdiff += int(((g_ >> 3) != (r_ >> 3)).sum())
        for s in np.nonzero(bad.any(axis=1))[0]:
            xh, lut = rotated_of(int(s), is_key)
            xd = xh.astype(np.float64)
            u = xd * 8.0 / np.linalg.norm(xd)
            t = 0.5 * (lut[:-1].astype(np.float64) + lut[1:])
            dist = np.min(np.abs(u[:, None] - t[None, :]), axis=1)
            b = bad[s]
            assert np.all(dist[b] < 1e-4), (int(s), is_key, dist[b])
            assert np.all(np.abs((g_[s][b] & 7).astype(int) - (r_[s][b] & 7)) == 1)
        diff += int(bad.sum())
    assert diff <= 1e-3 * total
    assert sdiff <= 64 * diff + 1e-4 * total
    return total, diff
