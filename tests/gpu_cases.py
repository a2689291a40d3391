"""Shared helpers of the GPU parity tests: seeded inputs for both sides,
running the library through its C ABI, moving the oracle's cache to the
device, and reading the device cache back for comparison with the oracle's
(never as an oracle input)."""
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


def to_oracle(cache: tq.Cache) -> oracle.Cache:
    oc = oracle.Cache(cache.num_layers, cache.num_heads, cache.slots)
    oc.k[:] = cache.k_codes.cpu().numpy()
    oc.v[:] = cache.v_codes.cpu().numpy()
    oc.s[:] = cache.scalars.cpu().numpy().view(np.uint16)
    return oc


def fp16_ulp(x):
    """Spacing of binary16 at |x| (subnormal spacing near 0)."""
    a = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -14)
    return 2.0 ** (np.floor(np.log2(a)) - 10)
