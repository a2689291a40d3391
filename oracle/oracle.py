"""CPU oracle of the TurboESM KV-cache path (arXiv 2603.26110).

TEST INFRASTRUCTURE ONLY: the slow, obviously-correct reference that the GPU
library is checked against. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import it. It shares no code with the GPU
library and never imports it.

Contents
  C core (``tq_oracle.c``, loaded through ctypes):
    rope_table, rotated_input, quantize_vector, quantize_pack, decode, dequantize,
    f32_to_f16 / f16_to_f32, pack/unpack of one slot.
  NumPy / SciPy:
    lloyd_max_gaussian  3-bit Lloyd-Max levels for N(0, 1)     (Sec. 3.3, Eq. 5)
    kmeans_1d           1-D Lloyd iteration on samples          (Sec. 4.1, LUT calibration)
    calibrate_rotation  Pi = V^T of the SVD of post-RoPE keys   (Sec. 3.2)
    calibrate_ebar      per-head mean |u - c(u)| of a table      (Sec. 3.4, Eq. 7)
    qjl_estimate        sqrt(pi/2)/m ||r|| <S y, sign(S r)>     (Sec. 3.4, projected form)
    paper_memory_table  the accounting of Table 4               (Sec. 5.2)
Parity status: all functions are pinned by ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tq_oracle.c")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(BUILD_DIR, "libtq_oracle.so")

D = 64
# Flag bits, as documented for the library's tq_params.flags.
V_ROTATE, V_QJL, QJL_PAPER, ROPE_HALF, INPUT_ROTATED = 1, 2, 4, 8, 16
SIGN_NONE, SIGN_PROJECTED, SIGN_ELEMENT = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the C core with gcc (binary32 steps need -ffp-contract=off)."""
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    os.makedirs(BUILD_DIR, exist_ok=True)
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-shared", "-fPIC", SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i32, i64, u32, dbl = ctypes.c_int, ctypes.c_int64, ctypes.c_uint32, ctypes.c_double
        L.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.orc_f16_to_f32.restype = ctypes.c_float
        L.orc_f32_to_f16.argtypes = [ctypes.c_float]
        L.orc_f32_to_f16.restype = ctypes.c_uint16
        L.orc_rope_table.argtypes = [i32, dbl, P]
        L.orc_rope_apply.argtypes = [P, P, i32, P]
        L.orc_rotated_input.argtypes = [P, i32, i32, P, i32, P, i32, P]
        L.orc_quantize_vector.argtypes = [P, P, P, i32, P, P, P]
        L.orc_pack_slot.argtypes = [P, i64, P]
        L.orc_unpack_slot.argtypes = [P, i64, P]
        L.orc_pack_slot_v.argtypes = [P, i64, P]
        L.orc_unpack_slot_v.argtypes = [P, i64, P]
        L.orc_quantize_pack.argtypes = [i32, i32, i64, u32, P, i32, P, P, i32, i32,
                                        i32, i32, P, P, P, P, P, P, P, P, P]
        L.orc_decode.argtypes = [i32, i32, i64, u32, dbl, P, i32, P, i32, i32, i32,
                                 P, P, P, P, P, P, P, P, P, P, P, P, i64, i32, P]
        L.orc_dequantize.argtypes = [i32, i32, i64, u32, i32, i32, i32, P, P, i32,
                                     P, P, P, P, P, P, P, P, P]
        L.orc_set_threads.argtypes = [i32]
        L.orc_max_threads.restype = i32
        _lib = L
    return _lib


def set_threads(n: int) -> None:
    """Threads of the oracle's loops over units (timing only)."""
    lib().orc_set_threads(int(n))


def max_threads() -> int:
    return int(lib().orc_max_threads())


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# fp16 helpers (IEEE binary16, round to nearest even)
# --------------------------------------------------------------------------
def f32_to_f16_bits(x) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    f = lib().orc_f32_to_f16
    for i, v in enumerate(x.reshape(-1)):
        out.reshape(-1)[i] = f(float(v))
    return out


def f16_bits_to_f32(h) -> np.ndarray:
    h = np.asarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float32)
    f = lib().orc_f16_to_f32
    for i, v in enumerate(h.reshape(-1)):
        out.reshape(-1)[i] = f(int(v))
    return out


# --------------------------------------------------------------------------
# RoPE (Sec. 2.1, Eq. 1-2) and the RoPE-first rotation (Sec. 3.1, Eq. 4)
# --------------------------------------------------------------------------
def rope_table(positions: int, base: float = 10000.0) -> np.ndarray:
    """[positions][32][2] fp32 (cos, sin) of p * base^(-2m/64), fp64 before rounding."""
    cs = np.empty((positions, 32, 2), dtype=np.float32)
    lib().orc_rope_table(positions, float(base), _p(cs))
    return cs


def rope_apply(x, pos: int, cs: np.ndarray, half: bool = False) -> np.ndarray:
    """R_{theta,pos} x in fp64 for one 64-vector."""
    xin = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty(D, dtype=np.float64)
    row = np.ascontiguousarray(cs[pos], dtype=np.float32)
    lib().orc_rope_apply(_p(xin), _p(row), int(half), _p(y))
    return y


def rotated_input(x, is_key: bool, pos: int, cs, pi, half=False, rotate_v=True):
    """x^ as binary32: Pi R_pos k for keys, Pi v (or v) for values."""
    xin = _f32(x)
    out = np.empty(D, dtype=np.float32)
    lib().orc_rotated_input(_p(xin), int(is_key), int(pos), _p(_f32(cs)), int(half),
                            _p(_f32(pi)), int(rotate_v), _p(out))
    return out


# --------------------------------------------------------------------------
# Quantizer (Sec. 3.3-3.4) and packing (Sec. 4.2)
# --------------------------------------------------------------------------
def quantize_vector(xhat, lut, S, sign_mode=SIGN_PROJECTED):
    """(nibbles[64] uint8, n16 bits, g16 bits) of one rotated vector."""
    nib = np.empty(D, dtype=np.uint8)
    n16 = ctypes.c_uint16()
    g16 = ctypes.c_uint16()
    lib().orc_quantize_vector(_p(_f32(xhat)), _p(_f32(lut)), _p(_f32(S)), int(sign_mode),
                              _p(nib), ctypes.byref(n16), ctypes.byref(g16))
    return nib, n16.value, g16.value


def pack_slot(region: np.ndarray, slot: int, nib, plane: str = "k") -> None:
    """Write one slot's 64 nibbles into a (layer, head) region of the K plane
    (token-major tiles) or the V plane (dimension-major tiles)."""
    f = lib().orc_pack_slot if plane == "k" else lib().orc_pack_slot_v
    f(_p(region), int(slot), _p(np.ascontiguousarray(nib, np.uint8)))


def unpack_slot(region: np.ndarray, slot: int, plane: str = "k") -> np.ndarray:
    nib = np.empty(D, dtype=np.uint8)
    f = lib().orc_unpack_slot if plane == "k" else lib().orc_unpack_slot_v
    f(_p(np.ascontiguousarray(region)), int(slot), _p(nib))
    return nib


class Cache:
    """Host copy of a packed cache: [L][H][slots] of 32 + 32 + 8 bytes."""

    def __init__(self, L: int, H: int, slots: int):
        assert slots % 64 == 0 and slots > 0
        self.L, self.H, self.slots = L, H, slots
        self.k = np.zeros(L * H * slots * 32, dtype=np.uint8)
        self.v = np.zeros(L * H * slots * 32, dtype=np.uint8)
        self.s = np.zeros(L * H * slots * 4, dtype=np.uint16)

    def region(self, which: str, l: int, h: int) -> np.ndarray:
        n = self.slots * 32
        base = (l * self.H + h) * n
        return (self.k if which == "k" else self.v)[base:base + n]

    def scalars(self, l: int, h: int) -> np.ndarray:
        base = (l * self.H + h) * self.slots * 4
        return self.s[base:base + self.slots * 4].reshape(self.slots, 4)


def quantize_pack(cache: Cache, flags: int, cs, k, v, pos0, slot0, pi, lut_k, lut_v, S,
                  layer0: int = 0) -> None:
    """Prefill quantize-and-pack. k, v: [nl][B][T][H][64] (values of the io dtype)."""
    k = _f32(k)
    v = _f32(v)
    nl, B, T, H, d = k.shape
    assert d == D and H == cache.H and v.shape == k.shape
    cs = _f32(cs)
    pos0 = np.ascontiguousarray(pos0, dtype=np.int32)
    slot0 = np.ascontiguousarray(slot0, dtype=np.int64)
    lib().orc_quantize_pack(cache.L, cache.H, cache.slots, int(flags), _p(cs), cs.shape[0],
                            _p(k), _p(v), B, T, layer0, nl, _p(pos0), _p(slot0),
                            _p(_f32(pi)), _p(_f32(lut_k)), _p(_f32(lut_v)), _p(_f32(S)),
                            _p(cache.k), _p(cache.v), _p(cache.s))


def decode(cache: Cache, flags: int, cs, q, q_pos, seq_slot0, seq_len, pi, lut_k, lut_v, S,
           ebar=None, softmax_scale: float = 0.125, layer0: int = 0, units=None,
           twostep: bool = False) -> np.ndarray:
    """Decode attention, fp64. q: [nl][B][H][64]. Returns [nl][B][H][64] float64.
    ``units`` optionally lists flat unit indices (li*B + b)*H + h to compute
    (others are left NaN)."""
    q = _f32(q)
    nl, B, H, d = q.shape
    assert d == D and H == cache.H
    cs = _f32(cs)
    out = np.full((nl, B, H, D), np.nan, dtype=np.float64)
    qp = np.ascontiguousarray(q_pos, dtype=np.int32)
    s0 = np.ascontiguousarray(seq_slot0, dtype=np.int64)
    sl = np.ascontiguousarray(seq_len, dtype=np.int32)
    eb = _f32(ebar) if ebar is not None else None
    if units is not None:
        units = np.ascontiguousarray(units, dtype=np.int64)
    lib().orc_decode(cache.L, cache.H, cache.slots, int(flags), float(np.float32(softmax_scale)),
                     _p(cs), cs.shape[0], _p(q), B, layer0, nl, _p(qp), _p(s0), _p(sl),
                     _p(_f32(pi)), _p(_f32(lut_k)), _p(_f32(lut_v)), _p(_f32(S)),
                     _p(eb) if eb is not None else None,
                     _p(cache.k), _p(cache.v), _p(cache.s),
                     _p(units) if units is not None else None,
                     0 if units is None else len(units), int(twostep), _p(out))
    return out


def dequantize(cache: Cache, flags: int, seq_slot0, seq_len, max_len: int, lut_k, lut_v, S,
               ebar=None, layer0: int = 0, nl: int | None = None):
    """The dequantized keys and values of every cached token (the first step of
    a dequantize-then-attend path), fp64 [nl][B][H][max_len][64] each:
    k~ = (n_k/8)(c_K[idx] + alpha g_k S^T(2s - 1)) (per-element form:
    ebar_K (2s - 1)), v~ = (n_v/8)(c_V[idx] + the V residual estimate with
    V_QJL), so that q^ . k~ is the decode score and v~ the decoded value.
    Rows past a sequence's length (or of an invalid sequence) are NaN."""
    s0 = np.ascontiguousarray(seq_slot0, dtype=np.int64)
    sl = np.ascontiguousarray(seq_len, dtype=np.int32)
    B = len(sl)
    nl = cache.L - layer0 if nl is None else nl
    H = cache.H
    ko = np.full((nl, B, H, max_len, D), np.nan, dtype=np.float64)
    vo = np.full((nl, B, H, max_len, D), np.nan, dtype=np.float64)
    eb = _f32(ebar) if ebar is not None else None
    lib().orc_dequantize(cache.L, H, cache.slots, int(flags), B, layer0, nl, _p(s0), _p(sl),
                         int(max_len), _p(_f32(lut_k)), _p(_f32(lut_v)), _p(_f32(S)),
                         _p(eb) if eb is not None else None, _p(cache.k), _p(cache.v), _p(cache.s),
                         _p(ko), _p(vo))
    return ko, vo


# --------------------------------------------------------------------------
# Lloyd-Max levels (Sec. 3.3, Eq. 5) and 1-D k-means LUT calibration (Sec. 4.1)
# --------------------------------------------------------------------------
def lloyd_max_gaussian(levels: int = 8, tol: float = 1e-15, max_iter: int = 100000):
    """MSE-optimal scalar quantizer of N(0, 1) by the Lloyd-Max iteration:
    thresholds at midpoints of neighbouring levels, each level the conditional
    mean of its cell, c_k = (phi(t_{k-1}) - phi(t_k)) / (Phi(t_k) - Phi(t_{k-1})).
    Returns (levels, thresholds, mse), all float64."""
    from scipy.stats import norm
    c = np.linspace(-2.0, 2.0, levels)
    for _ in range(max_iter):
        t = 0.5 * (c[:-1] + c[1:])
        edges = np.concatenate(([-np.inf], t, [np.inf]))
        mass = norm.cdf(edges[1:]) - norm.cdf(edges[:-1])
        cn = (norm.pdf(edges[:-1]) - norm.pdf(edges[1:])) / mass
        delta = np.max(np.abs(cn - c))
        c = cn
        if delta < tol:
            break
    t = 0.5 * (c[:-1] + c[1:])
    edges = np.concatenate(([-np.inf], t, [np.inf]))
    mass = norm.cdf(edges[1:]) - norm.cdf(edges[:-1])
    mse = 1.0 - float(np.sum(mass * c * c))   # E[X^2] - sum P_k c_k^2 at the centroid condition
    return c, t, mse


def assign_levels(x, c) -> np.ndarray:
    """Nearest level index, ties to the lower level (midpoint thresholds)."""
    t = 0.5 * (np.asarray(c[:-1], np.float64) + np.asarray(c[1:], np.float64))
    return np.searchsorted(t, np.asarray(x, np.float64), side="left")


def kmeans_1d(samples, init, max_iter: int = 100, tol: float = 1e-7):
    """1-D Lloyd iteration (k-means) on samples, fp64 sums; an empty cell keeps
    its level. Returns ascending levels (float64)."""
    x = np.asarray(samples, dtype=np.float64).reshape(-1)
    c = np.sort(np.asarray(init, dtype=np.float64))
    for _ in range(max_iter):
        idx = assign_levels(x, c)
        sums = np.bincount(idx, weights=x, minlength=len(c))
        cnt = np.bincount(idx, minlength=len(c))
        cn = np.where(cnt > 0, sums / np.maximum(cnt, 1), c)
        delta = np.max(np.abs(cn - c))
        c = np.sort(cn)
        if delta < tol:
            break
    return c


def normalized_coordinates(x, pi=None) -> np.ndarray:
    """The coordinates a table quantizes: u = 8 x^ / ||x^|| with x^ = Pi x in
    fp64 (x^ = x when pi is None); a zero vector gives zeros, as the
    quantizer's inv = 0 does. x: [n][64]. Returns [n][64] float64."""
    X = np.asarray(x, dtype=np.float64).reshape(-1, D)
    xh = X if pi is None else X @ np.asarray(pi, dtype=np.float64).T
    n = np.sqrt(np.sum(xh * xh, axis=1, keepdims=True))
    return np.where(n > 0, xh * (8.0 / np.where(n > 0, n, 1.0)), 0.0)


def calibrate_lut(x, pi, init, max_iter: int = 100, tol: float = 1e-7) -> np.ndarray:
    """Calibrated 8-level table of one head (Sec. 3.3, calibrated LUTs): the
    1-D Lloyd iteration of kmeans_1d on every normalized coordinate of the
    calibration vectors x [n][64] (rotated by pi unless None)."""
    return kmeans_1d(normalized_coordinates(x, pi).reshape(-1), init, max_iter, tol)


def calibrate_ebar(x, pi, lut) -> float:
    """Per-head mean absolute residual ebar of the per-element residual
    correction (Sec. 3.4, Eq. 7; the correction adds sign(r_i) ebar): the mean
    of |u - c[idx(u)]| over every normalized coordinate u of the calibration
    vectors x [n][64] (rotated by pi unless None), idx by the midpoint rule of
    assign_levels, fp64 throughout."""
    u = normalized_coordinates(x, pi).reshape(-1)
    c = np.asarray(lut, dtype=np.float64)
    return float(np.mean(np.abs(u - c[assign_levels(u, c)])))


# --------------------------------------------------------------------------
# Head-wise SVD calibration (Sec. 3.2)
# --------------------------------------------------------------------------
def canonical_signs(rows: np.ndarray) -> np.ndarray:
    """Flip each row so its largest-magnitude entry (lowest index on ties) is positive."""
    rows = np.array(rows, dtype=np.float64)
    for i in range(rows.shape[0]):
        j = int(np.argmax(np.abs(rows[i])))   # argmax returns the first maximum
        if rows[i, j] < 0:
            rows[i] = -rows[i]
    return rows


def calibrate_rotation(X):
    """X: [ncal][64] post-RoPE keys (not centered). X = U S V^T, Pi = V^T with
    rows by descending singular value, signs canonical. Returns (Pi fp32, sigma fp64)."""
    X = np.asarray(X, dtype=np.float64)
    _, s, vt = np.linalg.svd(X, full_matrices=False)
    order = np.argsort(-s, kind="stable")
    pi = canonical_signs(vt[order])
    return pi.astype(np.float32), s[order]


# --------------------------------------------------------------------------
# QJL estimator (Sec. 3.4; projected form) and memory accounting (Table 4)
# --------------------------------------------------------------------------
def qjl_estimate(y, r, S) -> float:
    """sqrt(pi/2)/m * ||r|| * <S y, sign(S r)> with sign(0) = +1, m = rows of S."""
    S = np.asarray(S, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    m = S.shape[0]
    sg = np.where(S @ r < 0, -1.0, 1.0)
    return float(np.sqrt(np.pi / 2) / m * np.linalg.norm(r) * np.dot(S @ y, sg))


def cache_bytes(L: int, H: int, slots: int) -> int:
    """72 bytes per cached token-head: 32 B K nibbles (3-bit code + 1 QJL bit),
    32 B V nibbles, 4 fp16 scalars."""
    return L * H * slots * (32 + 32 + 8)


def paper_memory_table(L: int, H: int, d: int, seq: int) -> dict:
    """Bytes of the memory breakdown of Table 4 (Sec. 5.2): fp32 K+V baseline
    (Eq. 3), 3-bit codes in 32-bit containers of 8, and 1-bit K signs."""
    fp32 = 2 * L * H * d * seq * 4
    packed = 2 * L * H * seq * (d // 8) * 4
    signs = L * H * seq * d // 8
    return {"fp32": fp32, "packed_kv": packed, "qjl_signs": signs,
            "codes_and_signs": packed + signs}
