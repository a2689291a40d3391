"""TurboESM 3-bit KV-cache quantizer and fused decode attention for MI355X.

Thin ctypes binding of ``libturboesm.so`` (C ABI in ``include/turboesm.h``).
PyTorch provides device memory and the current HIP stream; every step of the
path runs in the library's HIP kernels. If the library is not built, calls
raise ``RuntimeError`` (there is no fallback path).

Entry points (same names as the C ABI without the ``tq_`` prefix):
    rope_table, quantize_pack, decode_attend, decode_attend_noalloc, decode_step, dequantize,
    decode_workspace_bytes, calibrate_rotation, calibrate_lut, calibrate_ebar, set_step_wait_limit,
    cache_bytes, last_error, version
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

__all__ = [
    "Params", "Cache", "TQError", "rope_table", "quantize_pack", "decode_attend", "decode_step", "dequantize",
    "decode_attend_noalloc", "decode_workspace_bytes", "calibrate_rotation", "calibrate_lut", "calibrate_ebar", "set_step_wait_limit",
    "read_probe",
    "cache_bytes", "last_error", "version",
    "V_ROTATE", "V_QJL", "QJL_PAPER", "ROPE_HALF", "INPUT_ROTATED", "OUT_FP32", "lib_path",
]

V_ROTATE, V_QJL, QJL_PAPER, ROPE_HALF, INPUT_ROTATED, OUT_FP32 = 1, 2, 4, 8, 16, 32
_F32, _F16 = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libturboesm.so")


class TQError(RuntimeError):
    pass


class _Params(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("num_heads", ctypes.c_int32), ("io_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("softmax_scale", ctypes.c_float),
                ("rope_cs", ctypes.c_void_p), ("rope_positions", ctypes.c_int32)]


class _Cache(ctypes.Structure):
    _fields_ = [("k_codes", ctypes.c_void_p), ("v_codes", ctypes.c_void_p),
                ("scalars", ctypes.c_void_p), ("slots", ctypes.c_int64)]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(lib_path):
        raise RuntimeError(f"{lib_path} is not built; run __graft_entry__.build() "
                           "or python -m paper_2603_26110_amd.build")
    L = ctypes.CDLL(lib_path)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.tq_last_error.restype = ctypes.c_char_p
    L.tq_version.restype = ctypes.c_char_p
    L.tq_cache_bytes.argtypes = [i32, i32, i64]
    L.tq_cache_bytes.restype = i64
    L.tq_rope_table.argtypes = [P, i32, ctypes.c_double, P]
    L.tq_rope_table.restype = i32
    L.tq_quantize_pack.argtypes = [P, P, P, P, i32, i32, i32, i32, P, P, P, P, P, P, P, P]
    L.tq_quantize_pack.restype = i32
    L.tq_quantize_pack_ragged.argtypes = [P, P, P, P, i32, i32, P, i32, i32, P, P, P, P, P, P, P, P]
    L.tq_quantize_pack_ragged.restype = i32
    L.tq_decode_attend.argtypes = [P, P, P, i32, i32, i32, P, P, P, i32, P, P, P, P, P, P, P, sz, P]
    L.tq_decode_attend.restype = i32
    L.tq_decode_step.argtypes = [P, P, P, P, P, i32, i32, i32, P, P, P, i32, P, P, P, P, P, P, P, sz, P]
    L.tq_decode_step.restype = i32
    L.tq_dequantize.argtypes = [P, P, i32, i32, i32, P, P, i32, P, P, P, P, P, P, P]
    L.tq_dequantize.restype = i32
    L.tq_decode_workspace_bytes.argtypes = [P, i32, i32, i32]
    L.tq_decode_workspace_bytes.restype = sz
    L.tq_calibrate_rotation.argtypes = [P, i32, i32, P, P, P]
    L.tq_calibrate_lut.argtypes = [P, i32, i32, P, P, i32, ctypes.c_double, P, P]
    L.tq_calibrate_lut.restype = i32
    L.tq_calibrate_rotation.restype = i32
    L.tq_calibrate_ebar.argtypes = [P, i32, i32, P, P, P, i32, P]
    L.tq_calibrate_ebar.restype = i32
    L.tq_decode_attend_noalloc.argtypes = [P, P, P, i32, i32, i32, P, P, P, i32, P, P, P, P, P, P, P]
    L.tq_decode_attend_noalloc.restype = i32
    L.tq_set_step_wait_limit.argtypes = [i32]
    L.tq_set_step_wait_limit.restype = i32
    L.tq_read_probe.argtypes = [P, i64, i32, P, P]
    L.tq_read_probe.restype = i32
    _lib = L
    return L


def last_error() -> str:
    return _load().tq_last_error().decode()


def version() -> str:
    return _load().tq_version().decode()


def _check(status: int) -> None:
    if status != 0:
        raise TQError(f"status {status}: {last_error()}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


@dataclass
class Params:
    """Model-level parameters (tq_params). ``rope_cs`` comes from rope_table()."""
    num_layers: int
    num_heads: int
    rope_cs: torch.Tensor
    io_dtype: torch.dtype = torch.float16
    flags: int = V_ROTATE
    softmax_scale: float = 0.125

    def c(self) -> _Params:
        _dev(self.rope_cs, "rope_cs", torch.float32)
        io = {torch.float16: _F16, torch.float32: _F32}[self.io_dtype]
        return _Params(64, self.num_layers, self.num_heads, io, self.flags, self.softmax_scale,
                       self.rope_cs.data_ptr(), self.rope_cs.shape[0])


class Cache:
    """Packed cache in device memory: [L][H][slots] x (32 B K, 32 B V, 8 B scalars)."""

    def __init__(self, num_layers: int, num_heads: int, slots: int, device="cuda"):
        if slots <= 0 or slots % 64:
            raise ValueError("slots must be a positive multiple of 64")
        n = num_layers * num_heads * slots
        self.num_layers, self.num_heads, self.slots = num_layers, num_heads, slots
        self.k_codes = torch.zeros(n * 32, dtype=torch.uint8, device=device)
        self.v_codes = torch.zeros(n * 32, dtype=torch.uint8, device=device)
        self.scalars = torch.zeros(n * 4, dtype=torch.int16, device=device)

    def c(self) -> _Cache:
        return _Cache(self.k_codes.data_ptr(), self.v_codes.data_ptr(),
                      self.scalars.data_ptr(), self.slots)


def cache_bytes(num_layers: int, num_heads: int, slots: int) -> int:
    return int(_load().tq_cache_bytes(num_layers, num_heads, slots))


def rope_table(positions: int, base: float = 10000.0, device="cuda") -> torch.Tensor:
    """[positions][32][2] fp32 (cos, sin) table built on the GPU."""
    L = _load()
    cs = torch.empty((positions, 32, 2), dtype=torch.float32, device=device)
    _check(L.tq_rope_table(_ptr(cs), positions, float(base), _stream(cs.device)))
    return cs


def quantize_pack(params: Params, cache: Cache, k, v, pos0, slot0, pi, lut_k, lut_v, qjl_s,
                  ebar=None, layer0: int = 0, seq_tokens=None) -> None:
    """k, v: [nlayers][B][T][H][64] (params.io_dtype; fp32 with INPUT_ROTATED).
    seq_tokens (int32 [B], optional): each sequence's token count for a
    ragged batch (tq_quantize_pack_ragged); rows beyond it are padding."""
    L = _load()
    want = torch.float32 if params.flags & INPUT_ROTATED else params.io_dtype
    _dev(k, "k", want)
    _dev(v, "v", want)
    if k.dim() != 5 or k.shape[-1] != 64 or k.shape != v.shape or k.shape[3] != params.num_heads:
        raise ValueError("k and v must be [nlayers][B][T][H][64] with matching shapes")
    nl, B, T = k.shape[:3]
    _dev(pos0, "pos0", torch.int32)
    _dev(slot0, "slot0", torch.int64)
    if pos0.numel() < B or slot0.numel() < B:
        raise ValueError("pos0 and slot0 need B entries")
    for name, t in (("pi", pi), ("lut_k", lut_k), ("lut_v", lut_v), ("qjl_s", qjl_s)):
        _dev(t, name, torch.float32)
    p = params.c()
    c = cache.c()
    if seq_tokens is not None:
        _dev(seq_tokens, "seq_tokens", torch.int32)
        if seq_tokens.numel() < B:
            raise ValueError("seq_tokens needs B entries")
        _check(L.tq_quantize_pack_ragged(ctypes.byref(p), ctypes.byref(c), _ptr(k), _ptr(v), B, T,
                                         _ptr(seq_tokens), layer0, nl, _ptr(pos0), _ptr(slot0), _ptr(pi),
                                         _ptr(lut_k), _ptr(lut_v), _ptr(qjl_s), _ptr(ebar),
                                         _stream(k.device)))
        return
    _check(L.tq_quantize_pack(ctypes.byref(p), ctypes.byref(c), _ptr(k), _ptr(v), B, T, layer0, nl,
                              _ptr(pos0), _ptr(slot0), _ptr(pi), _ptr(lut_k), _ptr(lut_v),
                              _ptr(qjl_s), _ptr(ebar), _stream(k.device)))


def decode_workspace_bytes(params: Params, B: int, nlayers: int, max_len: int) -> int:
    p = params.c()
    return int(_load().tq_decode_workspace_bytes(ctypes.byref(p), B, nlayers, max_len))


def decode_attend(params: Params, cache: Cache, q, q_pos, seq_slot0, seq_len, max_len: int,
                  pi, lut_k, lut_v, qjl_s, ebar=None, layer0: int = 0, out=None,
                  workspace=None) -> torch.Tensor:
    """q: [nlayers][B][H][64]. Returns out [nlayers][B][H][64]."""
    L = _load()
    _dev(q, "q", params.io_dtype)
    if q.dim() != 4 or q.shape[-1] != 64 or q.shape[2] != params.num_heads:
        raise ValueError("q must be [nlayers][B][H][64]")
    nl, B = q.shape[:2]
    _dev(q_pos, "q_pos", torch.int32)
    _dev(seq_slot0, "seq_slot0", torch.int64)
    _dev(seq_len, "seq_len", torch.int32)
    for name, t in (("pi", pi), ("lut_k", lut_k), ("lut_v", lut_v), ("qjl_s", qjl_s)):
        _dev(t, name, torch.float32)
    if ebar is not None:
        _dev(ebar, "ebar", torch.float32)
    out_dtype = torch.float32 if (params.flags & OUT_FP32 or params.io_dtype == torch.float32) \
        else torch.float16
    if out is None:
        out = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    _dev(out, "out", out_dtype)
    need = decode_workspace_bytes(params, B, nl, max_len)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.zeros(need, dtype=torch.uint8, device=q.device)
    p = params.c()
    c = cache.c()
    wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.tq_decode_attend(ctypes.byref(p), ctypes.byref(c), _ptr(q), B, layer0, nl, _ptr(q_pos),
                              _ptr(seq_slot0), _ptr(seq_len), int(max_len), _ptr(pi), _ptr(lut_k),
                              _ptr(lut_v), _ptr(qjl_s), _ptr(ebar), _ptr(out), _ptr(workspace),
                              wsz, _stream(q.device)))
    return out


def decode_attend_noalloc(params: Params, cache: Cache, q, q_pos, seq_slot0, seq_len, max_len: int,
                          pi, lut_k, lut_v, qjl_s, ebar=None, layer0: int = 0, out=None) -> torch.Tensor:
    """decode_attend without a workspace: the library's fixed split-K scratch
    (see tq_decode_attend_noalloc). ``out`` should be passed where nothing may
    be allocated."""
    L = _load()
    _dev(q, "q", params.io_dtype)
    if q.dim() != 4 or q.shape[-1] != 64 or q.shape[2] != params.num_heads:
        raise ValueError("q must be [nlayers][B][H][64]")
    nl, B = q.shape[:2]
    _dev(q_pos, "q_pos", torch.int32)
    _dev(seq_slot0, "seq_slot0", torch.int64)
    _dev(seq_len, "seq_len", torch.int32)
    for name, t in (("pi", pi), ("lut_k", lut_k), ("lut_v", lut_v), ("qjl_s", qjl_s)):
        _dev(t, name, torch.float32)
    if ebar is not None:
        _dev(ebar, "ebar", torch.float32)
    out_dtype = torch.float32 if (params.flags & OUT_FP32 or params.io_dtype == torch.float32) \
        else torch.float16
    if out is None:
        out = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    _dev(out, "out", out_dtype)
    p = params.c()
    c = cache.c()
    _check(L.tq_decode_attend_noalloc(ctypes.byref(p), ctypes.byref(c), _ptr(q), B, layer0, nl, _ptr(q_pos),
                                      _ptr(seq_slot0), _ptr(seq_len), int(max_len), _ptr(pi), _ptr(lut_k),
                                      _ptr(lut_v), _ptr(qjl_s), _ptr(ebar), _ptr(out), _stream(q.device)))
    return out


def dequantize(params: Params, cache: Cache, seq_slot0, seq_len, max_len: int, lut_k, lut_v, qjl_s,
               ebar=None, layer0: int = 0, nlayers: int | None = None, k_out=None, v_out=None):
    """The dequantized fp16 key and value rows of every cached token,
    [nlayers][B][H][max_len][64] each (rows past a sequence's length are not
    written). Returns (k_out, v_out)."""
    L = _load()
    _dev(seq_slot0, "seq_slot0", torch.int64)
    _dev(seq_len, "seq_len", torch.int32)
    for name, t in (("lut_k", lut_k), ("lut_v", lut_v)):
        _dev(t, name, torch.float32)
    if qjl_s is not None:
        _dev(qjl_s, "qjl_s", torch.float32)
    if ebar is not None:
        _dev(ebar, "ebar", torch.float32)
    B = seq_len.numel()
    nl = params.num_layers - layer0 if nlayers is None else nlayers
    shape = (nl, B, params.num_heads, int(max_len), 64)
    dev = seq_len.device
    if k_out is None:
        k_out = torch.empty(shape, dtype=torch.float16, device=dev)
    if v_out is None:
        v_out = torch.empty(shape, dtype=torch.float16, device=dev)
    for name, t in (("k_out", k_out), ("v_out", v_out)):
        _dev(t, name, torch.float16)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must be {list(shape)}")
    p = params.c()
    c = cache.c()
    _check(L.tq_dequantize(ctypes.byref(p), ctypes.byref(c), B, layer0, nl, _ptr(seq_slot0), _ptr(seq_len),
                           int(max_len), _ptr(lut_k), _ptr(lut_v), _ptr(qjl_s), _ptr(ebar), _ptr(k_out),
                           _ptr(v_out), _stream(dev)))
    return k_out, v_out


def decode_step(params: Params, cache: Cache, q, k, v, pos, seq_slot0, seq_len, max_len: int,
                pi, lut_k, lut_v, qjl_s, ebar=None, layer0: int = 0, out=None,
                workspace=None) -> torch.Tensor:
    """Append the new token (k, v) and attend with q, all [nlayers][B][H][64].
    seq_len holds the tokens cached before the step; the step attends over
    seq_len + 1 of them. Returns out [nlayers][B][H][64]."""
    L = _load()
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, params.io_dtype)
    if q.dim() != 4 or q.shape[-1] != 64 or q.shape[2] != params.num_heads:
        raise ValueError("q must be [nlayers][B][H][64]")
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("k and v must have the shape of q")
    nl, B = q.shape[:2]
    _dev(pos, "pos", torch.int32)
    _dev(seq_slot0, "seq_slot0", torch.int64)
    _dev(seq_len, "seq_len", torch.int32)
    for name, t in (("pi", pi), ("lut_k", lut_k), ("lut_v", lut_v), ("qjl_s", qjl_s)):
        _dev(t, name, torch.float32)
    if ebar is not None:
        _dev(ebar, "ebar", torch.float32)
    out_dtype = torch.float32 if (params.flags & OUT_FP32 or params.io_dtype == torch.float32) \
        else torch.float16
    if out is None:
        out = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    _dev(out, "out", out_dtype)
    need = decode_workspace_bytes(params, B, nl, max_len)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.zeros(need, dtype=torch.uint8, device=q.device)
    p = params.c()
    c = cache.c()
    wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.tq_decode_step(ctypes.byref(p), ctypes.byref(c), _ptr(q), _ptr(k), _ptr(v), B, layer0, nl,
                            _ptr(pos), _ptr(seq_slot0), _ptr(seq_len), int(max_len), _ptr(pi),
                            _ptr(lut_k), _ptr(lut_v), _ptr(qjl_s), _ptr(ebar), _ptr(out),
                            _ptr(workspace), wsz, _stream(q.device)))
    return out


def calibrate_lut(x: torch.Tensor, pi=None, init=None, max_iter: int = 100,
                  tol: float = 1e-7) -> torch.Tensor:
    """x: [nheads][ncal][64] fp32 calibration vectors (post-RoPE keys or values),
    pi: [nheads][64][64] rotations or None, init: 8 ascending starting levels
    (default: the Gaussian 8-level table). Returns the tables [nheads][8]."""
    L = _load()
    _dev(x, "x", torch.float32)
    if x.dim() != 3 or x.shape[-1] != 64:
        raise ValueError("x must be [nheads][ncal][64]")
    nh, ncal = x.shape[:2]
    if pi is not None:
        _dev(pi, "pi", torch.float32)
        if tuple(pi.shape) != (nh, 64, 64):
            raise ValueError("pi must be [nheads][64][64]")
    from .synth import GAUSS_LEVELS_MAX1960
    init_h = (GAUSS_LEVELS_MAX1960 if init is None else init)
    init_arr = (ctypes.c_float * 8)(*[float(v) for v in init_h])
    out = torch.empty((nh, 8), dtype=torch.float32, device=x.device)
    _check(L.tq_calibrate_lut(_ptr(x), nh, ncal, _ptr(pi), ctypes.cast(init_arr, ctypes.c_void_p),
                              int(max_iter), float(tol), _ptr(out), _stream(x.device)))
    return out


def calibrate_ebar(x: torch.Tensor, lut: torch.Tensor, pi=None, out=None, stride: int = 1) -> torch.Tensor:
    """x: [nheads][ncal][64] fp32 calibration vectors (post-RoPE keys with
    lut_k, or values with lut_v), lut: [nheads][8] tables, pi: [nheads][64][64]
    rotations or None. Returns the per-head mean absolute residual; with a
    contiguous fp32 ``out`` and ``stride`` the value of head h is written to
    out.view(-1)[h * stride] (e.g. out = ebar.view(-1)[1:] and stride 2 fill
    the V column of an [L][H][2] array), else a new [nheads] tensor."""
    L = _load()
    _dev(x, "x", torch.float32)
    if x.dim() != 3 or x.shape[-1] != 64:
        raise ValueError("x must be [nheads][ncal][64]")
    nh, ncal = x.shape[:2]
    _dev(lut, "lut", torch.float32)
    if tuple(lut.shape) != (nh, 8):
        raise ValueError("lut must be [nheads][8]")
    if pi is not None:
        _dev(pi, "pi", torch.float32)
        if tuple(pi.shape) != (nh, 64, 64):
            raise ValueError("pi must be [nheads][64][64]")
    if out is None:
        out = torch.empty(nh, dtype=torch.float32, device=x.device)
        stride = 1
    else:
        _dev(out, "out", torch.float32)
    if stride < 1 or out.numel() < (nh - 1) * stride + 1:
        raise ValueError("out is too small for nheads at this stride")
    _check(L.tq_calibrate_ebar(_ptr(x), nh, ncal, _ptr(pi), _ptr(lut), _ptr(out), int(stride),
                               _stream(x.device)))
    return out


def read_probe(data: torch.Tensor, blocks: int, sink: torch.Tensor) -> None:
    """Streaming read of every byte of `data` (a measurement, not part of the
    method; see tq_read_probe). sink: int32 device tensor of >= blocks words."""
    L = _load()
    if not data.is_cuda or not data.is_contiguous():
        raise ValueError("data must be a contiguous device tensor")
    _dev(sink, "sink", torch.int32)
    if sink.numel() < blocks:
        raise ValueError("sink must hold >= blocks words")
    _check(L.tq_read_probe(_ptr(data), data.numel() * data.element_size(), int(blocks), _ptr(sink),
                           _stream(data.device)))


def set_step_wait_limit(limit: int) -> int:
    """Bound of a decode step's wait for its appends (tests of the failure
    path; a negative limit restores the default). Returns the previous one."""
    return int(_load().tq_set_step_wait_limit(int(limit)))


def calibrate_rotation(x: torch.Tensor):
    """x: [nheads][ncal][64] fp32 post-RoPE keys. Returns (pi [nheads][64][64], sigma [nheads][64])."""
    L = _load()
    _dev(x, "x", torch.float32)
    if x.dim() != 3 or x.shape[-1] != 64:
        raise ValueError("x must be [nheads][ncal][64]")
    nh, ncal = x.shape[:2]
    pi = torch.empty((nh, 64, 64), dtype=torch.float32, device=x.device)
    sg = torch.empty((nh, 64), dtype=torch.float32, device=x.device)
    _check(L.tq_calibrate_rotation(_ptr(x), nh, ncal, _ptr(pi), _ptr(sg), _stream(x.device)))
    return pi, sg
