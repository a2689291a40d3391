"""The C ABI without a GPU: the built library loads, exports exactly the entry
points the public header declares, agrees with the binding on constants and
struct layout, and rejects bad arguments on the host before anything is
launched (every call here fails validation, so no device code runs)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2603_26110_amd as tq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "turboesm.h")

pytestmark = pytest.mark.skipif(not os.path.exists(tq.lib_path),
                                reason="libturboesm.so is not built (run __graft_entry__.build())")


def _header():
    with open(HEADER) as f:
        return f.read()


def _declared_functions():
    text = re.sub(r"/\*.*?\*/", "", _header(), flags=re.S)
    return sorted(set(re.findall(r"\bTQ_API\b[^;(]*?\b(tq_\w+)\s*\(", text)))


def _defines():
    out = {}
    for name, val in re.findall(r"#define\s+(TQ_\w+)\s+(\(?[-0-9xXa-fA-Fu<\s]+\)?)", _header()):
        out[name] = int(eval(val.replace("u", "")))
    return out


def test_header_declares_the_entry_points():
    assert _declared_functions() == sorted([
        "tq_cache_bytes", "tq_rope_table", "tq_quantize_pack", "tq_quantize_pack_ragged",
        "tq_decode_attend", "tq_decode_step",
        "tq_dequantize", "tq_decode_workspace_bytes", "tq_calibrate_rotation", "tq_calibrate_lut",
        "tq_calibrate_ebar", "tq_set_step_wait_limit", "tq_decode_attend_noalloc", "tq_read_probe",
        "tq_last_error", "tq_version"])


def test_library_exports_exactly_the_declared_symbols():
    out = subprocess.run(["nm", "-D", "--defined-only", tq.lib_path], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(ln.split()[-1] for ln in out.splitlines() if " T " in ln)
    assert exported == _declared_functions()
    lib = ctypes.CDLL(tq.lib_path)
    for name in _declared_functions():
        assert getattr(lib, name) is not None


def test_binding_constants_match_header():
    d = _defines()
    assert (tq.V_ROTATE, tq.V_QJL, tq.QJL_PAPER, tq.ROPE_HALF, tq.INPUT_ROTATED, tq.OUT_FP32) == (
        d["TQ_V_ROTATE"], d["TQ_V_QJL"], d["TQ_QJL_PAPER"], d["TQ_ROPE_HALF"],
        d["TQ_INPUT_ROTATED"], d["TQ_OUT_FP32"])
    assert d["TQ_FLAGS_ALL"] == 0x3F
    assert (tq._F32, tq._F16) == (d["TQ_F32"], d["TQ_F16"])


def test_struct_layout_matches_header():
    # tq_params: 5 x int32, float, pointer (8-aligned), int32 -> 40 bytes on x86-64
    assert ctypes.sizeof(tq._Params) == 40
    assert tq._Params.rope_cs.offset == 24
    assert ctypes.sizeof(tq._Cache) == 32
    assert tq._Cache.slots.offset == 24


def test_version_and_cache_bytes():
    assert tq.version().startswith("turboesm-gfx950")
    # 72 bytes per slot per head (Table 4 accounting: 4-bit K and V containers + norms)
    assert tq.cache_bytes(33, 20, 1024) == 33 * 20 * 1024 * 72
    assert tq.cache_bytes(-1, 20, 1024) == -1


# ------------------------------------------------------------ host validation
FAKE = 0x10000          # a 64 KiB-aligned non-null address that is never dereferenced


def _params(**kw):
    p = dict(head_dim=64, num_layers=2, num_heads=3, io_dtype=1, flags=1, softmax_scale=0.125,
             rope_cs=FAKE, rope_positions=128)
    p.update(kw)
    return tq._Params(p["head_dim"], p["num_layers"], p["num_heads"], p["io_dtype"], p["flags"],
                      p["softmax_scale"], p["rope_cs"], p["rope_positions"])


def _cache(**kw):
    c = dict(k=FAKE, v=FAKE, s=FAKE, slots=128)
    c.update(kw)
    return tq._Cache(c["k"], c["v"], c["s"], c["slots"])


def _quantize(p, c, B=1, T=4, layer0=0, nlayers=1, k=FAKE, v=FAKE, ptrs=FAKE):
    L = tq._load()
    P = ctypes.c_void_p
    return L.tq_quantize_pack(ctypes.byref(p) if p is not None else None,
                              ctypes.byref(c) if c is not None else None, P(k), P(v), B, T,
                              layer0, nlayers, P(ptrs), P(ptrs), P(ptrs), P(ptrs), P(ptrs),
                              P(ptrs), None, None)


def _decode(p, c, B=1, layer0=0, nlayers=1, max_len=64, ws=None, ws_bytes=0, ptrs=FAKE, out=FAKE):
    L = tq._load()
    P = ctypes.c_void_p
    return L.tq_decode_attend(ctypes.byref(p), ctypes.byref(c), P(ptrs), B, layer0, nlayers,
                              P(ptrs), P(ptrs), P(ptrs), max_len, P(ptrs), P(ptrs), P(ptrs),
                              P(ptrs), None, P(out), P(ws) if ws else None, ws_bytes, None)


@pytest.mark.parametrize("kw,code,msg", [
    (dict(head_dim=128), -2, "head_dim"),
    (dict(num_layers=0), -1, "positive"),
    (dict(io_dtype=7), -1, "io_dtype"),
    (dict(flags=0x40), -1, "flag"),
    (dict(rope_cs=0), -1, "rope_cs"),
    (dict(rope_cs=FAKE + 4), -3, "aligned"),
    (dict(rope_positions=0), -1, "rope_positions"),
])
def test_quantize_rejects_bad_params(kw, code, msg):
    assert _quantize(_params(**kw), _cache()) == code
    assert msg in tq.last_error()


@pytest.mark.parametrize("kw,code,msg", [
    (dict(k=0), -1, "NULL"),
    (dict(k=FAKE + 8), -3, "16-byte"),
    (dict(s=FAKE + 4), -3, "8-byte"),
    (dict(slots=100), -5, "multiple of 64"),
    (dict(slots=0), -5, "multiple of 64"),
])
def test_quantize_rejects_bad_cache(kw, code, msg):
    assert _quantize(_params(), _cache(**kw)) == code
    assert msg in tq.last_error()


def test_quantize_argument_checks():
    assert _quantize(None, _cache()) == -1 and "params" in tq.last_error()
    assert _quantize(_params(), None) == -1 and "cache" in tq.last_error()
    assert _quantize(_params(), _cache(), B=-1) == -1
    assert _quantize(_params(), _cache(), layer0=1, nlayers=2) == -2
    assert _quantize(_params(), _cache(), ptrs=0) == -1
    assert _quantize(_params(), _cache(), k=FAKE + 2) == -3
    # nothing to do is success, with nothing launched
    assert _quantize(_params(), _cache(), T=0) == 0
    assert _quantize(_params(), _cache(), nlayers=0) == 0
    assert tq.last_error() == ""


def test_quantize_ragged_argument_checks():
    L = tq._load()
    P = ctypes.c_void_p
    p, c = _params(), _cache()

    def call(tokens, B=2, T=4, ptrs=FAKE):
        return L.tq_quantize_pack_ragged(ctypes.byref(p), ctypes.byref(c), P(FAKE), P(FAKE), B, T,
                                         P(tokens) if tokens else None, 0, 1, P(ptrs), P(ptrs), P(ptrs),
                                         P(ptrs), P(ptrs), P(ptrs), None, None)
    assert call(None) == -1 and "seq_tokens" in tq.last_error()
    assert call(FAKE, B=-1) == -1
    assert call(FAKE, ptrs=0) == -1
    # nothing to do is success, with nothing launched (seq_tokens may then be NULL)
    assert call(None, T=0) == 0 and tq.last_error() == ""


def test_decode_argument_checks():
    assert _decode(_params(flags=1 | 16), _cache()) == -1          # INPUT_ROTATED is quantize-only
    assert "TQ_INPUT_ROTATED" in tq.last_error()
    assert _decode(_params(flags=1 | 4), _cache()) == -1           # paper form needs ebar
    assert "ebar" in tq.last_error()
    assert _decode(_params(), _cache(), layer0=2) == -2
    assert _decode(_params(), _cache(), max_len=-1) == -1
    assert _decode(_params(), _cache(), max_len=129) == -5          # beyond the cache slots
    assert _decode(_params(), _cache(), out=FAKE + 4) == -3
    assert _decode(_params(), _cache(), ptrs=0) == -1
    assert _decode(_params(), _cache(), B=0) == 0


def test_decode_workspace_size_is_checked():
    p = _params(num_layers=1, num_heads=1)
    # one unit over 4096 tokens is split across blocks, which needs partials
    need = tq._load().tq_decode_workspace_bytes(ctypes.byref(p), 1, 1, 4096)
    assert need > 0
    c = _cache(slots=4096)
    assert _decode(p, c, max_len=4096) == -5 and "workspace" in tq.last_error()
    assert _decode(p, c, max_len=4096, ws=FAKE, ws_bytes=need - 1) == -5
    assert _decode(p, c, max_len=4096, ws=FAKE + 4, ws_bytes=need) == -3


def test_workspace_bytes_of_degenerate_shapes_is_zero():
    p = _params()
    L = tq._load()
    assert L.tq_decode_workspace_bytes(None, 1, 1, 64) == 0
    assert L.tq_decode_workspace_bytes(ctypes.byref(p), 0, 1, 64) == 0
    assert L.tq_decode_workspace_bytes(ctypes.byref(p), 1, 1, -1) == 0


def test_rope_table_and_calibration_argument_checks():
    L = tq._load()
    P = ctypes.c_void_p
    assert L.tq_rope_table(None, 10, 1e4, None) == -1
    assert L.tq_rope_table(P(FAKE + 4), 10, 1e4, None) == -3
    assert L.tq_rope_table(P(FAKE), 0, 1e4, None) == -1
    assert L.tq_rope_table(P(FAKE), 10, -1.0, None) == -1
    assert L.tq_rope_table(P(FAKE), 10, float("inf"), None) == -1
    assert L.tq_calibrate_rotation(None, 0, 10, None, None, None) == 0
    assert L.tq_calibrate_rotation(None, 2, 10, None, None, None) == -1
    assert L.tq_calibrate_rotation(P(FAKE), 2, 0, P(FAKE), None, None) == -1
    assert L.tq_calibrate_rotation(P(FAKE), -1, 10, P(FAKE), None, None) == -1


def _step(p, c, B=1, max_len=64, kv=FAKE, ws=None, ws_bytes=0, ptrs=FAKE, out=FAKE):
    L = tq._load()
    P = ctypes.c_void_p
    return L.tq_decode_step(ctypes.byref(p), ctypes.byref(c), P(ptrs), P(kv), P(kv), B, 0, 1, P(ptrs),
                            P(ptrs), P(ptrs), max_len, P(ptrs), P(ptrs), P(ptrs), P(ptrs), None, P(out),
                            P(ws) if ws else None, ws_bytes, None)


def test_decode_step_argument_checks():
    assert _step(_params(flags=1 | 16), _cache()) == -1
    assert "TQ_INPUT_ROTATED" in tq.last_error()
    assert _step(_params(), _cache(), max_len=0) == -1 and "max_len" in tq.last_error()
    assert _step(_params(), _cache(), kv=0) == -1 and "k and v" in tq.last_error()
    assert _step(_params(), _cache(), kv=FAKE + 4) == -3
    assert _step(_params(), _cache(), max_len=129) == -5
    assert _step(_params(), _cache(), B=0) == 0


def test_calibrate_lut_argument_checks():
    L = tq._load()
    P = ctypes.c_void_p
    good = (ctypes.c_float * 8)(-2.0, -1.3, -0.75, -0.25, 0.25, 0.75, 1.3, 2.0)
    flat = (ctypes.c_float * 8)(0.0, 0.0, -0.75, -0.25, 0.25, 0.75, 1.3, 2.0)
    nan = (ctypes.c_float * 8)(float("nan"), -1.3, -0.75, -0.25, 0.25, 0.75, 1.3, 2.0)
    c = lambda init, nh=2, ncal=10, it=100, tol=1e-7, x=FAKE, out=FAKE: L.tq_calibrate_lut(
        P(x) if x else None, nh, ncal, None, ctypes.cast(init, P) if init is not None else None, it, tol,
        P(out) if out else None, None)
    assert c(None) == -1 and "init" in tq.last_error()
    assert c(flat) == -4 and "ascending" in tq.last_error()
    assert c(nan) == -1 and "finite" in tq.last_error()
    assert c(good, it=0) == -1
    assert c(good, tol=-1.0) == -1
    assert c(good, tol=float("inf")) == -1
    assert c(good, nh=-1) == -1
    assert c(good, ncal=0) == -1
    assert c(good, x=0) == -1
    assert c(good, nh=0) == 0 and tq.last_error() == ""


def _dequant(p, c, B=1, max_len=64, ptrs=FAKE, out=FAKE, S=FAKE, ebar=None, layer0=0, nlayers=1):
    L = tq._load()
    P = ctypes.c_void_p
    return L.tq_dequantize(ctypes.byref(p) if p is not None else None, ctypes.byref(c) if c is not None else None,
                           B, layer0, nlayers, P(ptrs), P(ptrs), max_len, P(ptrs), P(ptrs),
                           P(S) if S else None, P(ebar) if ebar else None, P(out), P(out), None)


def test_dequantize_argument_checks():
    assert _dequant(None, _cache()) == -1 and "params" in tq.last_error()
    assert _dequant(_params(flags=1 | 16), _cache()) == -1 and "TQ_INPUT_ROTATED" in tq.last_error()
    assert _dequant(_params(flags=1 | 4), _cache()) == -1 and "ebar" in tq.last_error()
    assert _dequant(_params(), _cache(), S=0) == -1                     # the projected form needs S
    assert _dequant(_params(), _cache(), layer0=2) == -2
    assert _dequant(_params(), _cache(), max_len=129) == -5
    assert _dequant(_params(), _cache(), out=FAKE + 2) == -3
    assert _dequant(_params(), _cache(), ptrs=0) == -1
    # nothing to do is success, with nothing launched
    assert _dequant(_params(), _cache(), B=0) == 0
    assert _dequant(_params(), _cache(), max_len=0) == 0
    assert tq.last_error() == ""
