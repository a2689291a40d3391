"""Attention-output quality of the quantized cache against exact attention, on
the seeded synthetic stand-ins for ESM-2 activations (ESM-2 weights and
protein data are not available): the ablations of TurboESM Table 7 (rotation,
tables, QJL correction), measured on one ESM-2 650M layer shape.

Each variant quantizes the same keys and values with tq_quantize_pack and
decodes one query per head with tq_decode_attend (fp32 output). The reference
is exact attention in fp64 over the RoPE'd keys (positions 0 .. T-1, query at
T-1, softmax scale 1/8) and the raw values. Reported per variant: the mean and
the minimum over heads of the cosine similarity of the two outputs, and the
mean relative L2 error.

Calibration follows the paper's recipe (Sec. 3.2, Sec. 3.3): the head-wise
rotation is the SVD basis of calibration keys (tq_calibrate_rotation), the
tables are the 1-D Lloyd iteration on the normalized rotated coordinates of
calibration keys and values (tq_calibrate_lut), and the per-head mean
residual magnitudes of the per-element sign correction come from
tq_calibrate_ebar on the same calibration vectors. Calibration vectors are drawn from the same
distributions at seeded positions.

    python -m paper_2603_26110_amd.quality [--heads 20] [--tokens 1024] [--calib 4096]
"""
from __future__ import annotations

import argparse

import numpy as np
import torch

from . import synth


def _rope(x: np.ndarray, pos: np.ndarray, base: float = 10000.0) -> np.ndarray:
    """RoPE in fp64 on pairs (2m, 2m+1), theta_m = base^(-2m/64). x: [..., n, 64],
    pos: [n]."""
    m = np.arange(32, dtype=np.float64)
    ang = pos.astype(np.float64)[:, None] * base ** (-2.0 * m / 64.0)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., 0::2].astype(np.float64), x[..., 1::2].astype(np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def exact_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, qpos: int) -> np.ndarray:
    """q [H][64], k, v [T][H][64] (positions 0 .. T-1). Returns [H][64] fp64."""
    T = k.shape[0]
    kr = _rope(np.transpose(k, (1, 0, 2)), np.arange(T))          # [H][T][64]
    qr = _rope(q[:, None, :], np.array([qpos]))[:, 0, :]           # [H][64]
    logits = np.einsum("hd,htd->ht", qr, kr) * 0.125
    logits -= logits.max(axis=1, keepdims=True)
    w = np.exp(logits)
    w /= w.sum(axis=1, keepdims=True)
    return np.einsum("ht,htd->hd", w, np.transpose(v, (1, 0, 2)).astype(np.float64))


def inputs(heads: int = 20, tokens: int = 1024, calib: int = 4096, seed: int = 20261) -> dict:
    """The seeded raw inputs of the ablation (numpy): keys and values
    [1][1][T][H][64] and the query [1][1][H][64] (fp16 values), S, a random
    rotation per head, and the calibration sets: post-RoPE keys and values
    [H][calib][64] (fp32). Also the fp64 exact-attention reference [H][64]."""
    g = synth.rng(seed)
    H, T = heads, tokens
    ch = synth.outlier_channels(g, 1, H)
    k = synth.as_io(synth.keys(g, 1, 1, T, H, ch), "f16")             # [1][1][T][H][64]
    v = synth.as_io(synth.values(g, 1, 1, T, H), "f16")
    q = synth.as_io(synth.queries(g, 1, 1, H), "f16")                 # [1][1][H][64]
    S = synth.qjl_matrix(g)
    pi_qr = synth.rotations(g, 1, H)[0]                                # [H][64][64]
    kc = synth.keys(g, 1, 1, calib, H, ch)[0, 0].astype(np.float32)   # [n][H][64]
    vc = synth.values(g, 1, 1, calib, H)[0, 0].astype(np.float32)
    pc = synth.calibration_positions(g, calib, T)
    kc_r = _rope(np.transpose(kc, (1, 0, 2)), pc).astype(np.float32)  # [H][n][64]
    vc_h = np.ascontiguousarray(np.transpose(vc, (1, 0, 2)))
    ref = exact_attention(q[0, 0].astype(np.float64), k[0, 0], v[0, 0], T - 1)
    return {"H": H, "T": T, "k": k, "v": v, "q": q, "S": S, "pi_qr": pi_qr, "kc": kc_r, "vc": vc_h, "ref": ref}


# Variant names, in the order of the table (the Table 7 ablations).
VARIANTS = [
    "no rotation (Pi = I), Gaussian tables, QJL",
    "random-QR Pi, Gaussian tables, QJL",
    "random-QR Pi, Gaussian tables, no QJL (S = 0)",
    "random-QR Pi, Gaussian tables, per-element signs + ebar (paper QJL)",
    "random-QR Pi, one calibrated table for K and V, QJL",
    "random-QR Pi, calibrated K and V tables, QJL",
    "SVD Pi, Gaussian tables, QJL",
    "SVD Pi, calibrated K and V tables, QJL",
    "SVD Pi, calibrated K and V tables, no QJL (S = 0)",
]


def variant_parameters(inp: dict, rotation, table, ebar) -> list[dict]:
    """Pi, tables, S, flags and ebar of every variant (numpy, fp32), from the
    calibration callables rotation(x [H][n][64]) -> Pi [H][64][64],
    table(x, pi) -> [H][8] and ebar(x, pi, lut) -> [H] (the library's, or
    any other implementation of Sec. 3.2-3.4)."""
    H = inp["H"]
    eye = np.broadcast_to(np.eye(64, dtype=np.float32), (H, 64, 64)).copy()
    gauss = np.broadcast_to(synth.GAUSS_LEVELS_MAX1960, (H, 8)).copy()
    S, S0 = inp["S"], np.zeros((64, 64), np.float32)
    pi_qr = inp["pi_qr"]
    pi_svd = rotation(inp["kc"])
    lk_qr, lv_qr = table(inp["kc"], pi_qr), table(inp["vc"], pi_qr)
    lk_svd, lv_svd = table(inp["kc"], pi_svd), table(inp["vc"], pi_svd)
    shared_qr = table(np.concatenate([inp["kc"], inp["vc"]], 1), pi_qr)
    eb = np.stack([ebar(inp["kc"], pi_qr, gauss), ebar(inp["vc"], pi_qr, gauss)], 1).astype(np.float32)
    R = 1   # V_ROTATE
    rows = [
        (eye, gauss, gauss, S, R, None), (pi_qr, gauss, gauss, S, R, None), (pi_qr, gauss, gauss, S0, R, None),
        (pi_qr, gauss, gauss, S, R | 4, eb), (pi_qr, shared_qr, shared_qr, S, R, None),
        (pi_qr, lk_qr, lv_qr, S, R, None), (pi_svd, gauss, gauss, S, R, None),
        (pi_svd, lk_svd, lv_svd, S, R, None), (pi_svd, lk_svd, lv_svd, S0, R, None),
    ]
    return [{"variant": name, "pi": np.ascontiguousarray(p, np.float32), "lut_k": np.ascontiguousarray(a, np.float32),
             "lut_v": np.ascontiguousarray(b, np.float32), "S": np.ascontiguousarray(sm, np.float32), "flags": f,
             "ebar": e} for name, (p, a, b, sm, f, e) in zip(VARIANTS, rows)]


def decode_variant(inp: dict, var: dict) -> np.ndarray:
    """tq_quantize_pack of the T tokens, then tq_decode_attend of the query at
    position T - 1 (fp32 output): [H][64]."""
    import paper_2603_26110_amd as tq
    dev = torch.device("cuda")
    H, T = inp["H"], inp["T"]
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    cs = tq.rope_table(T + 64)
    params = tq.Params(1, H, cs, io_dtype=torch.float16, flags=var["flags"] | tq.OUT_FP32)
    cache = tq.Cache(1, H, (T + 63) // 64 * 64)
    i32 = lambda x: torch.tensor([x], dtype=torch.int32, device=dev)
    i64 = lambda x: torch.tensor([x], dtype=torch.int64, device=dev)
    lk, lv = t_(var["lut_k"].reshape(1, H, 8)), t_(var["lut_v"].reshape(1, H, 8))
    pi1 = t_(var["pi"].reshape(1, H, 64, 64))
    s_mat = t_(var["S"])
    eb = None if var["ebar"] is None else t_(var["ebar"].reshape(1, H, 2))
    tq.quantize_pack(params, cache, t_(inp["k"]), t_(inp["v"]), i32(0), i64(0), pi1, lk, lv, s_mat, eb)
    out = tq.decode_attend(params, cache, t_(inp["q"]), i32(T - 1), i64(0), i32(T), T, pi1, lk, lv, s_mat, eb)
    return out.double().cpu().numpy()[0, 0]


def metrics(o: np.ndarray, ref: np.ndarray) -> dict:
    cos = (o * ref).sum(1) / (np.linalg.norm(o, axis=1) * np.linalg.norm(ref, axis=1))
    rel = np.linalg.norm(o - ref, axis=1) / np.linalg.norm(ref, axis=1)
    return {"cos_mean": float(cos.mean()), "cos_min": float(cos.min()), "rel_l2": float(rel.mean())}


def library_calibration():
    """The three calibration callables of variant_parameters, by the library
    (tq_calibrate_rotation, tq_calibrate_lut, tq_calibrate_ebar)."""
    import paper_2603_26110_amd as tq
    dev = torch.device("cuda")
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    rotation = lambda x: tq.calibrate_rotation(t_(x))[0].cpu().numpy()
    table = lambda x, pi: tq.calibrate_lut(t_(x), t_(pi)).cpu().numpy()
    ebar = lambda x, pi, lut: tq.calibrate_ebar(t_(x), t_(lut), t_(pi)).cpu().numpy()
    return rotation, table, ebar


def run(heads: int = 20, tokens: int = 1024, calib: int = 4096, seed: int = 20261) -> list[dict]:
    inp = inputs(heads, tokens, calib, seed)
    rows = []
    for var in variant_parameters(inp, *library_calibration()):
        r = metrics(decode_variant(inp, var), inp["ref"])
        r["variant"] = var["variant"]
        rows.append(r)
    return rows


def calibration_timing(layers: int = 33, heads: int = 20, ncal: int = 4096, seq: int = 1024,
                       seed: int = 20262) -> dict:
    """Wall time of the full calibration of one model on the GPU: the head-wise
    rotation (SVD basis of ncal post-RoPE keys per head) and the K and V tables
    for layers x heads heads. The calibration vectors are drawn on the GPU and
    RoPE'd there (torch elementwise ops on the library's cos/sin table)."""
    import time

    import paper_2603_26110_amd as tq
    dev = torch.device("cuda")
    g = synth.rng(seed)
    nh = layers * heads
    ch = synth.outlier_channels(g, layers, heads).reshape(nh, 1, -1)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    k = torch.randn((nh, ncal, 64), generator=gen, device=dev)
    idx = torch.from_numpy(ch).to(dev).expand(nh, ncal, ch.shape[-1])
    k.scatter_(2, idx, k.gather(2, idx) * synth.OUTLIER_SCALE)
    z = torch.randn((5, nh, ncal, 64), generator=gen, device=dev)
    v = z[0] / torch.sqrt((z[1:] ** 2).mean(0))          # Student-t, 4 degrees of freedom
    pos = torch.randint(0, seq, (ncal,), generator=gen, device=dev)
    cs = tq.rope_table(seq)[pos]                          # [ncal][32][2]
    c, s_ = cs[..., 0], cs[..., 1]
    a, b = k[..., 0::2], k[..., 1::2]
    kr = torch.empty_like(k)
    kr[..., 0::2] = a * c - b * s_
    kr[..., 1::2] = a * s_ + b * c
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pi, _ = tq.calibrate_rotation(kr)
    lk = tq.calibrate_lut(kr, pi)
    lv = tq.calibrate_lut(v, pi)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    assert torch.isfinite(lk).all() and torch.isfinite(lv).all()
    return {"heads": nh, "ncal": ncal, "seconds": dt}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--calib-timing", action="store_true",
                    help="time the full calibration of a 33 x 20 head model instead")
    ap.add_argument("--heads", type=int, default=20)
    ap.add_argument("--tokens", type=int, default=1024)
    ap.add_argument("--calib", type=int, default=4096)
    ap.add_argument("--seed", type=int, default=20261)
    a = ap.parse_args()
    if a.calib_timing:
        r = calibration_timing(ncal=a.calib)
        print(f"calibration of {r['heads']} heads ({r['ncal']} vectors each): rotation + K and V tables "
              f"{r['seconds']:.3f} s")
        return
    rows = run(a.heads, a.tokens, a.calib, a.seed)
    print(f"{a.heads} heads x 64, {a.tokens} cached tokens (fp16), {a.calib} calibration vectors per head, "
          f"seed {a.seed}")
    print("| variant | cosine (mean over heads) | cosine (min) | relative L2 error |")
    print("|---|---|---|---|")
    for r in rows:
        print(f"| {r['variant']} | {r['cos_mean']:.5f} | {r['cos_min']:.5f} | {r['rel_l2']:.4f} |")


if __name__ == "__main__":
    main()
