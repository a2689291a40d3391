"""Seeded synthetic inputs shaped like the ESM-2 workloads of TurboESM.

This module only draws random inputs; it holds none of the method's arithmetic
(no RoPE, rotation, quantization or attention). The GPU path and the CPU
oracle both take their inputs from here.

Distributions (ESM-2 activations are not available, so these stand in for
them; Sec. 2.2 describes channel-wise outliers 10-100x the median):
  keys      N(0, 1) per channel, 4 outlier channels per (layer, head) scaled x20
            (the first 4 entries of a seeded permutation of 0..63)
  values    Student-t with 4 degrees of freedom (heavy tailed, variance 2)
  queries   N(0, 1)
  QJL S     N(0, 1), 64 x 64, shared by all heads
  Pi        QR of a seeded Gaussian 64 x 64 with diag(R) > 0 (a random rotation)
  lengths   ragged batches: integers uniform in [lo, hi]
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

HEAD_DIM = 64
OUTLIER_CHANNELS = 4
OUTLIER_SCALE = 20.0
STUDENT_T_DOF = 4.0

# 8-level minimum-MSE quantizer of N(0, 1), as tabulated by J. Max,
# "Quantizing for minimum distortion", IRE Trans. Inf. Theory IT-6 (1960),
# Table I, N = 8 (four significant digits). A default table for callers that
# have no calibrated one.
GAUSS_LEVELS_MAX1960 = np.array(
    [-2.152, -1.344, -0.7560, -0.2451, 0.2451, 0.7560, 1.344, 2.152], dtype=np.float32)


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    heads: int
    batch: int
    seq: int                 # cached tokens per sequence before decode (max for ragged)
    io_dtype: str            # "f32" or "f16"
    decode_steps: int = 1
    ragged: tuple | None = None   # (lo, hi) of uniform sequence lengths
    rotation: str = "qr"     # "qr" random rotation, "svd" head-wise calibration
    calib_vectors: int = 0   # calibration keys per head for "svd"
    seed: int = 20260
    notes: str = field(default="")


WORKLOADS = {
    "tiny-1x1-seq256-fp32": Workload(
        "tiny-1x1-seq256-fp32", 1, 1, 1, 256, "f32", 1, seed=20260,
        notes="1 layer, 1 head, seq 256, fp32 I/O, one decode query"),
    "esm2-650m-1layer-seq1024": Workload(
        "esm2-650m-1layer-seq1024", 1, 20, 1, 1024, "f16", 64, rotation="svd",
        calib_vectors=4096, seed=20261,
        notes="one ESM-2 650M layer (20 heads), prefill 1024 then 64 decode steps"),
    "esm2-650m-33layer-seq1024": Workload(
        "esm2-650m-33layer-seq1024", 33, 20, 1, 1024, "f16", 1, seed=20262,
        notes="full ESM-2 650M cache, batch 1, decode across all 33 layers per step"),
    "esm2-650m-ragged-b64": Workload(
        "esm2-650m-ragged-b64", 33, 20, 64, 1024, "f16", 1, ragged=(50, 1024), seed=20263,
        notes="64 sequences, lengths uniform in [50, 1024], ESM-2 650M shape"),
    "esm2-3b-36layer-b16-seq8192": Workload(
        "esm2-3b-36layer-b16-seq8192", 36, 40, 16, 8192, "f16", 32, rotation="svd",
        calib_vectors=4096, seed=20264,
        notes="ESM-2 3B shape, batch 16, seq 8192, prefill then 32 decode steps"),
}


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def outlier_channels(g: np.random.Generator, layers: int, heads: int) -> np.ndarray:
    """[layers][heads][4] channel indices of the outlier channels."""
    out = np.empty((layers, heads, OUTLIER_CHANNELS), dtype=np.int64)
    for l in range(layers):
        for h in range(heads):
            out[l, h] = g.permutation(HEAD_DIM)[:OUTLIER_CHANNELS]
    return out


def keys(g: np.random.Generator, layers: int, batch: int, tokens: int, heads: int,
         channels: np.ndarray) -> np.ndarray:
    """[layers][batch][tokens][heads][64] float32 keys with outlier channels."""
    k = g.standard_normal((layers, batch, tokens, heads, HEAD_DIM), dtype=np.float32)
    for l in range(layers):
        for h in range(heads):
            k[l, :, :, h, channels[l, h]] *= OUTLIER_SCALE
    return k


def values(g: np.random.Generator, layers: int, batch: int, tokens: int, heads: int) -> np.ndarray:
    """[layers][batch][tokens][heads][64] float32 Student-t values."""
    return g.standard_t(STUDENT_T_DOF, (layers, batch, tokens, heads, HEAD_DIM)).astype(np.float32)


def queries(g: np.random.Generator, layers: int, batch: int, heads: int) -> np.ndarray:
    """[layers][batch][heads][64] float32 N(0, 1) queries."""
    return g.standard_normal((layers, batch, heads, HEAD_DIM), dtype=np.float32)


def qjl_matrix(g: np.random.Generator) -> np.ndarray:
    """64 x 64 float32 N(0, 1) projection."""
    return g.standard_normal((HEAD_DIM, HEAD_DIM), dtype=np.float32)


def random_rotation(g: np.random.Generator) -> np.ndarray:
    """64 x 64 orthogonal matrix: Q of a Gaussian matrix, columns signed so diag(R) > 0."""
    a = g.standard_normal((HEAD_DIM, HEAD_DIM))
    q, r = np.linalg.qr(a)
    q = q * np.where(np.diag(r) < 0, -1.0, 1.0)[None, :]
    return q.astype(np.float32)


def rotations(g: np.random.Generator, layers: int, heads: int) -> np.ndarray:
    """[layers][heads][64][64] float32 random rotations."""
    out = np.empty((layers, heads, HEAD_DIM, HEAD_DIM), dtype=np.float32)
    for l in range(layers):
        for h in range(heads):
            out[l, h] = random_rotation(g)
    return out


def ragged_lengths(g: np.random.Generator, batch: int, lo: int, hi: int) -> np.ndarray:
    return g.integers(lo, hi + 1, size=batch, dtype=np.int64).astype(np.int32)


def calibration_positions(g: np.random.Generator, n: int, seq: int) -> np.ndarray:
    """Positions in [0, seq) at which the calibration keys sit."""
    return g.integers(0, seq, size=n, dtype=np.int64).astype(np.int32)


def tile_aligned_offsets(lengths, extra: int = 0) -> tuple[np.ndarray, int]:
    """First slot of each sequence when capacities len+extra are rounded up to
    multiples of 64 and laid end to end; returns (offsets, total slots)."""
    caps = [((int(n) + extra + 63) // 64) * 64 for n in lengths]
    offs = np.zeros(len(caps), dtype=np.int64)
    acc = 0
    for i, c in enumerate(caps):
        offs[i] = acc
        acc += c
    return offs, max(acc, 64)


def as_io(x: np.ndarray, io_dtype: str) -> np.ndarray:
    """Round to the I/O type (fp16 for the ESM-2 workloads) and back to float32 values."""
    if io_dtype == "f16":
        return x.astype(np.float16)
    return x.astype(np.float32)


# ---------------------------------------------------------------------------
# The same distributions drawn on a torch device, for workloads too large to
# draw on the host (the ESM-2 3B shape has 2.7e9 key and value elements).
# Seeded by (seed, layer) so that one layer can be drawn at a time; the
# streams differ from the NumPy ones above, the distributions do not.
# ---------------------------------------------------------------------------
def device_generator(seed: int, layer: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + int(layer))
    return g


def keys_on(gen, batch: int, tokens: int, heads: int, channels_lh: np.ndarray, dtype, device):
    """[batch][tokens][heads][64] keys of one layer: N(0, 1), the 4 outlier
    channels of each head (channels_lh [heads][4]) scaled x20."""
    import torch
    k = torch.randn((batch, tokens, heads, HEAD_DIM), generator=gen, device=device, dtype=torch.float32)
    scale = torch.ones((heads, HEAD_DIM), dtype=torch.float32)
    for h in range(heads):
        scale[h, torch.as_tensor(channels_lh[h])] = OUTLIER_SCALE
    k *= scale.to(device)
    return k.to(dtype)


def values_on(gen, batch: int, tokens: int, heads: int, dtype, device):
    """[batch][tokens][heads][64] Student-t (4 degrees of freedom) values of
    one layer: z0 / sqrt((z1^2 + z2^2 + z3^2 + z4^2) / 4) with z ~ N(0, 1)."""
    import torch
    shape = (batch, tokens, heads, HEAD_DIM)
    chi = torch.zeros(shape, device=device, dtype=torch.float32)
    for _ in range(int(STUDENT_T_DOF)):
        z = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        chi.addcmul_(z, z)
    z0 = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    return (z0 / torch.sqrt(chi / STUDENT_T_DOF)).to(dtype)


def queries_on(gen, batch: int, heads: int, dtype, device):
    """[batch][heads][64] N(0, 1) queries of one layer."""
    import torch
    return torch.randn((batch, heads, HEAD_DIM), generator=gen, device=device,
                       dtype=torch.float32).to(dtype)
