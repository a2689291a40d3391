"""The quality ablation (Table 7 analog) on a small shape (4 heads, 256
tokens).

Every variant's HIP output is compared with the oracle decoding the same
variant: each variant's Pi, tables and ebar are computed by the oracle's
calibration (SVD, 1-D Lloyd, mean residual) and given to both sides, each
side quantizes the same raw keys and values into a cache of its own, and the
outputs agree within 2e-3 (fp32 output). With the library's own calibration
the outputs are finite and two orderings of the paper hold: a rotation beats
none on keys with outlier channels (Sec. 2.2, Sec. 3.2), and the per-element
sign correction beats leaving the residual out (Sec. 3.4)."""
import numpy as np
import pytest

from oracle import oracle
from paper_2603_26110_amd import synth

pytestmark = pytest.mark.gpu
TOL = 2e-3


def test_every_variant_matches_the_oracle():
    from paper_2603_26110_amd import quality
    inp = quality.inputs(heads=4, tokens=256, calib=1024, seed=7)
    H, T = inp["H"], inp["T"]
    init = synth.GAUSS_LEVELS_MAX1960

    def rotation(x):
        return np.stack([oracle.calibrate_rotation(x[h])[0] for h in range(len(x))])

    def table(x, pi):
        return np.stack([oracle.calibrate_lut(x[h], pi[h], init) for h in range(len(x))]).astype(np.float32)

    def ebar(x, pi, lut):
        return np.array([oracle.calibrate_ebar(x[h], pi[h], lut[h]) for h in range(len(x))])

    cs = oracle.rope_table(T + 64)
    variants = quality.variant_parameters(inp, rotation, table, ebar)
    assert [v["variant"] for v in variants] == quality.VARIANTS
    for var in variants:
        got = quality.decode_variant(inp, var)
        oc = oracle.Cache(1, H, (T + 63) // 64 * 64)
        oracle.quantize_pack(oc, var["flags"], cs, inp["k"].astype(np.float32), inp["v"].astype(np.float32), [0],
                             [0], var["pi"][None], var["lut_k"][None], var["lut_v"][None], var["S"])
        ref = oracle.decode(oc, var["flags"], cs, inp["q"].astype(np.float32), [T - 1], [0], [T], var["pi"][None],
                            var["lut_k"][None], var["lut_v"][None], var["S"],
                            ebar=None if var["ebar"] is None else var["ebar"][None])[0, 0]
        err = np.max(np.abs(got - ref))
        assert np.all(np.isfinite(got)) and err <= TOL, (var["variant"], err)


def test_quality_ablation_small():
    from paper_2603_26110_amd import quality
    rows = {r["variant"]: r for r in quality.run(heads=4, tokens=256, calib=1024, seed=7)}
    assert len(rows) == 9
    for name, r in rows.items():
        assert -1.0 <= r["cos_min"] <= r["cos_mean"] <= 1.0 + 1e-9, name
    qr = rows["random-QR Pi, Gaussian tables, QJL"]
    none = rows["no rotation (Pi = I), Gaussian tables, QJL"]
    assert qr["rel_l2"] < none["rel_l2"]
    paper = rows["random-QR Pi, Gaussian tables, per-element signs + ebar (paper QJL)"]
    no_qjl = rows["random-QR Pi, Gaussian tables, no QJL (S = 0)"]
    assert paper["rel_l2"] < no_qjl["rel_l2"]
