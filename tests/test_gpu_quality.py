"""The quality ablation on a small shape (4 heads, 256 tokens): outputs are
finite, the random rotation beats no rotation on keys with outlier channels
(Sec. 2.2, Sec. 3.2), and the per-element sign correction beats leaving the
residual out (Sec. 3.3)."""
import pytest

pytestmark = pytest.mark.gpu


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
