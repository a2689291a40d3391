"""The GPU tests decode the bytes the library wrote with their own unpacker
(tests/gpu_cases.py), never with the oracle; this checks that unpacker
against the oracle's packer on the CPU."""
import numpy as np
import pytest

from gpu_cases import DeviceBytes, unpack_slot
from oracle import oracle
from paper_2603_26110_amd import synth


@pytest.mark.parametrize("plane", ["k", "v"])
def test_unpacker_reads_what_the_oracle_packs(plane):
    g = synth.rng(51)
    slots = 192
    region = np.zeros(slots * 32, np.uint8)
    nibs = g.integers(0, 16, (slots, 64)).astype(np.uint8)
    for s in range(slots):
        oracle.pack_slot(region, s, nibs[s], plane)
    for s in range(slots):
        np.testing.assert_array_equal(unpack_slot(region, s, plane), nibs[s])


def test_device_bytes_regions():
    L, H, slots = 2, 3, 64
    k = np.arange(L * H * slots * 32, dtype=np.int64).astype(np.uint8)
    v = k[::-1].copy()
    s = np.arange(L * H * slots * 4, dtype=np.uint16)
    db = DeviceBytes(L, H, slots, k, v, s)
    oc = oracle.Cache(L, H, slots)
    oc.k[:], oc.v[:], oc.s[:] = k, v, s
    for l in range(L):
        for h in range(H):
            np.testing.assert_array_equal(db.region("k", l, h), oc.region("k", l, h))
            np.testing.assert_array_equal(db.region("v", l, h), oc.region("v", l, h))
            np.testing.assert_array_equal(db.scalars(l, h), oc.scalars(l, h))


def test_unpack_planes_matches_the_per_slot_unpackers():
    # the vectorized reader of whole regions against the per-slot reader of
    # the tests and the oracle's own unpacker, on random bytes
    from gpu_cases import unpack_planes, unpack_slot
    g = np.random.default_rng(3)
    reg_k = g.integers(0, 256, 3 * 2048, dtype=np.uint8)
    reg_v = g.integers(0, 256, 3 * 2048, dtype=np.uint8)
    kn, vn = unpack_planes(reg_k, reg_v)
    assert kn.shape == (192, 64) and vn.shape == (192, 64)
    for s in range(0, 192, 7):
        assert np.array_equal(kn[s], unpack_slot(reg_k, s, "k"))
        assert np.array_equal(vn[s], unpack_slot(reg_v, s, "v"))
        assert np.array_equal(kn[s], oracle.unpack_slot(reg_k, s, "k"))
        assert np.array_equal(vn[s], oracle.unpack_slot(reg_v, s, "v"))
