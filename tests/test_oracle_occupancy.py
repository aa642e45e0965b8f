"""Pins of the dynamic-voxel oracle (Eq. 1) by closed forms, brute force and
invariants of the Hamming distance."""
import itertools

import numpy as np

from oracle import occupancy as occ


def test_closed_forms():
    g = np.random.default_rng(0).random((8, 8, 8)) > 0.5
    assert occ.dynamic_voxels(g, g) == 0                    # no change
    assert occ.dynamic_voxels(g, ~g) == g.size              # every voxel flips
    h = g.copy()
    h[3, 4, 5] = ~h[3, 4, 5]
    assert occ.dynamic_voxels(h, g) == 1                    # one flip


def test_brute_force_triple_loop():
    rng = np.random.default_rng(1)
    for n in (1, 2, 3, 5):
        a = rng.random((n, n, n)) > 0.3
        b = rng.random((n, n, n)) > 0.6
        want = 0
        for i, j, k in itertools.product(range(n), repeat=3):
            want += int(bool(a[i, j, k]) != bool(b[i, j, k]))
        assert occ.dynamic_voxels(a, b) == want


def test_metric_properties():
    rng = np.random.default_rng(2)
    a, b, c = (rng.random((16, 16, 16)) > p for p in (0.2, 0.5, 0.7))
    dab, dbc, dac = occ.dynamic_voxels(a, b), occ.dynamic_voxels(b, c), occ.dynamic_voxels(a, c)
    assert dab == occ.dynamic_voxels(b, a)
    assert dac <= dab + dbc
    # counts of occupied voxels bound the distance from below
    assert dab >= abs(int(a.sum()) - int(b.sum()))


def test_occupancy_threshold_and_nan():
    x = np.array([-1.0, -0.0, 0.0, 1e-30, 2.0, np.nan, np.inf, -np.inf])
    assert occ.occupancy(x).tolist() == [False, False, False, True, True, False, True, False]


def test_pack_layout():
    # voxel n in bit n % 32 of word n // 32, zero padding in the tail word
    flat = np.zeros(70, dtype=bool)
    flat[[0, 31, 32, 69]] = True
    words = occ.pack(flat)
    assert words.tolist() == [0x80000001, 0x00000001, 0x00000020]
    # popcount of the XOR of packed grids equals the count of the unpacked ones
    rng = np.random.default_rng(3)
    a = rng.random(1000) > 0.5
    b = rng.random(1000) > 0.5
    x = occ.pack(a) ^ occ.pack(b)
    assert sum(bin(int(v)).count("1") for v in x) == occ.dynamic_voxels(a, b)
