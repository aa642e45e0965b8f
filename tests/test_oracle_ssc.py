"""Pins for the oracle's Spatiotemporal Stability Criterion (Eqs. 2, 6, 7) and selection.

Each check compares against something other than the oracle's own formula:
closed-form norms, exactly-representable sums, the correctly-rounded float64
route, brute-force ranking, and the omega in {0, 1} special cases that reduce
the criterion to the single-component rows of the SSC ablation table.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import ssc

F32 = np.float32


def test_magnitude_closed_forms():
    v = np.zeros((4, 8), F32)
    v[0, :2] = [3, 4]                      # 3-4-5 triangle
    v[1, :] = 1                            # sqrt(8)
    v[2, 7] = -2.5                         # single component, sign ignored
    mag = ssc.velocity_magnitude(v)
    assert mag[0] == F32(5.0)
    assert mag[1] == F32(math.sqrt(8.0))
    assert mag[2] == F32(2.5)
    assert mag[3] == F32(0.0)


def test_magnitude_is_correctly_rounded():
    # small integers: every partial sum of squares is exact in float32, so the
    # only rounding is the final sqrt, which must equal the float64 sqrt
    # rounded once to float32 (correct for sqrt since 53 >= 2*24 + 2).
    rng = np.random.default_rng(5)
    v = rng.integers(-300, 300, size=(5000, 8)).astype(F32)
    exact = np.array([math.fsum(float(x) ** 2 for x in row) for row in v])
    want = np.sqrt(exact).astype(F32)
    got = ssc.velocity_magnitude(v)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_magnitude_channel_order():
    # 1 + 2^-24 + 2^-24 ... : in channel order the tiny terms are absorbed one
    # at a time (each partial sum rounds back to 1); summed in another order they
    # would survive. Pins the sequential accumulation from 0 in channel order.
    tiny = F32(2.0 ** -12)                 # square is 2^-24 = half an ulp of 1
    v = np.array([[1.0] + [tiny] * 7], F32)
    s = ssc.velocity_magnitude(v)[0] ** 2
    assert ssc.velocity_magnitude(v)[0] == F32(1.0)
    assert s == F32(1.0)


def test_acceleration_zero_and_reduction():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((300, 8)).astype(F32)
    assert np.all(ssc.acceleration(v, v) == 0)
    assert np.array_equal(ssc.acceleration(v, np.zeros_like(v)), ssc.velocity_magnitude(v))
    assert np.array_equal(ssc.acceleration(v, -v), ssc.velocity_magnitude(v + v))


def test_normalise_range_and_extremes():
    rng = np.random.default_rng(2)
    a = rng.exponential(size=1000).astype(F32)
    n = ssc.minmax_normalise(a)
    assert n.dtype == F32
    assert n.min() == 0 and n.max() == 1
    assert n[np.argmin(a)] == 0 and n[np.argmax(a)] == 1
    assert np.all((n >= 0) & (n <= 1))
    # order preserving (monotone map)
    o = np.argsort(a, kind="stable")
    assert np.all(np.diff(n[o]) >= 0)


def test_normalise_degenerate_is_zero():
    assert np.all(ssc.minmax_normalise(np.full(17, 3.5, F32)) == 0)
    a = np.array([np.nan, 1.0, 1.0], F32)
    assert np.all(ssc.minmax_normalise(a) == 0)


def test_normalise_ignores_nan_in_extremes():
    a = np.array([np.nan, 1.0, 3.0, 2.0], F32)
    n = ssc.minmax_normalise(a)
    assert np.isnan(n[0]) and n[1] == 0 and n[2] == 1 and n[3] == F32(0.5)


def _brute_rank_select(score, c):
    n = len(score)
    def key(i):
        s = float(score[i])
        return (math.isnan(s), 0.0 if math.isnan(s) else s, i)
    order = sorted(range(n), key=key)
    cached = sorted(order[:c])
    active = [i for i in range(n) if i not in set(cached)]
    return cached, active


def test_select_matches_bruteforce_exhaustive_with_ties():
    values = [F32(0.0), F32(0.25), F32(0.5), F32(np.nan)]
    for n in (1, 2, 3, 5):
        for combo in itertools.product(range(len(values)), repeat=n):
            score = np.array([values[j] for j in combo], F32)
            for c in range(n + 1):
                cached, active = ssc.select(score, c)
                bc, ba = _brute_rank_select(score, c)
                assert cached.tolist() == bc and active.tolist() == ba


def test_select_lexsort_equivalence_large():
    rng = np.random.default_rng(3)
    score = rng.integers(0, 50, size=4096).astype(F32) / F32(49)   # many ties
    for c in (0, 1, 2047, 4095, 4096):
        cached, active = ssc.select(score, c)
        ref = np.sort(np.lexsort((np.arange(4096), score))[:c])
        assert np.array_equal(cached, ref)
        assert np.array_equal(np.sort(np.concatenate([cached, active])), np.arange(4096))
        assert np.all(np.diff(active) > 0)


def test_select_rejects_bad_quota():
    with pytest.raises(ValueError):
        ssc.select(np.zeros(4, F32), 5)
    with pytest.raises(ValueError):
        ssc.select(np.zeros(4, F32), -1)


def _rank_by(values, c):
    order = sorted(range(len(values)), key=lambda i: (float(values[i]), i))
    return sorted(order[:c])


def test_omega_one_is_acceleration_only_and_zero_is_velocity_only():
    rng = np.random.default_rng(4)
    vc = rng.standard_normal((512, 8)).astype(F32)
    vp = rng.standard_normal((512, 8)).astype(F32)
    acc = ssc.acceleration(vc, vp)
    mag = ssc.velocity_magnitude(vc)
    for c in (1, 100, 256, 511):
        cached_a, _ = ssc.select(ssc.cache_score(vc, vp, 1.0), c)
        assert cached_a.tolist() == _rank_by(acc, c)
        cached_v, _ = ssc.select(ssc.cache_score(vc, vp, 0.0), c)
        assert cached_v.tolist() == _rank_by(mag, c)


def test_score_weights_and_range():
    rng = np.random.default_rng(6)
    vc = rng.standard_normal((256, 8)).astype(F32)
    vp = rng.standard_normal((256, 8)).astype(F32)
    c = ssc.cache_score(vc, vp, 0.7)
    assert c.dtype == F32
    assert np.all((c >= 0) & (c <= F32(1.0000001)))
    # the token that is extreme in both components reaches the weight sum
    vc2 = vc.copy()
    vc2[7] = 100.0
    vp2 = vp.copy()
    vp2[7] = -100.0
    c2 = ssc.cache_score(vc2, vp2, 0.7)
    assert c2[7] == F32(0.7) + (F32(1.0) - F32(0.7))
