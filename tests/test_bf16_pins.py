"""Pins of the oracle's bf16 storage rounding (round to nearest, ties to even)."""
import numpy as np

import oracle


def _bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def test_hand_values():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -9, 1 + 2 ** -7 + 2 ** -8, -(1 + 2 ** -8 + 2 ** -20),
                  3.3895314e38, 3.39e38, 3.3961776e38, -np.inf, -0.0, 0.0], np.float32)
    want = [1.0, 1.0, 1 + 2 ** -7, 1 + 2 ** -6, -(1 + 2 ** -7),
            3.3895314e38, 3.3895314e38, np.inf, -np.inf, -0.0, 0.0]
    got = oracle.round_bf16(x)
    assert np.array_equal(_bits(got), _bits(np.array(want, np.float32)))
    assert np.isnan(oracle.round_bf16(np.array([np.nan], np.float32))).all()


def test_nearest_neighbour_property():
    """For random fp32 values the result is a bf16 value (low 16 bits zero), one of the
    two neighbours, and no farther than the other neighbour (exact fp64 distances)."""
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(4000) * np.exp(rng.uniform(-80, 80, 4000))).astype(np.float32)
    r = oracle.round_bf16(x)
    assert np.all((_bits(r) & 0xFFFF) == 0)
    lo = (_bits(x) & np.uint32(0xFFFF0000)).view(np.float32)
    hi = (_bits(lo) + np.uint32(0x10000)).view(np.float32)
    d = np.abs(r.astype(np.float64) - x.astype(np.float64))
    assert np.all((r == lo) | (r == hi))
    assert np.all(d <= np.minimum(np.abs(x.astype(np.float64) - lo), np.abs(hi.astype(np.float64) - x)))
    assert np.all(d <= np.abs(x.astype(np.float64)) * 2.0 ** -8)


def test_denormals_and_ties_to_even():
    tiny = np.array([2 ** -133, 3 * 2 ** -134, 2 ** -149], np.float32)   # bf16 subnormals / ties
    got = oracle.round_bf16(tiny)
    # 2^-133 is a bf16 subnormal (exact); 3*2^-134 lies halfway between 2^-133 and
    # 2^-132 and goes to the even one, 2^-132; 2^-149 ties between 0 and 2^-133: 0
    assert got.tolist() == [2 ** -133, 2 ** -132, 0.0]


def test_planted_mistake_is_caught():
    """Rounding half away from zero instead of to even differs on ties."""
    x = np.array([1 + 2 ** -8], np.float32)
    away = (_bits(x) + np.uint32(0x8000)) & np.uint32(0xFFFF0000)
    assert not np.array_equal(_bits(oracle.round_bf16(x)), away)
