"""Checks of the seeded workload generator (shapes, storage rounding, recipes)."""
import numpy as np

from paper_2608_11231_amd import inputs as I


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2.0**-8, 1.0 + 3 * 2.0**-9, -2.5, 1e-3], np.float64)
    r = I.round_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0          # tie -> even mantissa
    assert r[2] == 1.0 + 2.0**-7                 # tie -> even (odd mantissa rounds up)
    assert r[3] == -2.5
    assert (r.view(np.uint32) & 0xFFFF).max() == 0


def test_config_shapes_and_recipes():
    w = I.config(0)
    assert w.layer.io_dtype == "f32" and w.online.n_tok == 32 and w.cached.n_tok == 128
    assert np.allclose(np.linalg.norm(w.online.q, axis=-1), 1.0, atol=1e-6)
    a = np.exp(w.online.g)
    assert a.min() >= 0.9 - 1e-6 and a.max() <= 1.0
    w = I.config(2)
    assert w.online.k.shape == (1536, 1, 128) and w.online.v.shape == (1536, 64, 64)
    assert w.A.shape == (64,) and (w.A < 0).all() and w.online.beta is None
    assert (w.online.k.view(np.uint32) & 0xFFFF).max() == 0      # bf16-representable


def test_ragged_length_recipes():
    rng = np.random.default_rng(3)
    L = I.lengths_fixed_sum(rng, 32, 512, 2048, 32768)
    assert sum(L) == 32768 and min(L) >= 512 and max(L) <= 2048
    for _ in range(20):
        k = int(rng.integers(2, 17))
        L = I.lengths_capped(rng, k, 256, 4096, 16384)
        assert len(L) == k and sum(L) <= 16384 and min(L) >= 256 and max(L) <= 4096


def test_generator_is_deterministic():
    a, b = I.small(I.GDN), I.small(I.GDN)
    assert np.array_equal(a.online.k, b.online.k) and np.array_equal(a.cached.v, b.cached.v)
