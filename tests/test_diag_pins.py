"""Pins of the oracle's relative-error diagnostic and Eq. 7 mismatch recursion."""
import numpy as np

import oracle


def test_rel_error_closed_forms():
    rng = np.random.default_rng(0)
    R = rng.standard_normal((2, 3, 4, 5))
    rel, rg = oracle.rel_error(R, R, group=3)
    assert np.all(rel == 0) and np.all(rg == 0)
    rel, _ = oracle.rel_error(np.zeros_like(R), R)
    assert np.allclose(rel, 1.0, rtol=0, atol=1e-15)
    rel, _ = oracle.rel_error(3 * R, R)                  # ||2R|| / ||R|| = 2
    assert np.allclose(rel, 2.0, rtol=0, atol=1e-14)
    # group figure: one slice exact, one with error E: sqrt(|E|^2 / (|R0|^2 + |R1|^2))
    S = R.copy()
    E = rng.standard_normal((4, 5))
    S[1, 2] += E
    rel, rg = oracle.rel_error(S, R, group=3)
    want = np.sqrt((E ** 2).sum() / (R[1] ** 2).sum())
    assert abs(rg[1] - want) < 1e-14 * want and rg[0] == 0
    assert abs(rel[5] - np.sqrt((E ** 2).sum() / (R[1, 2] ** 2).sum())) < 1e-14 * rel[5]
    rel, _ = oracle.rel_error(np.ones((1, 2, 4)), np.zeros((1, 2, 4)))
    assert np.isinf(rel).all()


def test_mismatch_recursion_matches_composition():
    """Eq. 7: composing perturbed states minus composing the true ones equals the
    recursion, for both transition kinds (this ties the recursion to the composition
    of Eq. 6, whose own pins are brute force)."""
    rng = np.random.default_rng(1)
    K, h, dv, dk = 5, 2, 3, 4
    B = rng.standard_normal((K, h, dv, dk))
    d = 0.1 * rng.standard_normal((K, h, dv, dk))
    M = 0.7 * rng.standard_normal((K, h, dk, dk)) / np.sqrt(dk)
    cu = np.array([0, K], np.int32)
    ids = np.arange(K, dtype=np.int32)
    e = oracle.compose_gdn(cu, ids, B + d, M)[0] - oracle.compose_gdn(cu, ids, B, M)[0]
    assert np.max(np.abs(e - oracle.mismatch_recursion(d, M=M))) < 1e-13
    Lam = -rng.uniform(0, 2, (K, h))
    e = oracle.compose_ssd(cu, ids, B + d, Lam)[0] - oracle.compose_ssd(cu, ids, B, Lam)[0]
    assert np.max(np.abs(e - oracle.mismatch_recursion(d, Lam=Lam))) < 1e-13
    # scalar decays can only retain and sum: with Lambda = 0 the error is the plain sum
    assert np.allclose(oracle.mismatch_recursion(d, Lam=np.zeros((K, h))), d.sum(axis=0), atol=1e-15)
