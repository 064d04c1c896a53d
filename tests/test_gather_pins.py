"""Pins of the oracle's selected-position gather and of the synthetic selectors.

The gather's definition is fixed by Alg. 1 (replay only U, in context order);
pinned here by a hand-worked example, the all-positions identity, and the
paper's reading that dropping an unselected token equals running it as an
identity transition with no write (alpha = 1, beta = 0).
"""
import numpy as np

import oracle
from paper_2608_11231_amd import inputs as I


def test_hand_worked_rows():
    # request 0: context rows 0..2, request 1: empty, request 2: rows 3..6
    ctx_cu = np.array([0, 3, 3, 7], np.int32)
    sel_cu = np.array([0, 2, 3, 6], np.int32)
    pos = np.array([0, 2, 0, 1, 3, 4], np.int32)
    #   r0 -> rows 0, 2 ; r1 (empty context) -> no row ; r2 -> 4, 6, (position 4 is past its end)
    assert oracle.gather_rows(ctx_cu, sel_cu, pos).tolist() == [0, 2, -1, 4, 6, -1]
    x = np.arange(14, dtype=np.float32).reshape(7, 2)
    (g,) = oracle.gather_selected(ctx_cu, sel_cu, pos, x)
    assert g[[0, 1, 3, 4]].tolist() == [[0, 1], [4, 5], [8, 9], [12, 13]]
    assert np.isnan(g[[2, 5]]).all()


def test_all_positions_is_identity_and_none_passes():
    ctx_cu = np.array([0, 5, 12], np.int32)
    pos = np.concatenate([np.arange(5), np.arange(7)]).astype(np.int32)
    x = np.random.default_rng(0).standard_normal((12, 3, 4)).astype(np.float32)
    a, b = oracle.gather_selected(ctx_cu, ctx_cu, pos, x, None)
    assert np.array_equal(a, x) and b is None


def test_dropping_unselected_tokens_equals_identity_transitions():
    """The recurrence over U alone equals the full-context recurrence in which every
    unselected token has alpha = 1 and beta = 0 (Eq. 3 then gives A_t = I and no write)."""
    rng = np.random.default_rng(3)
    n, h, dk, dv = 40, 2, 8, 6
    k = rng.standard_normal((n, 1, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    q = rng.standard_normal((n, 1, dk))
    v = rng.standard_normal((n, h, dv))
    g = np.log(rng.uniform(0.6, 1.0, (n, h)))
    beta = rng.uniform(0.0, 1.0, (n, h))
    U = I.select_uniform(rng, n, 0.3)
    drop = np.setdiff1d(np.arange(n), U)
    g[drop], beta[drop] = 0.0, 0.0
    S0 = rng.standard_normal((1, h, dv, dk))
    cu = np.array([0, n], np.int32)
    _, S_full = oracle.gdn_scan(cu, q, k, v, g, beta, S0=S0)
    sel_cu = np.array([0, len(U)], np.int32)
    qs, ks, vs, gs, bs = oracle.gather_selected(cu, sel_cu, U, q, k, v, g, beta)
    o_sel, S_sel = oracle.gdn_scan(sel_cu, qs, ks, vs, gs, bs, S0=S0)
    assert np.max(np.abs(S_sel - S_full)) < 1e-12 * np.max(np.abs(S_full))
    o_full, _ = oracle.gdn_scan(cu, q, k, v, g, beta, S0=S0)
    assert np.max(np.abs(o_sel - o_full[U])) < 1e-12 * np.max(np.abs(o_full))


def test_selectors():
    assert I.select_seams([10, 5, 8], 4).tolist() == [8, 9, 10, 11, 13, 14, 15, 16]
    assert I.select_seams([7], 4).tolist() == []
    assert I.select_seams([1, 1, 1], 6).tolist() == [0, 1, 2]
    u = I.select_uniform(np.random.default_rng(1), 1000, 0.2)
    assert len(u) == 200 and np.all(np.diff(u) > 0) and u.min() >= 0 and u.max() < 1000
    cu, pos = I.pack_selection([np.array([1, 2]), np.array([], np.int32), np.array([0])])
    assert cu.tolist() == [0, 2, 2, 3] and pos.tolist() == [1, 2, 0]
