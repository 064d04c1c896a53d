"""Pins of the CPU oracle against what the paper and the mathematics fix.

The paper prints no numerical worked example for a recurrent layer, so each
pin is a closed form, an invariant, a special case or a brute-force evaluation
that does not share the oracle's rank-1 shortcuts:

P1  brute force with explicit dense per-token transition matrices (Eq. 1, 3),
    also in the paper's own (transposed) orientation;
P2  the chunkwise form equals the token recurrence (Eq. 5 applied per chunk);
P3  exact composition equals one scan over the concatenated blocks (Eq. 5, 6),
    equals the explicit sum form of Eq. 6, and (M,B) pairs compose associatively;
P4  K = 1 composition returns the cached state;
P5  identity gates (alpha = 1, beta = 0) leave the state unchanged;
    beta = 0 gives pure decay; Mamba-2 with A = 0 is plain linear attention;
P6  delta-rule overwrite with alpha = beta = 1 and a basis key;
P7  the Mamba-2 quadratic (dual) form;
P8  degenerate compositions (all M = 0, all M = I);
P9  the mismatch recursion of Eq. 7;
plus a hand-derived exact 2x2 example and the single-block copy.
"""
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
from oracle.chunkwise import gdn_chunkwise, ssd_chunkwise

RNG = np.random.default_rng(12345)


def _unit(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _gdn_slice(T, dk, dv, rng, alpha_lo=0.6):
    q = _unit(rng.standard_normal((T, dk)))
    k = _unit(rng.standard_normal((T, dk)))
    v = rng.standard_normal((T, dv))
    g = np.log(rng.uniform(alpha_lo, 1.0, T))
    beta = rng.uniform(0.0, 1.0, T)
    return q, k, v, g, beta


def _as_thd(*arrs):
    return [a[:, None, :] if a.ndim == 2 else a[:, None] for a in arrs]


def _brute_gdn(q, k, v, g, beta, S0, scale=1.0):
    """Dense per-token transitions: S_t = S_{t-1} A_t + beta v k^T, A_t = alpha (I - beta k k^T)."""
    dk = k.shape[1]
    S = S0.copy()
    o = []
    for t in range(k.shape[0]):
        A = np.exp(g[t]) * (np.eye(dk) - beta[t] * np.outer(k[t], k[t]))
        S = S @ A + beta[t] * np.outer(v[t], k[t])
        o.append(scale * S @ q[t])
    return np.array(o), S


def _brute_gdn_paper(k, v, g, beta, Sp0):
    """Paper orientation (Eq. 1, 3): S_i = T_i S_{i-1} + u_i, S in R^{dk x dv}, u = beta k v^T."""
    dk = k.shape[1]
    S = Sp0.copy()
    for t in range(k.shape[0]):
        Tt = np.exp(g[t]) * (np.eye(dk) - beta[t] * np.outer(k[t], k[t]))
        S = Tt @ S + beta[t] * np.outer(k[t], v[t])
    return S


def _brute_M(k, g, beta):
    dk = k.shape[1]
    M = np.eye(dk)
    for t in range(k.shape[0]):
        M = M @ (np.exp(g[t]) * (np.eye(dk) - beta[t] * np.outer(k[t], k[t])))
    return M


def _scan1(q, k, v, g, beta, S0=None, scale=1.0):
    cu = np.array([0, k.shape[0]], np.int32)
    qq, kk, vv, gg, bb = _as_thd(q, k, v, g, beta)
    o, S = oracle.gdn_scan(cu, qq, kk, vv, gg, bb, scale=scale,
                           S0=None if S0 is None else S0[None, None])
    return o[:, 0], S[0, 0]


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ---------------------------------------------------------------- P1
@pytest.mark.parametrize("dk,dv,T", [(4, 3, 9), (8, 8, 33), (16, 12, 64)])
def test_p1_gdn_brute_force(dk, dv, T):
    q, k, v, g, beta = _gdn_slice(T, dk, dv, RNG)
    S0 = RNG.standard_normal((dv, dk))
    o_b, S_b = _brute_gdn(q, k, v, g, beta, S0, scale=0.7)
    o, S = _scan1(q, k, v, g, beta, S0, scale=0.7)
    assert _rel(S, S_b) < 1e-13 and _rel(o, o_b) < 1e-13
    # the paper's left-multiplied dk x dv state is the transpose of the library state
    Sp = _brute_gdn_paper(k, v, g, beta, S0.T)
    assert _rel(S, Sp.T) < 1e-13
    M = oracle.gdn_transition(np.array([0, T], np.int32), k[:, None], g[:, None], beta[:, None])
    assert _rel(M[0, 0], _brute_M(k, g, beta)) < 1e-13


def test_p1_packed_grouped_heads():
    """Several segments and 2 value heads per q/k head: every slice equals brute force."""
    lens = [5, 0, 17, 9]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n, h_qk, h_v, dk, dv = cu[-1], 2, 4, 8, 6
    q = _unit(RNG.standard_normal((n, h_qk, dk)))
    k = _unit(RNG.standard_normal((n, h_qk, dk)))
    v = RNG.standard_normal((n, h_v, dv))
    g = np.log(RNG.uniform(0.7, 1.0, (n, h_v)))
    beta = RNG.uniform(0, 1, (n, h_v))
    S0 = RNG.standard_normal((len(lens), h_v, dv, dk))
    o, S = oracle.gdn_scan(cu, q, k, v, g, beta, scale=1.0, S0=S0)
    M = oracle.gdn_transition(cu, k, g, beta)
    for s in range(len(lens)):
        sl = slice(cu[s], cu[s + 1])
        for h in range(h_v):
            hq = h // (h_v // h_qk)
            ob, Sb = _brute_gdn(q[sl, hq], k[sl, hq], v[sl, h], g[sl, h], beta[sl, h], S0[s, h])
            assert _rel(S[s, h], Sb) < 1e-13
            if lens[s]:
                assert _rel(o[sl, h], ob) < 1e-13
            assert _rel(M[s, h], _brute_M(k[sl, hq], g[sl, h], beta[sl, h])) < 1e-13


def test_p1_ssd_brute_force():
    T, N, P = 41, 8, 5
    C = _unit(RNG.standard_normal((T, N)))
    B = _unit(RNG.standard_normal((T, N)))
    x = RNG.standard_normal((T, P))
    dt = np.log1p(np.exp(RNG.standard_normal(T) - 2.0))
    A = -2.5
    S0 = RNG.standard_normal((P, N))
    S = S0.copy()
    yb = []
    for t in range(T):   # S_t = S_{t-1} (a_t I) + dt x B^T
        S = S @ (np.exp(dt[t] * A) * np.eye(N)) + dt[t] * np.outer(x[t], B[t])
        yb.append(S @ C[t])
    y, So = oracle.ssd_scan(np.array([0, T], np.int32), C[:, None], B[:, None], x[:, None],
                            dt[:, None], np.array([A]), S0=S0[None, None])
    assert _rel(So[0, 0], S) < 1e-13 and _rel(y[:, 0], np.array(yb)) < 1e-13
    Lam = oracle.ssd_log_decay(np.array([0, T], np.int32), dt[:, None], np.array([A]))
    assert abs(Lam[0, 0] - A * dt.sum()) < 1e-13


# ---------------------------------------------------------------- hand-derived example
def test_worked_example_exact():
    """dk = dv = 2, two tokens, exact rationals worked by hand (Eq. 3, Eq. 5).

    t=1: k=(1,0), v=(2,3), alpha=1/2, beta=1/2, q=(0,1); t=2: k=(3/5,4/5),
    v=(1,-1), alpha=beta=1, q=(1,0); S0 = I.
    S1 = [[5/4,0],[3/2,1/2]], o1 = (0,1/2); S2 = [[7/5,1/5],[3/25,-67/50]],
    o2 = (7/5,3/25); M = [[4/25,-3/25],[-6/25,9/50]], B = [[31/25,8/25],[9/25,-38/25]].
    """
    k = np.array([[1, 0], [0.6, 0.8]])
    v = np.array([[2, 3], [1, -1]], float)
    q = np.array([[0, 1], [1, 0]], float)
    g = np.log(np.array([0.5, 1.0]))
    beta = np.array([0.5, 1.0])
    f = lambda m: np.array([[float(Fr(x)) for x in r] for r in m])
    o, S = _scan1(q, k, v, g, beta, np.eye(2))
    assert np.allclose(S, f([["7/5", "1/5"], ["3/25", "-67/50"]]), atol=1e-15, rtol=0)
    assert np.allclose(o, f([["0", "1/2"], ["7/5", "3/25"]]), atol=1e-15, rtol=0)
    M = oracle.gdn_transition(np.array([0, 2], np.int32), k[:, None], g[:, None], beta[:, None])
    assert np.allclose(M[0, 0], f([["4/25", "-3/25"], ["-6/25", "9/50"]]), atol=1e-15, rtol=0)
    _, Bst = _scan1(q, k, v, g, beta)
    assert np.allclose(Bst, f([["31/25", "8/25"], ["9/25", "-38/25"]]), atol=1e-15, rtol=0)


# ---------------------------------------------------------------- P2
@pytest.mark.parametrize("chunk", [1, 2, 16, 64, 150])
def test_p2_gdn_chunkwise_equals_sequential(chunk):
    T, dk, dv = 150, 16, 12
    q, k, v, g, beta = _gdn_slice(T, dk, dv, RNG, alpha_lo=0.8)
    S0 = RNG.standard_normal((dv, dk))
    o, S = _scan1(q, k, v, g, beta, S0, scale=0.5)
    oc, Sc = gdn_chunkwise(q, k, v, g, beta, S0, chunk, scale=0.5)
    assert _rel(Sc, S) < 1e-12 and _rel(oc, o) < 1e-12


@pytest.mark.parametrize("chunk", [1, 2, 16, 64, 150])
def test_p2_ssd_chunkwise_equals_sequential(chunk):
    T, N, P = 150, 16, 8
    C = _unit(RNG.standard_normal((T, N)))
    B = _unit(RNG.standard_normal((T, N)))
    x = RNG.standard_normal((T, P))
    dt = np.log1p(np.exp(RNG.standard_normal(T) - 3.0))
    A = -3.0
    S0 = RNG.standard_normal((P, N))
    y, S = oracle.ssd_scan(np.array([0, T], np.int32), C[:, None], B[:, None], x[:, None],
                           dt[:, None], np.array([A]), S0=S0[None, None])
    yc, Sc = ssd_chunkwise(C, B, x, dt, A, S0, chunk)
    assert _rel(Sc, S[0, 0]) < 1e-12 and _rel(yc, y[:, 0]) < 1e-12


# ---------------------------------------------------------------- P3, P4, P8, P9
def _gdn_blocks(lens, h=2, dk=8, dv=6, alpha_lo=0.93):
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = int(cu[-1])
    k = _unit(RNG.standard_normal((n, h, dk)))
    q = _unit(RNG.standard_normal((n, h, dk)))
    v = RNG.standard_normal((n, h, dv))
    g = np.log(RNG.uniform(alpha_lo, 1.0, (n, h)))
    beta = RNG.uniform(0, 0.5, (n, h))
    return cu, q, k, v, g, beta


def test_p3_compose_equals_concatenated_scan_gdn():
    lens = [13, 29, 7, 40]
    cu, q, k, v, g, beta = _gdn_blocks(lens)
    _, Bp = oracle.gdn_scan(cu, q, k, v, g, beta, want_o=False)
    Mp = oracle.gdn_transition(cu, k, g, beta)
    S = oracle.compose_gdn(np.array([0, 4], np.int32), np.arange(4, dtype=np.int32), Bp, Mp)
    _, Sfull = oracle.gdn_scan(np.array([0, cu[-1]], np.int32), q, k, v, g, beta, want_o=False)
    assert _rel(S[0], Sfull[0]) < 1e-12
    # Eq. 6 written out: sum_j B_j M_{j+1} ... M_K
    for h in range(Bp.shape[1]):
        acc = np.zeros_like(Bp[0, h])
        for j in range(4):
            P = np.eye(Mp.shape[-1])
            for m in range(j + 1, 4):
                P = P @ Mp[m, h]
            acc += Bp[j, h] @ P
        assert _rel(S[0, h], acc) < 1e-12
    # associativity of (M_a, B_a) o (M_b, B_b) = (M_a M_b, B_a M_b + B_b)
    cu2 = np.array([0, cu[2], cu[4]], np.int32)
    _, B2 = oracle.gdn_scan(cu2, q, k, v, g, beta, want_o=False)
    M2 = oracle.gdn_transition(cu2, k, g, beta)
    for h in range(Bp.shape[1]):
        assert _rel(M2[0, h], Mp[0, h] @ Mp[1, h]) < 1e-12
        assert _rel(B2[0, h], Bp[0, h] @ Mp[1, h] + Bp[1, h]) < 1e-12
    # split-point invariance: compose over the two halves equals the full compose
    Sh = oracle.compose_gdn(np.array([0, 2], np.int32), np.arange(2, dtype=np.int32), B2, M2)
    assert _rel(Sh[0], S[0]) < 1e-12


def test_p3_compose_equals_concatenated_scan_ssd():
    lens = [11, 30, 5]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n, G, H, N, P = int(cu[-1]), 1, 3, 8, 4
    C = _unit(RNG.standard_normal((n, G, N)))
    B = _unit(RNG.standard_normal((n, G, N)))
    x = RNG.standard_normal((n, H, P))
    dt = np.log1p(np.exp(RNG.standard_normal((n, H)) - 4.0))
    A = -np.exp(RNG.uniform(0, np.log(4.0), H))
    _, Bp = oracle.ssd_scan(cu, C, B, x, dt, A, want_y=False)
    Lam = oracle.ssd_log_decay(cu, dt, A)
    S = oracle.compose_ssd(np.array([0, 3], np.int32), np.arange(3, dtype=np.int32), Bp, Lam)
    _, Sf = oracle.ssd_scan(np.array([0, n], np.int32), C, B, x, dt, A, want_y=False)
    assert _rel(S[0], Sf[0]) < 1e-12
    for h in range(H):   # Eq. 6 with scalar transitions
        acc = sum(np.exp(sum(Lam[m, h] for m in range(j + 1, 3))) * Bp[j, h] for j in range(3))
        assert _rel(S[0, h], acc) < 1e-12


def test_p4_single_block_compose_returns_cached_state():
    cu, q, k, v, g, beta = _gdn_blocks([19, 5])
    _, Bp = oracle.gdn_scan(cu, q, k, v, g, beta, want_o=False)
    Mp = np.full((2, 2, 8, 8), np.nan)   # never read for a request's first block
    S = oracle.compose_gdn(np.array([0, 1, 2], np.int32), np.array([1, 0], np.int32), Bp, Mp)
    assert np.array_equal(S[0], Bp[1]) and np.array_equal(S[1], Bp[0])
    Lam = np.full((2, 2), np.nan)
    S2 = oracle.compose_ssd(np.array([0, 1], np.int32), np.array([1], np.int32), Bp, Lam)
    assert np.array_equal(S2[0], Bp[1])


def test_p8_degenerate_compositions():
    K, h, dv, dk = 5, 2, 3, 4
    Bp = RNG.standard_normal((K, h, dv, dk))
    ids = np.arange(K, dtype=np.int32)
    cu = np.array([0, K], np.int32)
    S0 = oracle.compose_gdn(cu, ids, Bp, np.zeros((K, h, dk, dk)))
    assert np.array_equal(S0[0], Bp[K - 1])
    assert np.array_equal(S0[0], oracle.init_single(Bp, np.array([K - 1], np.int32))[0])
    SI = oracle.compose_gdn(cu, ids, Bp, np.broadcast_to(np.eye(dk), (K, h, dk, dk)))
    assert _rel(SI[0], Bp.sum(axis=0)) < 1e-14
    Sz = oracle.compose_gdn(np.array([0, 0], np.int32), ids[:0], Bp, np.zeros((K, h, dk, dk)))
    assert np.array_equal(Sz[0], np.zeros((h, dv, dk)))


def test_p9_mismatch_recursion():
    """Eq. 7 (library form): perturbing each cached state by delta_j gives a composed-state
    error obeying e_j = e_{j-1} M_j + delta_j."""
    K, h, dv, dk = 6, 2, 3, 5
    Bp = RNG.standard_normal((K, h, dv, dk))
    Mp = 0.6 * RNG.standard_normal((K, h, dk, dk)) / np.sqrt(dk)
    d = 1e-3 * RNG.standard_normal((K, h, dv, dk))
    e_prev = np.zeros((h, dv, dk))
    for j in range(1, K + 1):
        cu = np.array([0, j], np.int32)
        ids = np.arange(j, dtype=np.int32)
        e = oracle.compose_gdn(cu, ids, Bp + d, Mp)[0] - oracle.compose_gdn(cu, ids, Bp, Mp)[0]
        pred = d[j - 1] if j == 1 else np.einsum("hij,hjk->hik", e_prev, Mp[j - 1]) + d[j - 1]
        assert np.max(np.abs(e - pred)) < 1e-12
        e_prev = e


# ---------------------------------------------------------------- P5, P6
def test_p5_identity_gates_leave_state_unchanged():
    T, dk, dv = 20, 8, 5
    q, k, v, _, _ = _gdn_slice(T, dk, dv, RNG)
    S0 = RNG.standard_normal((dv, dk))
    _, S = _scan1(q, k, v, np.zeros(T), np.zeros(T), S0)
    assert np.array_equal(S, S0)
    M = oracle.gdn_transition(np.array([0, T], np.int32), k[:, None], np.zeros((T, 1)),
                              np.zeros((T, 1)))
    assert np.array_equal(M[0, 0], np.eye(dk))
    _, Bz = _scan1(q, k, v, np.zeros(T), np.zeros(T))
    assert np.array_equal(Bz, np.zeros((dv, dk)))


def test_p5_pure_decay_and_transition_from_zero_values():
    T, dk, dv = 25, 8, 5
    q, k, v, g, beta = _gdn_slice(T, dk, dv, RNG)
    S0 = RNG.standard_normal((dv, dk))
    _, S = _scan1(q, k, v, g, np.zeros(T), S0)
    assert _rel(S, np.exp(g.sum()) * S0) < 1e-13
    # with v = 0 the block maps S0 to S0 M (Eq. 5 with zero local state)
    _, S = _scan1(q, k, np.zeros_like(v), g, beta, S0)
    M = oracle.gdn_transition(np.array([0, T], np.int32), k[:, None], g[:, None], beta[:, None])
    assert _rel(S, S0 @ M[0, 0]) < 1e-13


def test_p5_ssd_zero_decay_is_linear_attention():
    T, N, P = 30, 6, 4
    C = RNG.standard_normal((T, N))
    B = RNG.standard_normal((T, N))
    x = RNG.standard_normal((T, P))
    dt = RNG.uniform(0.01, 0.3, T)
    S0 = RNG.standard_normal((P, N))
    y, S = oracle.ssd_scan(np.array([0, T], np.int32), C[:, None], B[:, None], x[:, None],
                           dt[:, None], np.array([0.0]), S0=S0[None, None])
    Sc = S0[None] + np.cumsum(dt[:, None, None] * x[:, :, None] * B[:, None, :], axis=0)
    assert _rel(S[0, 0], Sc[-1]) < 1e-13
    assert _rel(y[:, 0], np.einsum("tpn,tn->tp", Sc, C)) < 1e-13
    # and with x = 0 the state decays by exp(Lambda)
    _, S = oracle.ssd_scan(np.array([0, T], np.int32), C[:, None], B[:, None],
                           np.zeros_like(x)[:, None], dt[:, None], np.array([-1.7]),
                           S0=S0[None, None])
    Lam = oracle.ssd_log_decay(np.array([0, T], np.int32), dt[:, None], np.array([-1.7]))
    assert _rel(S[0, 0], np.exp(Lam[0, 0]) * S0) < 1e-13


def test_p6_delta_rule_overwrite():
    dk, dv = 6, 4
    S0 = RNG.standard_normal((dv, dk))
    for j in range(dk):
        k = np.zeros((1, dk)); k[0, j] = 1.0
        v = RNG.standard_normal((1, dv))
        _, S = _scan1(np.zeros((1, dk)), k, v, np.zeros(1), np.ones(1), S0)
        others = [c for c in range(dk) if c != j]
        assert np.array_equal(S[:, others], S0[:, others])      # untouched columns: exact
        assert np.max(np.abs(S[:, j] - v[0])) < 1e-15          # s + (v - s): one rounding


# ---------------------------------------------------------------- P7
def test_p7_ssd_dual_form():
    T, N, P = 37, 8, 5
    C = _unit(RNG.standard_normal((T, N)))
    B = _unit(RNG.standard_normal((T, N)))
    x = RNG.standard_normal((T, P))
    dt = np.log1p(np.exp(RNG.standard_normal(T) - 2.0))
    A = -1.3
    S0 = RNG.standard_normal((P, N))
    y, _ = oracle.ssd_scan(np.array([0, T], np.int32), C[:, None], B[:, None], x[:, None],
                           dt[:, None], np.array([A]), S0=S0[None, None])
    l = A * np.cumsum(dt)
    L = np.tril(np.exp(l[:, None] - l[None, :]))
    Y = (L * (C @ B.T)) @ (dt[:, None] * x) + np.exp(l)[:, None] * (C @ S0.T)
    assert _rel(y[:, 0], Y) < 1e-12


# ---------------------------------------------------------------- single-block copy
def test_init_single_is_exact_copy():
    Bp = RNG.standard_normal((7, 3, 4, 5))
    src = np.array([6, -1, 0, 6], np.int32)
    S = oracle.init_single(Bp, src)
    assert np.array_equal(S[0], Bp[6]) and np.array_equal(S[2], Bp[0])
    assert np.array_equal(S[3], Bp[6]) and np.array_equal(S[1], np.zeros((3, 4, 5)))


# ---------------------------------------------------------------- planted mistakes are caught
def test_pins_detect_planted_mistakes():
    """Plausible slips in the recurrence (dropped gate on the read, wrong sign, transposed
    write) differ from brute force by far more than the tolerance used above."""
    T, dk, dv = 12, 6, 4
    q, k, v, g, beta = _gdn_slice(T, dk, dv, RNG)
    S0 = RNG.standard_normal((dv, dk))
    _, Sb = _brute_gdn(q, k, v, g, beta, S0)

    def variant(kind):
        S = S0.copy()
        for t in range(T):
            a, b = np.exp(g[t]), beta[t]
            sk = S @ k[t]
            if kind == "no_alpha_in_read":
                S = a * S + b * np.outer(v[t] - sk, k[t])
            elif kind == "sign":
                S = a * S + b * np.outer(v[t] + a * sk, k[t])
            elif kind == "transposed_write":
                S = a * S + b * np.outer(v[t] - a * sk, k[t])[:, ::-1]
        return S

    for kind in ("no_alpha_in_read", "sign", "transposed_write"):
        assert _rel(variant(kind), Sb) > 1e-3


# ---------------------------------------------------------------- decode step
def test_decode_step_matches_dense_transition():
    """One decode step per request (Eq. 1 with Eq. 3) against an explicit dense
    transition S A_t + beta v k^T, with grouped heads and distinct requests."""
    n_req, h_qk, h_v, dk, dv = 3, 2, 4, 6, 5
    q = _unit(RNG.standard_normal((n_req, h_qk, dk)))
    k = _unit(RNG.standard_normal((n_req, h_qk, dk)))
    v = RNG.standard_normal((n_req, h_v, dv))
    g = np.log(RNG.uniform(0.5, 1.0, (n_req, h_v)))
    beta = RNG.uniform(0.0, 1.0, (n_req, h_v))
    S0 = RNG.standard_normal((n_req, h_v, dv, dk))
    o, S = oracle.gdn_decode(q, k, v, g, beta, S0, scale=0.6)
    for r in range(n_req):
        for h in range(h_v):
            hq = h // (h_v // h_qk)
            A = np.exp(g[r, h]) * (np.eye(dk) - beta[r, h] * np.outer(k[r, hq], k[r, hq]))
            Sb = S0[r, h] @ A + beta[r, h] * np.outer(v[r, h], k[r, hq])
            assert _rel(S[r, h], Sb) < 1e-13
            assert _rel(o[r, h], 0.6 * Sb @ q[r, hq]) < 1e-13


def test_decode_from_zero_state_is_rank_one_write():
    """From S = 0 one step writes beta v k^T, so o = scale beta (k.q) v."""
    dk, dv = 8, 3
    q = _unit(RNG.standard_normal((1, 1, dk)))
    k = _unit(RNG.standard_normal((1, 1, dk)))
    v = RNG.standard_normal((1, 1, dv))
    o, S = oracle.gdn_decode(q, k, v, np.array([[-0.3]]), np.array([[0.4]]),
                             np.zeros((1, 1, dv, dk)), scale=2.0)
    assert _rel(S[0, 0], 0.4 * np.outer(v[0, 0], k[0, 0])) < 1e-14
    assert _rel(o[0, 0], 2.0 * 0.4 * (k[0, 0] @ q[0, 0]) * v[0, 0]) < 1e-14


def test_decode_steps_chain_to_one_scan():
    """T decode steps from S0 equal the brute-force recurrence over the T tokens."""
    T, dk, dv = 7, 5, 4
    q, k, v, g, beta = _gdn_slice(T, dk, dv, RNG)
    S0 = RNG.standard_normal((dv, dk))
    ob, Sb = _brute_gdn(q, k, v, g, beta, S0, scale=0.9)
    S = S0[None, None].copy()
    for t in range(T):
        o, S = oracle.gdn_decode(q[t][None, None], k[t][None, None], v[t][None, None],
                                 g[t].reshape(1, 1), beta[t].reshape(1, 1), S, scale=0.9)
        assert _rel(o[0, 0], ob[t]) < 1e-13
    assert _rel(S[0, 0], Sb) < 1e-13


def test_ssd_decode_closed_form():
    """Mamba-2 step (Eq. 2): S <- exp(dt A_h) S + dt x B^T, y = S C, per request and head."""
    n_req, G, H, N, P = 2, 1, 3, 6, 4
    C = RNG.standard_normal((n_req, G, N))
    B = RNG.standard_normal((n_req, G, N))
    x = RNG.standard_normal((n_req, H, P))
    dt = RNG.uniform(0.01, 0.5, (n_req, H))
    A = -RNG.uniform(0.5, 3.0, H)
    S0 = RNG.standard_normal((n_req, H, P, N))
    y, S = oracle.ssd_decode(C, B, x, dt, A, S0)
    for r in range(n_req):
        for h in range(H):
            Sb = np.exp(dt[r, h] * A[h]) * S0[r, h] + dt[r, h] * np.outer(x[r, h], B[r, 0])
            assert _rel(S[r, h], Sb) < 1e-13
            assert _rel(y[r, h], Sb @ C[r, 0]) < 1e-13
