"""Relative-error diagnostic and the mismatch recursion (test infrastructure only).

Sec. 3.2 probes a constructed initial state against the true full-prefix state
S* by the relative error ||S_init - S*|| / ||S*||, one number per layer; the
norm is read as the Frobenius norm over the layer's state (all its heads).
Eq. 7 says how the gap between the composed state and the true state evolves
block by block when each cached summary carries a fresh mismatch delta_j:
e_j = T_j e_{j-1} + delta_j (paper orientation), i.e. e_j = e_{j-1} M_j +
delta_j in the library's right-multiplied form.
"""
from __future__ import annotations

import numpy as np


def rel_error(S, S_ref, slice_dims: int = 2, group: int = 0):
    """(rel per slice, rel per group of ``group`` consecutive slices or None), fp64."""
    S = np.asarray(S, np.float64)
    R = np.asarray(S_ref, np.float64)
    n = int(np.prod(S.shape[:S.ndim - slice_dims]))
    d2 = ((S - R) ** 2).reshape(n, -1).sum(axis=1)
    r2 = (R ** 2).reshape(n, -1).sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.sqrt(d2) / np.sqrt(r2)
        rg = None
        if group:
            rg = np.sqrt(d2.reshape(-1, group).sum(axis=1)) / np.sqrt(r2.reshape(-1, group).sum(axis=1))
    return rel, rg


def mismatch_recursion(deltas, M=None, Lam=None):
    """e_K of Eq. 7 for one request: deltas [K, h, dv, dk]; Gated DeltaNet
    transitions M [K, h, dk, dk] or Mamba-2 log-decays Lam [K, h].  The first
    block's transition is never applied (e_1 = delta_1)."""
    deltas = np.asarray(deltas, np.float64)
    e = deltas[0].copy()
    for j in range(1, deltas.shape[0]):
        if M is not None:
            e = np.einsum("hij,hjk->hik", e, np.asarray(M[j], np.float64)) + deltas[j]
        else:
            e = np.exp(np.asarray(Lam[j], np.float64))[:, None, None] * e + deltas[j]
    return e
