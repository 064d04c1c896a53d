"""Chunkwise fp64 forms of the two recurrences (test infrastructure only).

Splitting a token stream into chunks of C tokens and applying the block map of
Eq. 5 to each chunk gives closed forms per chunk; these are what a chunked GPU
kernel evaluates.  They exist here only so that a test can check, in fp64, that
the chunked algebra reproduces the token recurrence of Eq. 1-3 for any chunk
size, ragged tails and non-zero incoming state.

Library form (state S in R^{dv x dk}, see ``lkv_oracle.c``).  Within one chunk
with token rows Q, K (C x dk), V (C x dv):

Gated DeltaNet
  g_t = sum_{i<=t} log alpha_i,  b_t = exp(g_t),  D_ti = exp(g_t - g_i) (i<=t)
  A   = strictly-lower(D * K K^T),  T = (I + diag(beta) A)^{-1} diag(beta)
  U   = T (V - diag(b) K S0^T)
  O   = scale (diag(b) Q S0^T + (D * Q K^T) U)
  S_C = b_C S0 + U^T diag(b_C / b) K

Mamba-2 SSD (q = C, k = B, v = x, gates l_t = A_h sum_{i<=t} dt_i)
  L_ti = exp(l_t - l_i) (i<=t)
  Y    = (L * C B^T) diag(dt) X + diag(exp(l)) C S0^T
  S_C  = exp(l_C) S0 + X^T diag(dt * exp(l_C - l)) B
"""
from __future__ import annotations

import numpy as np


def gdn_chunkwise(q, k, v, g, beta, S0, chunk: int, scale: float = 1.0):
    """One (segment, head) slice: q,k [T,dk], v [T,dv], g,beta [T], S0 [dv,dk]."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    g, beta = np.asarray(g, np.float64), np.asarray(beta, np.float64)
    S = np.array(S0, dtype=np.float64, copy=True)
    T = k.shape[0]
    o = np.zeros((T, v.shape[1]))
    for c0 in range(0, T, chunk):
        sl = slice(c0, min(T, c0 + chunk))
        Q, K, V, gg, bb = q[sl], k[sl], v[sl], g[sl], beta[sl]
        n = K.shape[0]
        gc = np.cumsum(gg)
        b = np.exp(gc)
        D = np.tril(np.exp(gc[:, None] - gc[None, :]))
        A = np.tril(D * (K @ K.T), -1)
        Tm = np.linalg.inv(np.eye(n) + bb[:, None] * A) * bb[None, :]
        U = Tm @ (V - b[:, None] * (K @ S.T))
        o[sl] = scale * (b[:, None] * (Q @ S.T) + (D * (Q @ K.T)) @ U)
        w = np.exp(gc[-1] - gc)
        S = b[-1] * S + U.T @ (w[:, None] * K)
    return o, S


def ssd_chunkwise(C, B, x, dt, A_h: float, S0, chunk: int):
    """One (segment, head) slice: C,B [T,N], x [T,P], dt [T], S0 [P,N]."""
    C, B, x = (np.asarray(a, dtype=np.float64) for a in (C, B, x))
    dt = np.asarray(dt, np.float64)
    S = np.array(S0, dtype=np.float64, copy=True)
    T = B.shape[0]
    y = np.zeros((T, x.shape[1]))
    for c0 in range(0, T, chunk):
        sl = slice(c0, min(T, c0 + chunk))
        Cc, Bc, X, d = C[sl], B[sl], x[sl], dt[sl]
        l = A_h * np.cumsum(d)
        L = np.tril(np.exp(l[:, None] - l[None, :]))
        y[sl] = (L * (Cc @ Bc.T)) @ (d[:, None] * X) + np.exp(l)[:, None] * (Cc @ S.T)
        w = d * np.exp(l[-1] - l)
        S = np.exp(l[-1]) * S + X.T @ (w[:, None] * Bc)
    return y, S
