"""ctypes front-end of the C oracle (test infrastructure only).

Every function takes plain numpy arrays in the packed "THD" layout, widens them
to fp64 (exact for fp32/bf16 storage) and returns fp64 results.  See
``lkv_oracle.c`` for the definitions each call evaluates and the passages of the
paper they follow.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Tuple

import numpy as np

from . import build as _build

_lib = None
_lock = threading.Lock()

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)


def load():
    """Load (building first if absent) ``liblkv_oracle.so``."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_build.LIB):
                _build.build()
            lib = ctypes.CDLL(_build.LIB)
            i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
            lib.lkvo_gdn_scan.argtypes = [i64, _ip, i32, i32, i32, i32, _dp, _dp, _dp, _dp, _dp,
                                          dbl, _dp, _dp, _dp]
            lib.lkvo_gdn_transition.argtypes = [i64, _ip, i32, i32, i32, _dp, _dp, _dp, _dp]
            lib.lkvo_ssd_scan.argtypes = [i64, _ip, i32, i32, i32, i32, _dp, _dp, _dp, _dp, _dp,
                                          _dp, _dp, _dp]
            lib.lkvo_ssd_log_decay.argtypes = [i64, _ip, i32, _dp, _dp, _dp]
            lib.lkvo_init_single.argtypes = [i32, i64, _dp, _ip, _dp]
            lib.lkvo_compose_gdn.argtypes = [i32, _ip, _ip, i32, i32, i32, _dp, _dp, _dp]
            lib.lkvo_compose_ssd.argtypes = [i32, _ip, _ip, i32, i32, i32, _dp, _dp, _dp]
            for f in ("lkvo_gdn_scan", "lkvo_gdn_transition", "lkvo_ssd_scan",
                      "lkvo_ssd_log_decay", "lkvo_init_single", "lkvo_compose_gdn",
                      "lkvo_compose_ssd"):
                getattr(lib, f).restype = None
            _lib = lib
    return _lib


def _f64(x):
    return None if x is None else np.ascontiguousarray(x, dtype=np.float64)


def _i32(x):
    return np.ascontiguousarray(x, dtype=np.int32)


def _p(a):
    if a is None:
        return None
    if a.dtype == np.int32:
        return a.ctypes.data_as(_ip)
    return a.ctypes.data_as(_dp)


def gdn_scan(cu, q, k, v, g, beta, scale: float = 1.0, S0=None,
             want_o: bool = True) -> Tuple[Optional[np.ndarray], np.ndarray]:
    """Gated DeltaNet token recurrence (Eq. 1, Eq. 3).  Returns (o, S_final):
    o [n_tok,h_v,dv] (None unless ``want_o``), S_final [n_seq,h_v,dv,dk]."""
    cu = _i32(cu)
    k, v, g, beta = _f64(k), _f64(v), _f64(g), _f64(beta)
    q = _f64(q) if want_o else None
    n_seq = cu.shape[0] - 1
    n_tok, h_qk, dk = k.shape
    h_v, dv = v.shape[1], v.shape[2]
    S0 = _f64(S0)
    S = np.empty((n_seq, h_v, dv, dk), dtype=np.float64)
    o = np.empty((n_tok, h_v, dv), dtype=np.float64) if want_o else None
    load().lkvo_gdn_scan(n_seq, _p(cu), h_qk, h_v, dk, dv, _p(q), _p(k), _p(v), _p(g),
                         _p(beta), float(scale), _p(S0), _p(o), _p(S))
    return o, S


def gdn_transition(cu, k, g, beta) -> np.ndarray:
    """Per-segment Gated DeltaNet transition M = A_1...A_L (Eq. 5), [n_seq,h_v,dk,dk]."""
    cu = _i32(cu)
    k, g, beta = _f64(k), _f64(g), _f64(beta)
    n_seq = cu.shape[0] - 1
    _, h_qk, dk = k.shape
    h_v = g.shape[1]
    M = np.empty((n_seq, h_v, dk, dk), dtype=np.float64)
    load().lkvo_gdn_transition(n_seq, _p(cu), h_qk, h_v, dk, _p(k), _p(g), _p(beta), _p(M))
    return M


def ssd_scan(cu, C, B, x, dt, A, S0=None,
             want_y: bool = True) -> Tuple[Optional[np.ndarray], np.ndarray]:
    """Mamba-2 token recurrence (Eq. 1, Eq. 2).  Returns (y, S_final):
    y [n_tok,H,P], S_final [n_seq,H,P,N]."""
    cu = _i32(cu)
    B, x, dt, A = _f64(B), _f64(x), _f64(dt), _f64(A)
    C = _f64(C) if want_y else None
    n_seq = cu.shape[0] - 1
    n_tok, G, N = B.shape
    H, P = x.shape[1], x.shape[2]
    S0 = _f64(S0)
    S = np.empty((n_seq, H, P, N), dtype=np.float64)
    y = np.empty((n_tok, H, P), dtype=np.float64) if want_y else None
    load().lkvo_ssd_scan(n_seq, _p(cu), G, H, N, P, _p(C), _p(B), _p(x), _p(dt), _p(A),
                         _p(S0), _p(y), _p(S))
    return y, S


def ssd_log_decay(cu, dt, A) -> np.ndarray:
    """Per-segment Mamba-2 log-decay Lambda = A_h sum dt (Eq. 5 scalar), [n_seq,H]."""
    cu = _i32(cu)
    dt, A = _f64(dt), _f64(A)
    n_seq = cu.shape[0] - 1
    H = dt.shape[1]
    Lam = np.empty((n_seq, H), dtype=np.float64)
    load().lkvo_ssd_log_decay(n_seq, _p(cu), H, _p(dt), _p(A), _p(Lam))
    return Lam


def init_single(B_pool, src) -> np.ndarray:
    """Single-block initialisation (Sec. 3.2): S_init[r] = B_pool[src[r]], or 0 for -1."""
    B_pool = _f64(B_pool)
    src = _i32(src)
    n_req = src.shape[0]
    elems = int(np.prod(B_pool.shape[1:]))
    out = np.empty((n_req,) + B_pool.shape[1:], dtype=np.float64)
    load().lkvo_init_single(n_req, elems, _p(B_pool), _p(src), _p(out))
    return out


def compose_gdn(blk_cu, blk_ids, B_pool, M_pool) -> np.ndarray:
    """Exact composition (Eq. 5 back to back = Eq. 6) for Gated DeltaNet."""
    blk_cu, blk_ids = _i32(blk_cu), _i32(blk_ids)
    B_pool, M_pool = _f64(B_pool), _f64(M_pool)
    n_req = blk_cu.shape[0] - 1
    _, h_v, dv, dk = B_pool.shape
    out = np.empty((n_req, h_v, dv, dk), dtype=np.float64)
    load().lkvo_compose_gdn(n_req, _p(blk_cu), _p(blk_ids), h_v, dv, dk, _p(B_pool),
                            _p(M_pool), _p(out))
    return out


def compose_ssd(blk_cu, blk_ids, B_pool, Lam_pool) -> np.ndarray:
    """Exact composition (Eq. 6 with scalar transitions) for Mamba-2."""
    blk_cu, blk_ids = _i32(blk_cu), _i32(blk_ids)
    B_pool, Lam_pool = _f64(B_pool), _f64(Lam_pool)
    n_req = blk_cu.shape[0] - 1
    _, H, P, N = B_pool.shape
    out = np.empty((n_req, H, P, N), dtype=np.float64)
    load().lkvo_compose_ssd(n_req, _p(blk_cu), _p(blk_ids), H, P, N, _p(B_pool),
                            _p(Lam_pool), _p(out))
    return out


def gdn_decode(q, k, v, g, beta, S, scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """One decode step per request (one token each, Eq. 1 and Eq. 3): the token
    recurrence run over single-token segments from the requests' states S
    [n_req,h_v,dv,dk].  Returns (o [n_req,h_v,dv], S_new)."""
    n_req = np.asarray(k).shape[0]
    cu = np.arange(n_req + 1, dtype=np.int32)
    return gdn_scan(cu, q, k, v, g, beta, scale=scale, S0=S)


def ssd_decode(C, B, x, dt, A, S) -> Tuple[np.ndarray, np.ndarray]:
    """One Mamba-2 decode step per request (Eq. 1 and Eq. 2), from states S
    [n_req,H,P,N].  Returns (y [n_req,H,P], S_new)."""
    n_req = np.asarray(B).shape[0]
    cu = np.arange(n_req + 1, dtype=np.int32)
    return ssd_scan(cu, C, B, x, dt, A, S0=S)
