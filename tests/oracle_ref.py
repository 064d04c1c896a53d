"""Oracle evaluation of a whole workload and the comparison metrics of the tests."""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_11231_amd import inputs as I


def rel_slices(x, ref, lead: int = 2) -> float:
    """max over leading-dim slices of max|x - ref| / max|ref| (normwise-inf relative error)."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    if x.size == 0:
        return 0.0
    x = x.reshape(int(np.prod(x.shape[:lead])), -1)
    ref = ref.reshape(x.shape)
    num = np.max(np.abs(x - ref), axis=1)
    den = np.maximum(np.max(np.abs(ref), axis=1), 1e-30)
    bad = ~np.isfinite(num)
    if bad.any():
        return float("inf")
    return float(np.max(num / den))


def max_abs(x, ref) -> float:
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    if x.size == 0:
        return 0.0
    d = np.abs(x - ref)
    return float("inf") if not np.isfinite(d).all() else float(d.max())


def summaries(w: I.Workload):
    """(B_pool, M_pool) of every cached block: GDN M dense, SSD Lambda."""
    c = w.cached
    if w.layer.family == I.GDN:
        _, B = oracle.gdn_scan(c.cu, None, c.k, c.v, c.g, c.beta, want_o=False)
        M = oracle.gdn_transition(c.cu, c.k, c.g, c.beta)
    else:
        _, B = oracle.ssd_scan(c.cu, None, c.k, c.v, c.g, w.A, want_y=False)
        M = oracle.ssd_log_decay(c.cu, c.g, w.A)
    return B, M


def init_single(w: I.Workload, B):
    return oracle.init_single(B, w.last_blk)


def init_compose(w: I.Workload, B, M):
    if w.layer.family == I.GDN:
        return oracle.compose_gdn(w.blk_cu, w.blk_ids, B, M)
    return oracle.compose_ssd(w.blk_cu, w.blk_ids, B, M)


def scan(w: I.Workload, S0, want_out: bool = True):
    o = w.online
    if w.layer.family == I.GDN:
        return oracle.gdn_scan(o.cu, o.q, o.k, o.v, o.g, o.beta, scale=w.scale, S0=S0, want_o=want_out)
    return oracle.ssd_scan(o.cu, o.q, o.k, o.v, o.g, w.A, S0=S0, want_y=want_out)
