"""Selected-position gather (test infrastructure only).

Alg. 1's recompute step replays only the selected positions U = {i_1 < ... <
i_m} of each request's context, in context order (Sec. 3.1): the recurrent
layer's online stream is the context's token rows at U, and the unselected
tokens' transitions are dropped.  This is the plain definition of that stream,
one row at a time.
"""
from __future__ import annotations

import numpy as np


def gather_rows(ctx_cu, sel_cu, pos):
    """Context row of every selected row j of request r: ctx_cu[r] + pos[j] when the
    position lies inside the request's context, else -1 (no such token)."""
    ctx_cu = np.asarray(ctx_cu, np.int64)
    sel_cu = np.asarray(sel_cu, np.int64)
    pos = np.asarray(pos, np.int64)
    rows = np.full(int(sel_cu[-1]) if len(sel_cu) else 0, -1, np.int64)
    for r in range(len(sel_cu) - 1):
        n_ctx = ctx_cu[r + 1] - ctx_cu[r]
        for j in range(sel_cu[r], sel_cu[r + 1]):
            if 0 <= pos[j] < n_ctx:
                rows[j] = ctx_cu[r] + pos[j]
    return rows


def gather_selected(ctx_cu, sel_cu, pos, *arrays):
    """Each array's rows at the selected positions (None passes through); rows
    with no source token are NaN."""
    rows = gather_rows(ctx_cu, sel_cu, pos)
    out = []
    for a in arrays:
        if a is None:
            out.append(None)
            continue
        res = np.empty((len(rows),) + a.shape[1:], dtype=a.dtype)
        for j, row in enumerate(rows):
            res[j] = a[row] if row >= 0 else np.nan
        out.append(res)
    return out
