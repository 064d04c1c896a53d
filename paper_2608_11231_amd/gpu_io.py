"""Move seeded workloads (``inputs.Workload``) onto the GPU and run the path.

Marshalling only: tensors are created with torch on the current GPU and the
computation is done by liblkv.so through ``lkv``.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import inputs as I
from . import lkv

_TORCH = {"bf16": torch.bfloat16, "f32": torch.float32}


def layer_struct(layer: I.Layer) -> lkv.Layer:
    return lkv.make_layer(layer.family, layer.h_qk, layer.h_v, layer.dk, layer.dv, layer.chunk,
                          _TORCH[layer.io_dtype], _TORCH[layer.gate_dtype])


def _t(x: Optional[np.ndarray], dtype, device) -> Optional[torch.Tensor]:
    if x is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dtype)


def sp_pieces(w: I.Workload) -> int:
    """Piece count for the sequence-parallel scan, or 0 for the serial one: split
    the requests' streams only when their (request, head, 64-row tile) chains
    fill less than the 256 CUs, into at most as many pieces as fill them, each
    of at least two chunks."""
    L = w.layer
    chains = w.n_req * L.h_v * max(1, L.dv // 64)
    if chains >= 256 or w.n_req == 0:
        return 0
    mean_chunks = w.online.n_tok / w.n_req / L.chunk
    p = 1
    while p * 2 * chains <= 256 and p * 2 <= mean_chunks / 2 and p * 2 <= 8:
        p *= 2
    return p if p > 1 else 0


def fold_dropped_blocks(w: I.Workload):
    """Pool rows whose transition no composition of ``w`` reads: every block that
    is not at position 2..K of some request."""
    read = set()
    for r in range(w.n_req):
        read.update(int(b) for b in w.blk_ids[w.blk_cu[r] + 1:w.blk_cu[r + 1]])
    return sorted(set(range(w.n_blk)) - read)


class GpuTokens:
    """A token stream resident in HBM plus its C struct."""

    def __init__(self, tok: I.Tokens, layer: I.Layer, A: Optional[np.ndarray], device="cuda",
                 with_q: bool = True):
        io = _TORCH[layer.io_dtype]
        gate = _TORCH[layer.gate_dtype] if layer.family == I.GDN else torch.float32
        self.n_tok = tok.n_tok
        self.cu = _t(tok.cu, torch.int32, device)
        self.q = _t(tok.q, io, device) if with_q else None
        self.k = _t(tok.k, io, device)
        self.v = _t(tok.v, io, device)
        self.g = _t(tok.g, gate, device)
        self.beta = _t(tok.beta, gate, device)
        self.A = _t(A, torch.float32, device) if layer.family == I.SSD else None
        self.struct = lkv.make_tokens(self.cu, self.n_tok, self.q, self.k, self.v, self.g, self.beta,
                                      self.A)


class GpuWorkload:
    """All device tensors of a workload: cached blocks, online tokens, index arrays,
    the block pools and the state buffers."""

    def __init__(self, w: I.Workload, device="cuda", with_cached: bool = True):
        self.w = w
        L = w.layer
        self.layer = layer_struct(L)
        self.online = GpuTokens(w.online, L, w.A, device)
        self.cached = GpuTokens(w.cached, L, w.A, device, with_q=False) if with_cached else None
        self.blk_ids = _t(w.blk_ids, torch.int32, device)
        self.blk_cu = _t(w.blk_cu, torch.int32, device)
        self.last_blk = _t(w.last_blk, torch.int32, device)
        f32 = dict(device=device, dtype=torch.float32)
        self.B_pool = torch.empty((w.n_blk, L.h_v, L.dv, L.dk), **f32)
        if L.family == I.GDN:
            self.M_pool = torch.empty((w.n_blk, L.h_v, L.dk, L.dk), **f32)
        else:
            self.M_pool = torch.empty((w.n_blk, L.h_v), **f32)
        self.S_single = torch.empty((w.n_req, L.h_v, L.dv, L.dk), **f32)
        self.S_exact = torch.empty_like(self.S_single)
        self.S_final = torch.empty_like(self.S_single)
        self.out = torch.empty((w.online.n_tok, L.h_v, L.dv), device=device, dtype=_TORCH[L.io_dtype])

    # -- the path's calls ---------------------------------------------------------
    def block_summary(self, B: bool = True, M: bool = True, stream=None):
        lkv.block_summary(self.layer, self.cached.struct, self.B_pool if B else None,
                          self.M_pool if M else None, stream)

    def fold_view(self) -> "GpuTokens":
        """The cached stream as the composition's transition fold needs it.  The
        composition never reads the transition of a request's first block (Eq. 6
        starts from that block's state), so a block whose transition no request
        reads -- one that is only ever some request's first block, or is in no
        request at all -- becomes an empty segment (its M_pool row turns into the
        identity, or Lambda = 0).  A block that is first in one request and a
        later block of another keeps its rows: position-independent caching
        reuses one cached block in any position (Sec. 3.2).  Pool row b stays
        segment b."""
        if getattr(self, "_fold_view", None) is None:
            w, c = self.w, self.w.cached
            drop = fold_dropped_blocks(w)
            lens = np.diff(c.cu).astype(np.int64)
            keep = np.ones(c.n_tok, bool)
            for b in drop:
                keep[c.cu[b]:c.cu[b + 1]] = False
                lens[b] = 0
            cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
            tok = I.Tokens(cu, None, c.k[keep], None, c.g[keep], None if c.beta is None else c.beta[keep])
            self._fold_view = GpuTokens(tok, w.layer, w.A, with_q=False)
        return self._fold_view

    def fold_transitions(self, stream=None):
        """The transitions M_k (Lambda_k) of blocks 2..K of every request, as the
        exact composition reads them (the online fold of exact composition)."""
        lkv.block_summary(self.layer, self.fold_view().struct, None, self.M_pool, stream)

    def init_single(self, stream=None):
        lkv.init_single(self.layer, self.w.n_blk, self.B_pool, self.last_blk, self.S_single, stream)

    def init_compose(self, stream=None):
        lkv.init_compose(self.layer, self.w.n_blk, self.B_pool, self.M_pool, self.blk_ids, self.blk_cu,
                         int(self.w.blk_cu[-1]), self.S_exact, stream)

    def scan(self, S_init: Optional[torch.Tensor], stream=None, pieces: int = 0):
        """The online chunk scan from S_init; with ``pieces`` > 1 the sequence-parallel
        form (each request's stream in that many pieces), its workspace kept here."""
        if pieces > 1:
            need = lkv.chunk_scan_sp_workspace(self.layer, self.w.n_req, pieces)
            ws = getattr(self, "_sp_ws", None)
            if ws is None or ws.numel() < need:
                self._sp_ws = ws = torch.empty(need, dtype=torch.uint8, device=self.out.device)
            lkv.chunk_scan_sp(self.layer, self.online.struct, self.w.scale, S_init, self.out, self.S_final, pieces,
                              ws, stream)
            return
        if self.w.layer.family == I.GDN:
            lkv.gdn_chunk_scan(self.layer, self.online.struct, self.w.scale, S_init, self.out, self.S_final,
                               stream)
        else:
            lkv.ssd_chunk_scan(self.layer, self.online.struct, S_init, self.out, self.S_final, stream)


class GpuStep:
    """One token per request for a decode step: rows ``idx`` of a token stream,
    gathered on the host and copied to HBM."""

    def __init__(self, tok: I.Tokens, idx: np.ndarray, layer: I.Layer, A: Optional[np.ndarray],
                 scale: float = 1.0, device="cuda"):
        io = _TORCH[layer.io_dtype]
        gate = _TORCH[layer.gate_dtype] if layer.family == I.GDN else torch.float32
        self.family = layer.family
        self.layer = layer_struct(layer)
        self.n_req = int(len(idx))
        self.scale = scale
        self.q = _t(tok.q[idx], io, device)
        self.k = _t(tok.k[idx], io, device)
        self.v = _t(tok.v[idx], io, device)
        self.g = _t(tok.g[idx], gate, device)
        self.beta = _t(tok.beta[idx], gate, device) if tok.beta is not None else None
        self.A = _t(A, torch.float32, device) if layer.family == I.SSD else None
        self.out = torch.empty((self.n_req, layer.h_v, layer.dv), device=device, dtype=io)

    def decode(self, S: torch.Tensor, with_out: bool = True, stream=None):
        """Advance ``S`` [n_req,h_v,dv,dk] by this step in place; the outputs land in ``out``."""
        o = self.out if with_out else None
        if self.family == I.GDN:
            lkv.gdn_decode(self.layer, self.q, self.k, self.v, self.g, self.beta, self.scale, S, o, stream)
        else:
            lkv.ssd_decode(self.layer, self.q, self.k, self.v, self.g, self.A, S, o, stream)


class GpuSelection:
    """The recompute's online stream, gathered on the GPU from a context stream at
    the selected positions (``sel_cu``, ``pos``); ``struct`` is that stream for
    the chunk scan.  ``q`` of the context may be given separately (``ctx_q``)."""

    def __init__(self, ctx: GpuTokens, ctx_cu: np.ndarray, sel_cu: np.ndarray, pos: np.ndarray,
                 layer: I.Layer, ctx_q: Optional[torch.Tensor] = None, device="cuda"):
        self.layer = layer_struct(layer)
        self.ctx_cu = _t(ctx_cu, torch.int32, device)
        cq = ctx.q if ctx_q is None else ctx_q
        self.ctx_struct = lkv.make_tokens(self.ctx_cu, ctx.n_tok, cq, ctx.k, ctx.v, ctx.g, ctx.beta, ctx.A)
        self.sel_cu = _t(sel_cu, torch.int32, device)
        self.pos = _t(pos, torch.int32, device)
        self.n_sel = int(sel_cu[-1])

        def like(x):
            return None if x is None else torch.empty((self.n_sel,) + tuple(x.shape[1:]), device=device,
                                                      dtype=x.dtype)
        self.q, self.k, self.v, self.g, self.beta = (like(x) for x in (cq, ctx.k, ctx.v, ctx.g, ctx.beta))
        self.struct = lkv.make_tokens(self.sel_cu, self.n_sel, self.q, self.k, self.v, self.g, self.beta,
                                      ctx.A)

    def gather(self, stream=None):
        lkv.gather_selected(self.layer, self.ctx_struct, self.pos, self.sel_cu, self.n_sel, self.q, self.k,
                            self.v, self.g, self.beta, stream)


def compact_rows(blk_ids: np.ndarray):
    """The distinct pool rows a batch reads (ascending) and its block ids remapped
    onto them: ``rows[remapped[i]] == blk_ids[i]``."""
    rows, remapped = np.unique(np.asarray(blk_ids, np.int64), return_inverse=True)
    return rows.astype(np.int32), remapped.astype(np.int32)


class HostCache:
    """The cache as the paper keeps it: per-block end states in bf16 and, for exact
    composition, the cached blocks' key/gate streams (Mamba-2: dt only), in
    pinned host memory."""

    def __init__(self, w: I.Workload, B_bf16: np.ndarray):
        L = w.layer
        io = _TORCH[L.io_dtype]
        gate = _TORCH[L.gate_dtype] if L.family == I.GDN else torch.float32

        def pinned(x, dtype):
            t = torch.empty(x.shape, dtype=dtype, pin_memory=True)
            t.copy_(torch.from_numpy(np.ascontiguousarray(x)))
            return t
        self.w = w
        self.B = pinned(B_bf16, torch.bfloat16)          # [n_blk,h_v,dv,dk]
        c = w.cached
        self.cu = c.cu.astype(np.int64)
        # Gated DeltaNet transitions need the keys and both gates; Mamba-2's only dt
        self.k = pinned(c.k, io) if L.family == I.GDN else None
        self.g = pinned(c.g, gate)
        self.beta = pinned(c.beta, gate) if c.beta is not None else None


class StagedBatch:
    """A batch's cache rows moved into HBM by ``lkv_stage_rows`` on ``stream``:
    the single-block rows (one per request) and, for exact composition, the
    distinct blocks' states plus their key/gate token streams, compacted."""

    def __init__(self, hc: HostCache, blk_ids: np.ndarray, blk_cu: np.ndarray, last_blk: np.ndarray,
                 exact: bool = True, device="cuda"):
        self.hc = hc
        L = hc.w.layer
        self.layer = layer_struct(L)
        self.n_req = len(blk_cu) - 1
        st = (L.h_v, L.dv, L.dk)
        self.single_rows = np.asarray(last_blk, np.int32)
        assert (self.single_rows >= 0).all()
        self.B_single = torch.empty((self.n_req,) + st, device=device, dtype=torch.bfloat16)
        self.single_src = torch.arange(self.n_req, dtype=torch.int32, device=device)
        self.exact = exact
        if exact:
            self.rows, remapped = compact_rows(blk_ids)
            self.blk_ids = torch.from_numpy(remapped).to(device)
            self.blk_cu = torch.from_numpy(np.asarray(blk_cu, np.int32)).to(device)
            self.n_ids = int(len(remapped))
            self.B_exact = torch.empty((len(self.rows),) + st, device=device, dtype=torch.bfloat16)
            lens = hc.cu[self.rows + 1] - hc.cu[self.rows]
            self.tok_rows = (np.concatenate([np.arange(hc.cu[b], hc.cu[b + 1]) for b in self.rows])
                             if len(self.rows) else np.zeros(0)).astype(np.int32)
            cu = np.zeros(len(self.rows) + 1, np.int32)
            cu[1:] = np.cumsum(lens)
            self.cu = torch.from_numpy(cu).to(device)
            n = int(cu[-1])
            self.k = (torch.empty((n,) + tuple(hc.k.shape[1:]), device=device, dtype=hc.k.dtype)
                      if hc.k is not None else None)
            self.g = torch.empty((n,) + tuple(hc.g.shape[1:]), device=device, dtype=hc.g.dtype)
            self.beta = (torch.empty((n,) + tuple(hc.beta.shape[1:]), device=device, dtype=hc.beta.dtype)
                         if hc.beta is not None else None)
            self.blocks = lkv.make_tokens(self.cu, n, None, self.k, None, self.g, self.beta,
                                          _t(hc.w.A, torch.float32, device) if L.family == I.SSD else None)
            f32 = dict(device=device, dtype=torch.float32)
            self.M = (torch.empty((len(self.rows), L.h_v, L.dk, L.dk), **f32) if L.family == I.GDN
                      else torch.empty((len(self.rows), L.h_v), **f32))

    def stage_single(self, stream=None):
        lkv.stage_rows(self.B_single, self.hc.B, self.single_rows, stream)

    def stage_exact(self, stream=None):
        lkv.stage_rows(self.B_exact, self.hc.B, self.rows, stream)
        if self.k is not None:
            lkv.stage_rows(self.k, self.hc.k, self.tok_rows, stream)
        lkv.stage_rows(self.g, self.hc.g, self.tok_rows, stream)
        if self.beta is not None:
            lkv.stage_rows(self.beta, self.hc.beta, self.tok_rows, stream)

    def staged_bytes(self, exact: bool) -> int:
        if not exact:
            return self.B_single.numel() * 2
        return sum(t.numel() * t.element_size() for t in (self.B_exact, self.k, self.g, self.beta)
                   if t is not None)

    def init_single(self, S, stream=None):
        lkv.init_single_bf16(self.layer, self.n_req, self.B_single, self.single_src, S, stream)

    def init_compose(self, S, stream=None):
        """Fold the staged blocks' transitions from their key/gate streams, then compose."""
        lkv.block_summary(self.layer, self.blocks, None, self.M, stream)
        lkv.init_compose_bf16(self.layer, len(self.rows), self.B_exact, self.M, self.blk_ids, self.blk_cu,
                              self.n_ids, S, stream)
