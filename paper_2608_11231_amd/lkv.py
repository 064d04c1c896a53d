"""Thin Python binding of liblkv.so (include/lkv.h).

Argument marshalling only: every function takes torch tensors that already
live on the GPU, passes their device pointers and the current torch stream to
the C ABI, and raises ``LkvError`` on a non-zero status.  All computation
happens in the library's HIP kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblkv.so")

GDN, SSD = 0, 1
F32, BF16 = 0, 1

_STATUS = {0: "LKV_OK", 1: "LKV_E_NULL", 2: "LKV_E_SHAPE", 3: "LKV_E_DTYPE", 4: "LKV_E_ALIGN",
           5: "LKV_E_UNSUPPORTED", 6: "LKV_E_WORKSPACE", 7: "LKV_E_HIP"}


class LkvError(RuntimeError):
    def __init__(self, status: int, call: str, hip: int = 0):
        self.status = status
        msg = f"{call}: {_STATUS.get(status, status)}"
        if status == 7:
            msg += f" (hipError {hip})"
        super().__init__(msg)


class Layer(ctypes.Structure):
    _fields_ = [("family", ctypes.c_int32), ("h_qk", ctypes.c_int32), ("h_v", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("gate_dtype", ctypes.c_int32)]


class Tokens(ctypes.Structure):
    _fields_ = [("cu", ctypes.c_void_p), ("n_seq", ctypes.c_int32), ("n_tok", ctypes.c_int64),
                ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("beta", ctypes.c_void_p), ("A", ctypes.c_void_p)]


_lib = None
_lock = threading.Lock()
EXPORTS = ("lkv_abi_version", "lkv_status_string", "lkv_last_hip_error", "lkv_block_summary",
           "lkv_init_single", "lkv_init_compose", "lkv_gdn_chunk_scan", "lkv_ssd_chunk_scan",
           "lkv_gdn_decode", "lkv_ssd_decode", "lkv_gather_selected", "lkv_init_single_bf16",
           "lkv_init_compose_bf16", "lkv_round_bf16", "lkv_stage_rows", "lkv_state_rel_error",
           "lkv_chunk_scan_from_pool", "lkv_set_wait_limit", "lkv_chunk_scan_sp_workspace",
           "lkv_chunk_scan_sp", "lkv_chunk_scan_sp_noalloc")


def load() -> ctypes.CDLL:
    """Load liblkv.so; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                                   "`python -m paper_2608_11231_amd.build` (hipcc, gfx950)")
            lib = ctypes.CDLL(LIB_PATH)
            vp, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
            LP, TP = ctypes.POINTER(Layer), ctypes.POINTER(Tokens)
            lib.lkv_abi_version.restype = ctypes.c_int
            lib.lkv_status_string.restype = ctypes.c_char_p
            lib.lkv_status_string.argtypes = [ctypes.c_int]
            lib.lkv_last_hip_error.restype = ctypes.c_int
            lib.lkv_set_wait_limit.argtypes = [i32]
            lib.lkv_chunk_scan_sp_workspace.argtypes = [LP, i32, i32, ctypes.POINTER(ctypes.c_size_t)]
            lib.lkv_chunk_scan_sp.argtypes = [LP, TP, f32, vp, vp, vp, i32, vp, ctypes.c_size_t, vp]
            lib.lkv_chunk_scan_sp_noalloc.argtypes = [LP, TP, f32, vp, vp, vp, i32, vp]
            lib.lkv_set_wait_limit.restype = i32
            lib.lkv_block_summary.argtypes = [LP, TP, vp, vp, vp]
            lib.lkv_init_single.argtypes = [LP, i32, i32, vp, vp, vp, vp]
            lib.lkv_init_compose.argtypes = [LP, i32, i32, vp, vp, vp, vp, i32, vp, vp]
            lib.lkv_gdn_chunk_scan.argtypes = [LP, TP, f32, vp, vp, vp, vp]
            lib.lkv_ssd_chunk_scan.argtypes = [LP, TP, vp, vp, vp, vp]
            lib.lkv_gdn_decode.argtypes = [LP, i32, vp, vp, vp, vp, vp, f32, vp, vp, vp]
            lib.lkv_ssd_decode.argtypes = [LP, i32, vp, vp, vp, vp, vp, vp, vp, vp]
            lib.lkv_gather_selected.argtypes = [LP, TP, vp, vp, ctypes.c_int64, vp, vp, vp, vp, vp, vp]
            lib.lkv_init_single_bf16.argtypes = [LP, i32, i32, vp, vp, vp, vp]
            lib.lkv_init_compose_bf16.argtypes = [LP, i32, i32, vp, vp, vp, vp, i32, vp, vp]
            lib.lkv_round_bf16.argtypes = [vp, vp, ctypes.c_int64, vp]
            lib.lkv_stage_rows.argtypes = [vp, vp, vp, i32, ctypes.c_int64, vp]
            lib.lkv_state_rel_error.argtypes = [vp, vp, i32, ctypes.c_int64, i32, vp, vp, vp, vp]
            lib.lkv_chunk_scan_from_pool.argtypes = [LP, TP, f32, vp, i32, i32, vp, vp, vp, vp]
            for f in ("lkv_block_summary", "lkv_init_single", "lkv_init_compose", "lkv_gdn_chunk_scan",
                      "lkv_ssd_chunk_scan", "lkv_gdn_decode", "lkv_ssd_decode", "lkv_gather_selected",
                      "lkv_init_single_bf16", "lkv_init_compose_bf16", "lkv_round_bf16", "lkv_stage_rows",
                      "lkv_state_rel_error", "lkv_chunk_scan_from_pool"):
                getattr(lib, f).restype = ctypes.c_int
            _lib = lib
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if t.device.type != "cuda":
        raise ValueError("lkv tensors must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("lkv tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(st: int, call: str):
    if st != 0:
        raise LkvError(st, call, load().lkv_last_hip_error())


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return F32
    if dt == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported dtype {dt}")


def make_layer(family: int, h_qk: int, h_v: int, dk: int, dv: int, chunk: int,
               io_dtype: torch.dtype = torch.bfloat16, gate_dtype: torch.dtype = torch.bfloat16) -> Layer:
    return Layer(family, h_qk, h_v, dk, dv, chunk, dtype_code(io_dtype), dtype_code(gate_dtype))


def make_tokens(cu: torch.Tensor, n_tok: int, q=None, k=None, v=None, g=None, beta=None, A=None) -> Tokens:
    """``cu`` int32 [n_seq+1] on the GPU; ``n_tok`` its last entry (host value)."""
    t = Tokens()
    t.cu = _ptr(cu)
    t.n_seq = int(cu.shape[0]) - 1
    t.n_tok = int(n_tok)
    t.q, t.k, t.v, t.g, t.beta, t.A = (_ptr(x) for x in (q, k, v, g, beta, A))
    t._keep = (cu, q, k, v, g, beta, A)  # keep tensors alive while the struct is in use
    return t


def block_summary(layer: Layer, blocks: Tokens, B_out: Optional[torch.Tensor],
                  M_out: Optional[torch.Tensor], stream=None) -> None:
    _check(load().lkv_block_summary(ctypes.byref(layer), ctypes.byref(blocks), _ptr(B_out), _ptr(M_out),
                                    _stream(stream)), "lkv_block_summary")


def init_single(layer: Layer, n_blk: int, B_pool: torch.Tensor, src_blk: torch.Tensor,
                S_init: torch.Tensor, stream=None) -> None:
    _check(load().lkv_init_single(ctypes.byref(layer), int(src_blk.shape[0]), int(n_blk), _ptr(B_pool),
                                  _ptr(src_blk), _ptr(S_init), _stream(stream)), "lkv_init_single")


def init_compose(layer: Layer, n_blk: int, B_pool: torch.Tensor, M_pool: torch.Tensor,
                 blk_ids: torch.Tensor, blk_cu: torch.Tensor, n_ids: int, S_init: torch.Tensor,
                 stream=None) -> None:
    _check(load().lkv_init_compose(ctypes.byref(layer), int(blk_cu.shape[0]) - 1, int(n_blk), _ptr(B_pool),
                                   _ptr(M_pool), _ptr(blk_ids), _ptr(blk_cu), int(n_ids), _ptr(S_init),
                                   _stream(stream)), "lkv_init_compose")


def gdn_chunk_scan(layer: Layer, online: Tokens, scale: float, S_init: Optional[torch.Tensor],
                   o: Optional[torch.Tensor], S_final: Optional[torch.Tensor], stream=None) -> None:
    _check(load().lkv_gdn_chunk_scan(ctypes.byref(layer), ctypes.byref(online), float(scale), _ptr(S_init),
                                     _ptr(o), _ptr(S_final), _stream(stream)), "lkv_gdn_chunk_scan")


def ssd_chunk_scan(layer: Layer, online: Tokens, S_init: Optional[torch.Tensor], y: Optional[torch.Tensor],
                   S_final: Optional[torch.Tensor], stream=None) -> None:
    _check(load().lkv_ssd_chunk_scan(ctypes.byref(layer), ctypes.byref(online), _ptr(S_init), _ptr(y),
                                     _ptr(S_final), _stream(stream)), "lkv_ssd_chunk_scan")


def gdn_decode(layer: Layer, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
               beta: torch.Tensor, scale: float, S: torch.Tensor, o: Optional[torch.Tensor], stream=None) -> None:
    """One decode step for every request (``q.shape[0]`` requests); ``S`` is updated in place."""
    _check(load().lkv_gdn_decode(ctypes.byref(layer), int(q.shape[0]), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                                 _ptr(beta), float(scale), _ptr(S), _ptr(o), _stream(stream)), "lkv_gdn_decode")


def ssd_decode(layer: Layer, C: torch.Tensor, B: torch.Tensor, x: torch.Tensor, dt: torch.Tensor,
               A: torch.Tensor, S: torch.Tensor, y: Optional[torch.Tensor], stream=None) -> None:
    """One Mamba-2 decode step for every request; ``S`` is updated in place."""
    _check(load().lkv_ssd_decode(ctypes.byref(layer), int(C.shape[0]), _ptr(C), _ptr(B), _ptr(x), _ptr(dt),
                                 _ptr(A), _ptr(S), _ptr(y), _stream(stream)), "lkv_ssd_decode")


def gather_selected(layer: Layer, ctx: Tokens, pos: torch.Tensor, sel_cu: torch.Tensor, n_sel: int,
                    q: Optional[torch.Tensor], k: Optional[torch.Tensor], v: Optional[torch.Tensor],
                    g: Optional[torch.Tensor], beta: Optional[torch.Tensor], stream=None) -> None:
    """Copy the context rows at the selected positions into q/k/v/g/beta (any may be None)."""
    _check(load().lkv_gather_selected(ctypes.byref(layer), ctypes.byref(ctx), _ptr(pos), _ptr(sel_cu),
                                      int(n_sel), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                      _stream(stream)), "lkv_gather_selected")


def init_single_bf16(layer: Layer, n_blk: int, B_pool: torch.Tensor, src_blk: torch.Tensor, S_init: torch.Tensor,
                     stream=None) -> None:
    """Single-block initial state from a bf16 pool (exact widening)."""
    assert B_pool.dtype == torch.bfloat16
    _check(load().lkv_init_single_bf16(ctypes.byref(layer), int(src_blk.shape[0]), int(n_blk), _ptr(B_pool),
                                       _ptr(src_blk), _ptr(S_init), _stream(stream)), "lkv_init_single_bf16")


def init_compose_bf16(layer: Layer, n_blk: int, B_pool: torch.Tensor, M_pool: torch.Tensor, blk_ids: torch.Tensor,
                      blk_cu: torch.Tensor, n_ids: int, S_init: torch.Tensor, stream=None) -> None:
    """Exact composition from a bf16 B pool and an fp32 M (Lambda) pool."""
    assert B_pool.dtype == torch.bfloat16
    _check(load().lkv_init_compose_bf16(ctypes.byref(layer), int(blk_cu.shape[0]) - 1, int(n_blk), _ptr(B_pool),
                                        _ptr(M_pool), _ptr(blk_ids), _ptr(blk_cu), int(n_ids), _ptr(S_init),
                                        _stream(stream)), "lkv_init_compose_bf16")


def round_bf16(src: torch.Tensor, dst: torch.Tensor, stream=None) -> None:
    """dst (bf16) <- src (fp32) rounded to nearest even, elementwise."""
    assert src.dtype == torch.float32 and dst.dtype == torch.bfloat16 and src.numel() == dst.numel()
    _check(load().lkv_round_bf16(_ptr(src), _ptr(dst), int(src.numel()), _stream(stream)), "lkv_round_bf16")


def stage_rows(dst: torch.Tensor, src: torch.Tensor, rows, stream=None) -> None:
    """dst[i] <- src[rows[i]] for a host (preferably pinned) ``src`` and device ``dst``;
    ``rows`` is a host int32 array."""
    import numpy as np
    r = np.ascontiguousarray(rows, dtype=np.int32)
    row_bytes = src[0].numel() * src.element_size() if src.shape[0] else 0
    assert dst.shape[0] >= len(r) and dst[0].numel() * dst.element_size() == row_bytes
    if len(r) and r.max() >= src.shape[0]:
        raise ValueError("row index beyond the source pool")
    if src.device.type != "cpu" or not src.is_contiguous():
        raise ValueError("stage_rows: the source pool must be a contiguous host tensor")
    _check(load().lkv_stage_rows(_ptr(dst), ctypes.c_void_p(src.data_ptr()), r.ctypes.data_as(ctypes.c_void_p),
                                 len(r), int(row_bytes), _stream(stream)), "lkv_stage_rows")


def state_rel_error(S: torch.Tensor, S_ref: torch.Tensor, slice_dims: int = 2, group: int = 0, stream=None):
    """Per-slice (the trailing ``slice_dims`` dims) and, with ``group`` > 0, per-group
    relative Frobenius error of ``S`` against ``S_ref``.  Returns device fp64 tensors
    (sq [n,2], rel [n], rel_group [n/group] or None)."""
    assert S.shape == S_ref.shape and S.dtype == torch.float32 == S_ref.dtype
    elems = 1
    for d in S.shape[S.dim() - slice_dims:]:
        elems *= int(d)
    n = S.numel() // max(elems, 1)
    sq = torch.empty((n, 2), dtype=torch.float64, device=S.device)
    rel = torch.empty((n,), dtype=torch.float64, device=S.device)
    rg = torch.empty((n // group,), dtype=torch.float64, device=S.device) if group > 0 else None
    _check(load().lkv_state_rel_error(_ptr(S), _ptr(S_ref), int(n), int(elems), int(group), _ptr(sq), _ptr(rel),
                                      _ptr(rg), _stream(stream)), "lkv_state_rel_error")
    return sq, rel, rg


def chunk_scan_from_pool(layer: Layer, online: Tokens, scale: float, B_pool: Optional[torch.Tensor], n_blk: int,
                         src_blk: torch.Tensor, out: Optional[torch.Tensor], S_final: Optional[torch.Tensor],
                         stream=None) -> None:
    """The chunk scan starting each request from its cached pool row B_pool[src_blk[r]]."""
    dt = BF16 if (B_pool is not None and B_pool.dtype == torch.bfloat16) else F32
    _check(load().lkv_chunk_scan_from_pool(ctypes.byref(layer), ctypes.byref(online), float(scale), _ptr(B_pool), dt,
                                           int(n_blk), _ptr(src_blk), _ptr(out), _ptr(S_final), _stream(stream)),
           "lkv_chunk_scan_from_pool")


def set_wait_limit(polls: int) -> int:
    """Bound of the chunk kernels' stager-to-solver wait (polls; 0 = always give
    up, negative = the default).  A wait that gives up makes the results NaN.
    Returns the previous bound."""
    return int(load().lkv_set_wait_limit(int(polls)))


def chunk_scan_sp_workspace(layer: Layer, n_req: int, pieces: int) -> int:
    """Workspace bytes of chunk_scan_sp."""
    n = ctypes.c_size_t(0)
    _check(load().lkv_chunk_scan_sp_workspace(ctypes.byref(layer), int(n_req), int(pieces), ctypes.byref(n)),
           "lkv_chunk_scan_sp_workspace")
    return int(n.value)


def chunk_scan_sp(layer: Layer, online: Tokens, scale: float, S_init: Optional[torch.Tensor],
                  out: Optional[torch.Tensor], S_final: Optional[torch.Tensor], pieces: int, ws: torch.Tensor,
                  stream=None) -> None:
    """The chunk scan with each request's stream split into ``pieces`` pieces
    (sequence parallel); ``ws`` is a device workspace tensor."""
    _check(load().lkv_chunk_scan_sp(ctypes.byref(layer), ctypes.byref(online), float(scale), _ptr(S_init), _ptr(out),
                                    _ptr(S_final), int(pieces), _ptr(ws), int(ws.numel() * ws.element_size()),
                                    _stream(stream)), "lkv_chunk_scan_sp")


def chunk_scan_sp_noalloc(layer: Layer, online: Tokens, scale: float, S_init: Optional[torch.Tensor],
                          out: Optional[torch.Tensor], S_final: Optional[torch.Tensor], pieces: int,
                          stream=None) -> None:
    """chunk_scan_sp on the library's fixed per-GPU scratch (allocates nothing)."""
    _check(load().lkv_chunk_scan_sp_noalloc(ctypes.byref(layer), ctypes.byref(online), float(scale), _ptr(S_init),
                                            _ptr(out), _ptr(S_final), int(pieces), _stream(stream)),
           "lkv_chunk_scan_sp_noalloc")
