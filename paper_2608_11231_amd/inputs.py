"""Seeded synthetic workloads for one recurrent layer's online prefill.

This module draws random inputs and nothing else: it holds no part of the
recurrence, the block summaries or the composition. Both the CPU oracle and the
GPU library consume what it returns, so it is the only code they share.

Every floating-point field is a float32 numpy array whose entries are exactly
representable in the layer's storage dtype (bf16 fields are rounded from fp64
to fp32 and then to bf16, each step round-to-nearest-even), so widening to
fp64 on the oracle side and narrowing to bf16 on the GPU side are both exact.

Token streams are packed "THD": ``[n_tok, heads, dim]`` over consecutive
segments, with ``cu`` the int32 segment offsets (``cu[0] = 0``).

Workload shapes follow the paper's hybrid-model setting (Sec. 2 and Sec. 4:
8K-32K contexts reused as cached chunks, a recompute fraction r of about 0.2 of
the context replayed online) with gate laws taken from the Gated DeltaNet and
Mamba-2 parameterisations (alpha = exp(g), Eq. 3; per-head scalar decay, Eq. 2).
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Sequence

import numpy as np

GDN = 0
SSD = 1

_KIND_CACHED = 1
_KIND_ONLINE = 2
_KIND_LAYER = 3
_KIND_LENGTHS = 4


# --------------------------------------------------------------------------
# rounding helpers (storage formats only)
# --------------------------------------------------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bf16 (fp64 -> fp32 -> bf16, nearest-even), returned widened to fp32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    r = ((u + bias) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def _softplus(x: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, x)


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def _unit_rows(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.float64)
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    return x / np.maximum(n, 1e-30)


# --------------------------------------------------------------------------
# containers
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Layer:
    """Geometry of one recurrent layer.

    GDN: ``h_qk`` q/k heads, ``h_v`` value heads (one state each), key dim ``dk``,
    value dim ``dv``.  SSD: ``h_qk`` = number of B/C groups G, ``h_v`` = heads H,
    ``dk`` = state dim N, ``dv`` = head dim P.
    """
    family: int
    h_qk: int
    h_v: int
    dk: int
    dv: int
    chunk: int
    io_dtype: str = "bf16"      # q/k/v (C/B/x) and o (y)
    gate_dtype: str = "bf16"    # GDN g=log(alpha) and beta; SSD dt is always f32

    @property
    def state_elems(self) -> int:
        return self.h_v * self.dv * self.dk


@dataclasses.dataclass
class Tokens:
    """One packed token stream over ``n_seq`` segments.

    GDN: q, k [n_tok, h_qk, dk]; v [n_tok, h_v, dv]; g = log(alpha) and beta
    [n_tok, h_v].  SSD: q = C and k = B [n_tok, G, N]; v = x [n_tok, H, P];
    g = dt [n_tok, H] (after softplus, > 0); beta is None.
    """
    cu: np.ndarray
    q: Optional[np.ndarray]
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: Optional[np.ndarray]

    @property
    def n_seq(self) -> int:
        return int(self.cu.shape[0] - 1)

    @property
    def n_tok(self) -> int:
        return int(self.cu[-1])

    @property
    def max_len(self) -> int:
        return int(np.max(np.diff(self.cu))) if self.n_seq > 0 else 0

    def lengths(self) -> np.ndarray:
        return np.diff(self.cu)


@dataclasses.dataclass
class Workload:
    """A batch of requests: cached blocks (in context order) plus online tokens.

    ``blk_cu[r]:blk_cu[r+1]`` are request r's positions in ``blk_ids``; ``blk_ids``
    names rows of the block pool (segments of ``cached``).  ``last_blk[r]`` is the
    pool row of request r's last matched block (-1 when it has none).
    """
    name: str
    layer: Layer
    cached: Tokens
    online: Tokens
    blk_cu: np.ndarray
    blk_ids: np.ndarray
    last_blk: np.ndarray
    A: Optional[np.ndarray] = None   # SSD per-head A < 0, [H] f32
    scale: float = 1.0

    @property
    def n_req(self) -> int:
        return int(self.blk_cu.shape[0] - 1)

    @property
    def n_blk(self) -> int:
        return self.cached.n_seq


# --------------------------------------------------------------------------
# generation
# --------------------------------------------------------------------------

@dataclasses.dataclass
class GateLaw:
    """Distribution of the per-token gates.

    GDN: either ``alpha_uniform=(lo, hi)`` with g = log(alpha), or
    g = -softplus(N(x_mu, 1)); beta ~ U(0,1) when ``beta_uniform`` else
    sigmoid(N(beta_mu, 1)).  SSD: dt = softplus(N(dt_mu, 1) + dt_bias) and
    A_h = -exp(U(log a_lo, log a_hi)).
    """
    alpha_uniform: Optional[tuple] = None
    x_mu: float = -4.0
    beta_uniform: bool = False
    beta_mu: float = 0.0
    dt_mu: float = -3.0
    dt_bias: float = 0.0
    a_lo: float = 1.0
    a_hi: float = 16.0


def _rng(seed: int, *path: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *path])))


def _segment(layer: Layer, law: GateLaw, L: int, want_q: bool, rng: np.random.Generator):
    f32 = np.float32
    hq, hv, dk, dv = layer.h_qk, layer.h_v, layer.dk, layer.dv
    io = layer.io_dtype
    k = to_storage(_unit_rows(rng.standard_normal((L, hq, dk), dtype=f32)), io)
    q = to_storage(_unit_rows(rng.standard_normal((L, hq, dk), dtype=f32)), io) if want_q else None
    if layer.family == GDN:
        v = to_storage(rng.standard_normal((L, hv, dv), dtype=f32), io)
        if law.alpha_uniform is not None:
            lo, hi = law.alpha_uniform
            g = np.log(rng.uniform(lo, hi, size=(L, hv)))
        else:
            g = -_softplus(rng.standard_normal((L, hv)) + law.x_mu)
        if law.beta_uniform:
            beta = rng.uniform(0.0, 1.0, size=(L, hv))
        else:
            beta = _sigmoid(rng.standard_normal((L, hv)) + law.beta_mu)
        return q, k, v, to_storage(g, layer.gate_dtype), to_storage(beta, layer.gate_dtype)
    # SSD: q=C, k=B, v=x, g=dt
    x = to_storage(rng.standard_normal((L, hv, dv), dtype=f32), io)
    dt = _softplus(rng.standard_normal((L, hv)) + law.dt_mu + law.dt_bias)
    return q, k, x, to_storage(dt, "f32"), None


def _pack(layer: Layer, segs, lens: Sequence[int], want_q: bool) -> Tokens:
    cu = np.zeros(len(lens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(lens, dtype=np.int64))
    n = int(cu[-1])
    hq, hv, dk, dv = layer.h_qk, layer.h_v, layer.dk, layer.dv

    def cat(idx, shape):
        parts = [s[idx] for s in segs]
        if parts and parts[0] is None:
            return None
        if not parts:
            return np.zeros(shape, dtype=np.float32)
        return np.ascontiguousarray(np.concatenate(parts, axis=0), dtype=np.float32)

    q = cat(0, (n, hq, dk)) if want_q else None
    k = cat(1, (n, hq, dk))
    v = cat(2, (n, hv, dv))
    g = cat(3, (n, hv))
    beta = cat(4, (n, hv)) if layer.family == GDN else None
    return Tokens(cu=cu, q=q, k=k, v=v, g=g, beta=beta)


def _gen_many(layer, law, seed, kind, lens, want_q, workers):
    def one(i):
        return _segment(layer, law, int(lens[i]), want_q, _rng(seed, kind, i))
    n = len(lens)
    if workers > 1 and n > 1 and int(np.sum(lens)) * layer.h_v * layer.dv > (1 << 22):
        with ThreadPoolExecutor(min(workers, n)) as ex:
            segs = list(ex.map(one, range(n)))
    else:
        segs = [one(i) for i in range(n)]
    return _pack(layer, segs, lens, want_q)


def build_workload(name: str, layer: Layer, block_lens: Sequence[Sequence[int]],
                   online_lens: Sequence[int], law: GateLaw, seed: int,
                   scale: float = 1.0, workers: int = 8) -> Workload:
    """Draw a workload: ``block_lens[r]`` lists request r's cached block lengths in
    context order; ``online_lens[r]`` is its number of online tokens."""
    assert len(block_lens) == len(online_lens)
    n_req = len(online_lens)
    flat = [int(L) for lens in block_lens for L in lens]
    blk_cu = np.zeros(n_req + 1, dtype=np.int32)
    blk_cu[1:] = np.cumsum([len(b) for b in block_lens])
    blk_ids = np.arange(len(flat), dtype=np.int32)
    last = np.array([blk_cu[r + 1] - 1 if blk_cu[r + 1] > blk_cu[r] else -1
                     for r in range(n_req)], dtype=np.int32)
    cached = _gen_many(layer, law, seed, _KIND_CACHED, flat, False, workers)
    online = _gen_many(layer, law, seed, _KIND_ONLINE, list(online_lens), True, workers)
    A = None
    if layer.family == SSD:
        r = _rng(seed, _KIND_LAYER)
        A = to_storage(-np.exp(r.uniform(np.log(law.a_lo), np.log(law.a_hi), size=layer.h_v)), "f32")
    return Workload(name=name, layer=layer, cached=cached, online=online, blk_cu=blk_cu,
                    blk_ids=blk_ids, last_blk=last, A=A, scale=scale)


# --------------------------------------------------------------------------
# ragged length recipes
# --------------------------------------------------------------------------

def lengths_fixed_sum(rng: np.random.Generator, n: int, lo: int, hi: int, total: int) -> List[int]:
    """n iid draws from U{lo..hi}, then +-1 nudges on random entries (kept within
    [lo, hi]) until they sum to ``total``."""
    assert n * lo <= total <= n * hi
    x = rng.integers(lo, hi + 1, size=n).astype(np.int64)
    while x.sum() != total:
        i = int(rng.integers(0, n))
        if x.sum() < total and x[i] < hi:
            x[i] += 1
        elif x.sum() > total and x[i] > lo:
            x[i] -= 1
    return [int(v) for v in x]


def lengths_capped(rng: np.random.Generator, k: int, lo: int, hi: int, cap: int) -> List[int]:
    """k sequential draws from U{lo..min(hi, remaining - lo*blocks_left)}, total <= cap."""
    out, rem = [], cap
    for j in range(k):
        left = k - j - 1
        top = min(hi, rem - lo * left)
        L = int(rng.integers(lo, top + 1))
        out.append(L)
        rem -= L
    return out


# --------------------------------------------------------------------------
# synthetic selectors (which context positions the recompute replays)
# --------------------------------------------------------------------------

def select_uniform(rng: np.random.Generator, n_ctx: int, r: float) -> np.ndarray:
    """A recompute budget r: round(r * n_ctx) distinct positions drawn uniformly,
    ascending (context order)."""
    m = int(round(r * n_ctx))
    return np.sort(rng.choice(n_ctx, size=m, replace=False)).astype(np.int32)


def select_seams(block_lens: Sequence[int], window: int) -> np.ndarray:
    """Seam selection: a window of ``window`` positions around every boundary between
    consecutive cached blocks (window // 2 before it, the rest after), merged and
    ascending."""
    ends = np.cumsum(np.asarray(block_lens, np.int64))
    n_ctx = int(ends[-1]) if len(ends) else 0
    keep = np.zeros(n_ctx, bool)
    for b in ends[:-1]:
        keep[max(0, b - window // 2):min(n_ctx, b + window - window // 2)] = True
    return np.nonzero(keep)[0].astype(np.int32)


def pack_selection(per_request: Sequence[np.ndarray]):
    """(sel_cu, pos) of per-request position lists."""
    cu = np.zeros(len(per_request) + 1, np.int32)
    cu[1:] = np.cumsum([len(p) for p in per_request])
    pos = (np.concatenate([np.asarray(p, np.int32) for p in per_request])
           if per_request else np.zeros(0, np.int32))
    return cu, pos.astype(np.int32)


def context_cu(w: "Workload") -> np.ndarray:
    """Offsets of each request's context in the cached stream (its blocks are
    consecutive segments there, in context order)."""
    assert np.array_equal(w.blk_ids, np.arange(w.n_blk, dtype=np.int32))
    return w.cached.cu[w.blk_cu].astype(np.int32)


def random_block_src(rng: np.random.Generator, w: "Workload") -> np.ndarray:
    """One uniformly drawn matched block per request (the random-block
    single-source variant), as pool rows; -1 for a request with no blocks."""
    src = np.full(w.n_req, -1, np.int32)
    for r in range(w.n_req):
        k0, k1 = int(w.blk_cu[r]), int(w.blk_cu[r + 1])
        if k1 > k0:
            src[r] = w.blk_ids[int(rng.integers(k0, k1))]
    return src


# --------------------------------------------------------------------------
# the five reference workloads
# --------------------------------------------------------------------------

CONFIG_NAMES = (
    "gdn_tiny_f32",          # 1 head, dk=dv=16, 2x64 cached + 32 online, C=16
    "gdn_8k",                # 32 heads, d=128, K=8x1024, T=1536
    "ssd_8k",                # 64 heads, P=64, N=128, G=1, K=8x1024, T=1536
    "gdn_32k",               # 4 requests, K=32 ragged blocks summing to 32768, T=4096
    "gdn_16k_ragged_grouped",  # 16 requests, 16 qk / 32 v heads, ragged K and T
)

BASE_SEED = 20260


def config(index: int, seed: Optional[int] = None, mild: bool = False,
           workers: int = 8) -> Workload:
    """The reference workloads by index (see ``CONFIG_NAMES``).

    ``mild=True`` draws slower-decaying gates (GDN: x ~ N(-9,1), beta =
    sigmoid(N(-4,1)); SSD: dt bias -6) so that every cached block contributes a
    visible share of the composed state; used for parity only.
    """
    s = BASE_SEED + index if seed is None else seed
    name = CONFIG_NAMES[index] + ("_mild" if mild else "")
    lr = _rng(s, _KIND_LENGTHS)
    if index == 0:
        layer = Layer(GDN, 1, 1, 16, 16, 16, "f32", "f32")
        law = GateLaw(alpha_uniform=(0.90, 1.0), beta_uniform=True)
        return build_workload(name, layer, [[64, 64]], [32], law, s, workers=workers)
    if index == 1:
        layer = Layer(GDN, 32, 32, 128, 128, 64)
        law = GateLaw(x_mu=-9.0, beta_mu=-4.0) if mild else GateLaw()
        return build_workload(name, layer, [[1024] * 8], [1536], law, s, workers=workers)
    if index == 2:
        layer = Layer(SSD, 1, 64, 128, 64, 64, "bf16", "f32")
        law = GateLaw(dt_bias=-6.0) if mild else GateLaw()
        return build_workload(name, layer, [[1024] * 8], [1536], law, s, workers=workers)
    if index == 3:
        layer = Layer(GDN, 32, 32, 128, 128, 64)
        law = GateLaw(x_mu=-9.0, beta_mu=-4.0) if mild else GateLaw()
        blocks = [lengths_fixed_sum(lr, 32, 512, 2048, 32768) for _ in range(4)]
        return build_workload(name, layer, blocks, [4096] * 4, law, s, workers=workers)
    if index == 4:
        layer = Layer(GDN, 16, 32, 128, 128, 64)
        law = GateLaw(x_mu=-9.0, beta_mu=-4.0) if mild else GateLaw()
        blocks, online = [], []
        for _ in range(16):
            k = int(lr.integers(2, 17))
            blocks.append(lengths_capped(lr, k, 256, 4096, 16384))
            online.append(int(lr.integers(512, 3073)))
        return build_workload(name, layer, blocks, online, law, s, workers=workers)
    raise IndexError(index)


def small(family: int, *, n_req: int = 2, h_qk: int = 2, h_v: int = 2, dk: int = 32,
          dv: int = 32, chunk: int = 16, blocks=((40, 23), (17,)), online=(37, 70),
          io: str = "bf16", gate: str = "bf16", mild: bool = True, seed: int = 7,
          scale: float = 1.0) -> Workload:
    """A small ragged workload for parity tests (several chunks plus tails)."""
    layer = Layer(family, h_qk, h_v, dk, dv, chunk, io, gate if family == GDN else "f32")
    if family == GDN:
        law = GateLaw(x_mu=-3.0, beta_mu=0.0) if mild else GateLaw()
    else:
        law = GateLaw(dt_mu=-3.0, dt_bias=-2.0 if mild else 0.0)
    blocks = [list(b) for b in blocks][:n_req]
    online = list(online)[:n_req]
    return build_workload(f"small_{family}", layer, blocks, online, law, seed, scale=scale)
