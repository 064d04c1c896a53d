#!/usr/bin/env python3
"""Benchmark of one recurrent layer's online prefill on one MI355X.

One step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM:
  1. lkv_init_single   -- LinearKV's single-block initial state (last block),
  2. lkv_block_summary -- online fold of the cached blocks' transitions M_k that
                          the composition reads (blocks 2..K of each request;
                          the exact-composition mode's extra work),
  3. lkv_init_compose  -- exact composition of the K cached (M_k, B_k) pairs,
  4. the chunk scan    -- Gated DeltaNet (or Mamba-2) recurrence over the online
                          tokens from the composed state, with outputs.
The per-block states B_k are the cache's content (computed offline in the
paper), so they are built once before timing.

Prints ONE JSON line.  ``value`` = online tokens / step time, the step time
being the median over the timed steps, each run cold: an untimed write of a
512 MiB buffer before every step evicts the 256 MB Infinity Cache (warm,
back-to-back figures are reported alongside).  Per-kernel durations come from
HIP events on the stream the library launches on, inside the timed steps;
``roofline`` is given for the kernel that takes the most time and
``roofline_by_kernel`` for all four, against the published peaks and against
the peaks measured in the same run (``measured_peaks``: a 512 MiB device copy
and a large bf16 matrix product).  ``other_workloads`` holds the same figures
for the 8K Gated DeltaNet, 8K Mamba-2 and ragged 16K workloads.  ``cpu_baseline`` times the CPU oracle
on a bounded sample of the same workload and scales it to the whole step.
``lb_fused_*`` times LinearKV's path as a single launch (the scan reading its
initial state straight from the cached pool row).  ``decode_step`` times, after
the step and outside it, the decode call that
follows the prefill (one token per request) on the workload's final states and
on a 256-request batch; ``gather_selected`` times the gather that forms the
online stream from the cached context at selected positions;
``bf16_pool_staging`` times the cache's bf16 storage path (pool rounding,
host-to-device staging of a batch's rows, overlap with the scan);
``relative_error_probe`` gives both initial states' relative error against the
full-prefix state, at the workload's gates and at slowly decaying gates (where
every cached block contributes), and times the diagnostic kernel.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
RIDGE = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def fold_dropped_blocks(w):
    from paper_2608_11231_amd.gpu_io import fold_dropped_blocks as f
    return f(w)


# ---------------------------------------------------------------- algorithmic work
def work_model(w):
    """Algorithmic bytes and flops per launch of each kernel of the step.

    Bytes count every tensor the call must touch exactly once (q/k per q/k head,
    v/g/beta per value head, outputs written once).  Flops are the chunkwise
    minimum (matrix products of the chunk form, the triangular solve as C^3/3);
    the extra bf16 hi/lo passes the kernels issue for fp32 accuracy are not
    counted.
    """
    L = w.layer
    io = 2 if L.io_dtype == "bf16" else 4
    gb = 2 if (L.gate_dtype == "bf16" and L.family == 0) else 4
    C, dk, dv, hq, hv = L.chunk, L.dk, L.dv, L.h_qk, L.h_v
    T = w.online.n_tok
    Tc = w.cached.n_tok
    n_req, n_blk = w.n_req, w.n_blk
    state = n_req * hv * dv * dk * 4
    n_gates = 2 if L.family == 0 else 1
    out = {}
    out["init_single"] = dict(bytes=2 * state, flops=0)
    # scan: every chunk at its actual token count (a ragged tail chunk is not padded)
    def chunk_sizes(lens):
        for n in lens:
            n = int(n)
            for c0 in range(0, n, C):
                yield min(C, n - c0)
    if L.family == 0:
        scan_flops = sum(5 * 2 * n * n * dk + 3 * 2 * n * dk * dv + n ** 3 / 3 for n in chunk_sizes(np.diff(w.online.cu)))
    else:
        scan_flops = sum(2 * n * n * dk + 2 * n * n * dv + 2 * 2 * n * dk * dv for n in chunk_sizes(np.diff(w.online.cu)))
    out["scan"] = dict(bytes=T * (2 * hq * dk * io + hv * dv * io * 2 + n_gates * hv * gb) + 2 * state,
                       flops=scan_flops * hv)
    # fold: the transitions the composition reads (blocks at position 2..K of some request)
    K = np.diff(w.blk_cu)
    n_trans = int(np.sum(np.maximum(K - 1, 0)))
    dropped = set(fold_dropped_blocks(w))
    blens = [int(x) for b, x in enumerate(np.diff(w.cached.cu)) if b not in dropped]
    Tf = sum(blens)
    if L.family == 0:
        fold_flops = sum(2 * n * n * dk + n ** 3 / 3 + 2 * n * dk * dk + 2 * n * n * dk + 2 * n * dk * dk
                         for n in chunk_sizes(blens))
        out["fold"] = dict(bytes=Tf * (hq * dk * io + 2 * hv * gb) + (w.n_blk - len(dropped)) * hv * dk * dk * 4,
                           flops=fold_flops * hv)
    else:
        out["fold"] = dict(bytes=Tf * hv * 4 + (w.n_blk - len(dropped)) * hv * 4, flops=Tf * hv)
    # composition
    if L.family == 0:
        out["compose"] = dict(bytes=(n_blk * hv * dv * dk + n_trans * hv * dk * dk) * 4 + state,
                              flops=n_trans * hv * 2 * dv * dk * dk)
    else:
        out["compose"] = dict(bytes=n_blk * hv * dv * dk * 4 + n_trans * hv * 4 + state,
                              flops=n_trans * hv * 2 * dv * dk)
    return out


def roofline(name, work, ms, bound=None):
    """Achieved rate of one kernel against its roofline.  ``bound`` defaults to the
    side with the larger lower bound on time (bytes / HBM peak vs flops / bf16
    MFMA peak); both fractions are given."""
    secs = ms * 1e-3
    gbs = work["bytes"] / secs / 1e9
    tfs = work["flops"] / secs / 1e12
    if bound is None:
        bound = "mfma" if work["flops"] / MFMA_BF16_PEAK_TFLOPS / 1e12 > work["bytes"] / HBM_PEAK_GBS / 1e9 \
            else "hbm"
    common = dict(traffic=None, avg_us=round(ms * 1e3, 2), algorithmic_flops=work["flops"],
                  algorithmic_bytes=work["bytes"], frac_hbm=round(gbs / HBM_PEAK_GBS, 4),
                  frac_mfma=round(tfs / MFMA_BF16_PEAK_TFLOPS, 4))
    if bound == "mfma":
        return dict(kernel=name, bound="mfma", achieved=round(tfs, 2), peak=MFMA_BF16_PEAK_TFLOPS,
                    unit="TFLOP/s", frac=round(tfs / MFMA_BF16_PEAK_TFLOPS, 4), **common)
    return dict(kernel=name, bound="hbm", achieved=round(gbs, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(gbs / HBM_PEAK_GBS, 4), **common)


# ---------------------------------------------------------------- decode step
def decode_bench(w, S_final, steps: int, batches=(None, 256)):
    """Time the decode step (one token per request) of the workload's layer: on the
    workload's own final states and on a larger decode batch.  Algorithmic bytes =
    every state element read and written once (fp32) plus the token's q/k/v,
    gates and outputs; the bound is HBM."""
    import torch
    from paper_2608_11231_amd import gpu_io
    from paper_2608_11231_amd import inputs as I
    L = w.layer
    io = 2 if L.io_dtype == "bf16" else 4
    gb = 2 if (L.gate_dtype == "bf16" and L.family == I.GDN) else 4
    n_gates = 2 if L.family == I.GDN else 1
    res = {}
    for n_req in batches:
        n_req = w.n_req if n_req is None else n_req
        dw = I.build_workload("decode", L, [[] for _ in range(n_req)], [1] * n_req, I.GateLaw(), 77,
                              scale=w.scale)
        st = gpu_io.GpuStep(dw.online, dw.online.cu[:-1], L, w.A, w.scale)
        if n_req == w.n_req:
            S = S_final.clone()
        else:
            S = 0.1 * torch.randn((n_req, L.h_v, L.dv, L.dk), device="cuda")
        for _ in range(3):
            st.decode(S)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            st.decode(S)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / steps
        nbytes = n_req * (2 * L.h_v * L.dv * L.dk * 4 + 2 * L.h_qk * L.dk * io + 2 * L.h_v * L.dv * io
                          + n_gates * L.h_v * gb)
        gbs = nbytes / (us * 1e-6) / 1e9
        res[f"requests_{n_req}"] = dict(avg_us=round(us, 2), algorithmic_bytes=nbytes, achieved_GBs=round(gbs, 1),
                                        frac=round(gbs / HBM_PEAK_GBS, 4), bound="hbm")
        log(f"[bench] decode step, {n_req} requests: {us:.2f} us, {gbs:.0f} GB/s")
    return res


# ---------------------------------------------------------------- selected-position gather
def gather_bench(w, G, steps: int):
    """Time the gather that forms the recompute's online stream from the context:
    each request's cached context (its blocks, in order) and as many uniformly
    selected positions as it has online tokens.  The context's q rows are not
    part of the cached stream; a separate seeded buffer of the same shape and
    dtype is their source, so no row of one array is served from the cache by
    the read of another.  Algorithmic bytes = every gathered row read once and
    written once."""
    import torch
    from paper_2608_11231_amd import gpu_io
    from paper_2608_11231_amd import inputs as I
    L = w.layer
    ctx_cu = I.context_cu(w)
    rng = np.random.default_rng(2608)
    per = []
    for r in range(w.n_req):
        n_ctx = int(ctx_cu[r + 1] - ctx_cu[r])
        m = int(w.online.cu[r + 1] - w.online.cu[r])
        per.append(I.select_uniform(rng, n_ctx, m / n_ctx) if n_ctx else np.zeros(0, np.int32))
    sel_cu, pos = I.pack_selection(per)
    gen = torch.Generator(device="cuda").manual_seed(2608)
    ctx_q = torch.randn(tuple(G.cached.k.shape), generator=gen, device="cuda").to(G.cached.k.dtype)
    sel = gpu_io.GpuSelection(G.cached, ctx_cu, sel_cu, pos, L, ctx_q=ctx_q)
    for _ in range(3):
        sel.gather()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        sel.gather()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / steps
    row = sum(x.element_size() * x[0].numel() for x in (sel.q, sel.k, sel.v, sel.g, sel.beta) if x is not None)
    nbytes = 2 * sel.n_sel * row
    gbs = nbytes / (us * 1e-6) / 1e9
    log(f"[bench] gather of {sel.n_sel} selected tokens: {us:.2f} us, {gbs:.0f} GB/s")
    return dict(selected_tokens=sel.n_sel, avg_us=round(us, 2), algorithmic_bytes=nbytes,
                achieved_GBs=round(gbs, 1), frac=round(gbs / HBM_PEAK_GBS, 4), bound="hbm")


# ---------------------------------------------------------------- bf16 pool and staging
def staging_bench(w, G, steps: int):
    """The cache in its stored form (bf16 block states and, for exact composition,
    the cached key/gate streams, in pinned host memory) and the batch's
    host-to-device staging: the single-block rows (one per request) vs the
    exact-composition rows (every block's state plus its token stream).  Also
    times the fp32 -> bf16 pool rounding, the bf16-pool initialisations, and
    single-block staging on a side stream while the scan runs."""
    import torch
    from paper_2608_11231_amd import gpu_io, lkv
    L = w.layer
    Bq = torch.empty(G.B_pool.shape, dtype=torch.bfloat16, device="cuda")

    def timed(fn, n, stream=None):
        st = stream or torch.cuda.current_stream()
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(st)
        for _ in range(n):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    us_round = timed(lambda: lkv.round_bf16(G.B_pool, Bq), steps)
    hc = gpu_io.HostCache(w, Bq.float().cpu().numpy())
    sb = gpu_io.StagedBatch(hc, w.blk_ids, w.blk_cu, w.last_blk)
    side = torch.cuda.Stream()
    us_single = timed(lambda: sb.stage_single(side), steps, side)
    us_exact = timed(lambda: sb.stage_exact(side), max(2, steps // 10), side)
    S = torch.empty_like(G.S_single)
    us_init1 = timed(lambda: sb.init_single(S), steps)
    us_initx = timed(lambda: sb.init_compose(S), max(2, steps // 4))
    us_scan = timed(lambda: G.scan(G.S_exact), steps)
    main = torch.cuda.current_stream()

    def both():
        # the next batch's rows are staged while this batch's scan runs: the scan is
        # enqueued first, and the copy carries no cross-stream wait (a copy queued
        # behind an event of another stream holds the host until that event fires)
        G.scan(G.S_exact)
        sb.stage_single(side)
        main.wait_stream(side)
    us_both = timed(both, steps)
    b1, bx = sb.staged_bytes(False), sb.staged_bytes(True)
    log(f"[bench] staging: single-block rows {b1 / 2**20:.1f} MiB in {us_single:.1f} us, exact-composition "
        f"rows {bx / 2**20:.1f} MiB in {us_exact:.1f} us; scan {us_scan:.1f} us alone, {us_both:.1f} us "
        f"with single-block staging alongside")
    return dict(pool_round_bf16_us=round(us_round, 2),
                single_block=dict(bytes=b1, h2d_us=round(us_single, 2), GBs=round(b1 / us_single / 1e3, 1),
                                  init_from_bf16_us=round(us_init1, 2)),
                exact=dict(bytes=bx, h2d_us=round(us_exact, 2), GBs=round(bx / us_exact / 1e3, 1),
                           fold_plus_compose_from_bf16_us=round(us_initx, 2)),
                overlap=dict(scan_us=round(us_scan, 2), scan_with_single_staging_us=round(us_both, 2)))


# ---------------------------------------------------------------- relative-error probe
def diag_bench(w, G, steps: int):
    """The per-layer relative error of both initial states against the full-prefix
    state S* (the scan of each request's whole cached context from zero), as in
    the paper's construction-time probe, on this layer's synthetic inputs
    (first-layer-like: a block's tokens do not depend on what precedes it, so
    exact composition should land on S*); and the diagnostic kernel's time."""
    import torch
    from paper_2608_11231_amd import inputs as I
    from paper_2608_11231_amd import lkv
    ctx_cu = I.context_cu(w)
    cu = torch.from_numpy(ctx_cu).cuda()
    c = G.cached
    full = lkv.make_tokens(cu, int(ctx_cu[-1]), None, c.k, c.v, c.g, c.beta, c.A)
    S_star = torch.empty_like(G.S_exact)
    if w.layer.family == I.GDN:
        lkv.gdn_chunk_scan(G.layer, full, 1.0, None, None, S_star)
    else:
        lkv.ssd_chunk_scan(G.layer, full, None, None, S_star)
    G.fold_transitions()
    G.init_single()
    G.init_compose()
    h = w.layer.h_v
    _, _, rx = lkv.state_rel_error(G.S_exact, S_star, group=h)
    _, _, r1 = lkv.state_rel_error(G.S_single, S_star, group=h)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        lkv.state_rel_error(G.S_single, S_star, group=h)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / steps
    nbytes = 2 * G.S_single.numel() * 4
    log(f"[bench] layer-0 probe ({w.name}): exact {rx.max().item():.2e}, last block "
        f"{r1.min().item():.3e}..{r1.max().item():.3e}; diagnostic {us:.2f} us")
    return dict(workload=w.name, rel_exact_vs_full_prefix=[float(x) for x in rx.cpu()],
                rel_last_block_vs_full_prefix=[float(x) for x in r1.cpu()],
                kernel_us=round(us, 2), algorithmic_bytes=nbytes,
                achieved_GBs=round(nbytes / us / 1e3, 1))


# ---------------------------------------------------------------- CPU oracle baseline
def cpu_baseline(w, budget_s: float):
    """Time the fp64 CPU oracle on request 0 (all heads) and scale to the step."""
    import oracle
    from paper_2608_11231_amd import inputs as I
    L = w.layer
    gdn = L.family == I.GDN
    cores = int(os.environ.get("OMP_NUM_THREADS", 0) or len(os.sched_getaffinity(0)))
    oracle.load()
    c, o = w.cached, w.online
    b0, b1 = int(w.blk_cu[0]), int(w.blk_cu[1])
    t0, t1 = int(c.cu[b0]), int(c.cu[b1])
    # scan sample: request 0, every head
    s0, s1 = int(o.cu[0]), int(o.cu[1])
    cu = np.array([0, s1 - s0], np.int32)
    S0 = np.zeros((1, L.h_v, L.dv, L.dk))
    tic = time.perf_counter()
    if gdn:
        oracle.gdn_scan(cu, o.q[s0:s1], o.k[s0:s1], o.v[s0:s1], o.g[s0:s1], o.beta[s0:s1],
                        scale=w.scale, S0=S0)
    else:
        oracle.ssd_scan(cu, o.q[s0:s1], o.k[s0:s1], o.v[s0:s1], o.g[s0:s1], w.A, S0=S0)
    t_scan = time.perf_counter() - tic
    # fold sample: request 0's blocks 2..K (the transitions the composition reads),
    # as many as fit in the remaining budget
    fold_blocks = []
    est_per_tok = t_scan / max(s1 - s0, 1)
    room = max(budget_s - 2 * t_scan, budget_s * 0.25)
    tok = 0
    for b in range(b0 + 1 if b1 > b0 + 1 else b0, b1):
        L_b = int(c.cu[b + 1] - c.cu[b])
        if fold_blocks and (tok + L_b) * est_per_tok > room:
            break
        fold_blocks.append(b)
        tok += L_b
    fb0, fb1 = fold_blocks[0], fold_blocks[-1] + 1
    ft0, ft1 = int(c.cu[fb0]), int(c.cu[fb1])
    fcu = (c.cu[fb0:fb1 + 1] - c.cu[fb0]).astype(np.int32)
    tic = time.perf_counter()
    if gdn:
        oracle.gdn_transition(fcu, c.k[ft0:ft1], c.g[ft0:ft1], c.beta[ft0:ft1])
    else:
        oracle.ssd_log_decay(fcu, c.g[ft0:ft1], w.A)
    t_fold = time.perf_counter() - tic
    # compose sample: request 0 on synthetic pools of the real shapes
    K0 = b1 - b0
    rng = np.random.default_rng(0)
    Bp = rng.standard_normal((K0, L.h_v, L.dv, L.dk))
    Mp = rng.standard_normal((K0, L.h_v, L.dk, L.dk)) / np.sqrt(L.dk) if gdn else \
        -rng.uniform(0, 1, (K0, L.h_v))
    ids = np.arange(K0, dtype=np.int32)
    tic = time.perf_counter()
    (oracle.compose_gdn if gdn else oracle.compose_ssd)(np.array([0, K0], np.int32), ids, Bp, Mp)
    t_comp = time.perf_counter() - tic
    tic = time.perf_counter()
    oracle.init_single(Bp, np.array([K0 - 1], np.int32))
    t_single = time.perf_counter() - tic
    # scale each op to the whole batch by its units of work
    T_all = w.online.n_tok
    n_trans_all = int(np.sum(np.maximum(np.diff(w.blk_cu) - 1, 0)))
    dropped = set(fold_dropped_blocks(w))
    T_fold = sum(int(x) for b, x in enumerate(np.diff(c.cu)) if b not in dropped)
    step = (t_scan * T_all / (s1 - s0) + t_fold * T_fold / max(ft1 - ft0, 1)
            + t_comp * n_trans_all / max(K0 - 1, 1) + t_single * w.n_req)
    sample = (f"request 0 of {w.n_req}, all {L.h_v} heads: scan of {s1 - s0} online tokens "
              f"({t_scan:.2f} s), transition fold of {len(fold_blocks)} cached blocks / {ft1 - ft0} tokens "
              f"({t_fold:.2f} s), {K0}-block composition ({t_comp:.2f} s), single init; scaled by "
              f"tokens / transitions / requests to the whole step")
    return dict(value=round(T_all / step, 1), unit="tokens/s", cores=cores, kind="oracle", sample=sample,
                step_s_extrapolated=round(step, 3))


# ---------------------------------------------------------------- timing
FLUSH_BYTES = 512 << 20   # twice the 256 MB Infinity Cache


class Timer:
    """Per-step and per-op HIP-event timing of a step made of ops, on the stream
    the library launches on (torch's current stream).  Cold steps are each
    preceded by an untimed write of a 512 MiB buffer, which evicts the Infinity
    Cache; warm steps run back to back."""

    def __init__(self):
        import torch
        self.torch = torch
        self.flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda")

    def flush(self, k):
        self.flush_buf.fill_(k & 0x7fffffff)

    def run(self, ops, steps: int, cold: bool):
        torch = self.torch
        ev = lambda: torch.cuda.Event(enable_timing=True)
        marks = [[ev() for _ in range(len(ops) + 1)] for _ in range(steps)]
        torch.cuda.synchronize()
        for k in range(steps):
            if cold:
                self.flush(k)
            m = marks[k]
            m[0].record()
            for i, (_, f) in enumerate(ops):
                f()
                m[i + 1].record()
        torch.cuda.synchronize()
        step_ms = [m[0].elapsed_time(m[-1]) for m in marks]
        op_ms = {name: [m[i].elapsed_time(m[i + 1]) for m in marks] for i, (name, _) in enumerate(ops)}
        return step_ms, op_ms


def stats(xs):
    xs = sorted(xs)
    n = len(xs)
    med = xs[n // 2] if n % 2 else 0.5 * (xs[n // 2 - 1] + xs[n // 2])
    return dict(median_us=round(med * 1e3, 2), mean_us=round(sum(xs) / n * 1e3, 2), min_us=round(xs[0] * 1e3, 2),
                max_us=round(xs[-1] * 1e3, 2), n=n)


def measured_peaks():
    """Measured denominators on this GPU, each the best median (of 20 launches)
    over a few probes: HBM from plain device copies (read + write bytes / time)
    of 512 MiB and 2 GiB and an in-place fp32 scale of 2 GiB; bf16 matrix-core
    rate from torch.matmul (hipBLASLt) at 8192^3 and 16384 x 16384 x 8192."""
    import torch

    def med20(fn):
        for _ in range(3):
            fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
        torch.cuda.synchronize()
        for e0, e1 in evs:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        return sorted(e0.elapsed_time(e1) for e0, e1 in evs)[10] * 1e-3

    hbm, mfma = {}, {}
    for nbytes in (512 << 20, 2 << 30):
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        hbm[f"copy_{nbytes >> 20}MiB"] = 2 * nbytes / med20(lambda: dst.copy_(src)) / 1e9
        del src, dst
    x = torch.ones((2 << 30) // 4, dtype=torch.float32, device="cuda")
    hbm["scale_2048MiB"] = 2 * x.numel() * 4 / med20(lambda: x.mul_(1.0)) / 1e9
    del x
    for m_, n_, k_ in ((8192, 8192, 8192), (16384, 16384, 8192)):
        a = torch.randn((m_, k_), device="cuda").to(torch.bfloat16)
        b = torch.randn((k_, n_), device="cuda").to(torch.bfloat16)
        mfma[f"matmul_{m_}x{n_}x{k_}"] = 2 * m_ * n_ * k_ / med20(lambda: torch.matmul(a, b)) / 1e12
        del a, b
    torch.cuda.empty_cache()
    return dict(hbm_GBs=round(max(hbm.values()), 1), bf16_TFLOPs=round(max(mfma.values()), 1),
                hbm_probes={k: round(v, 1) for k, v in hbm.items()},
                mfma_probes={k: round(v, 1) for k, v in mfma.items()})


def traffic_table(w):
    """Measured HBM bytes per launch of each op of the step, from the committed
    rocprofv3 counter summary of this workload, when it was taken on the current
    kernel sources."""
    from paper_2608_11231_amd import rocprof_summary
    table = rocprof_summary.read_traffic(os.path.join(ROOT, "profiles", f"{w.name}_hbm_traffic.txt"))
    if not table:
        return {}
    fam = w.layer.family

    def chunk_mode(n):
        # lkv::chunk_kernel<FAM,DK,CH,F32IO,NB,SUMMARY,RT>: family and summary flag
        if not n.startswith("lkv::chunk_kernel<"):
            return None
        args = n[len("lkv::chunk_kernel<"):].rstrip(">").split(",")
        return (int(args[0]), args[5] == "true") if len(args) >= 6 else None

    pick = {"scan": lambda n: chunk_mode(n) == (fam, False),
            "fold": (lambda n: chunk_mode(n) == (fam, True)) if fam == 0 else (lambda n: "ssd_lambda" in n),
            # the step composes from and copies out of fp32 pools (the <..., false> variants)
            "compose": lambda n: "compose" in n and n.rstrip(">").endswith("false"),
            "init_single": lambda n: "init_single" in n and n.rstrip(">").endswith("false")}
    out = {}
    for op, pred in pick.items():
        cand = [v for (n, grid), v in table.items() if pred(n)]
        if len(cand) == 1:
            out[op] = round(cand[0])
    return out


def measure(w, G, steps: int, warmup: int, timer: Timer):
    """The step's four calls on workload ``w``: cold (the headline: Infinity Cache
    flushed before every step, medians) and warm (back to back).  Returns the
    per-op and per-step figures, the rooflines and the two paths' rates."""
    from paper_2608_11231_amd.gpu_io import sp_pieces
    pieces = sp_pieces(w)  # sequence-parallel scan where the (request, head) chains underfill the GPU
    ops = [("init_single", G.init_single),
           ("fold", G.fold_transitions),
           ("compose", G.init_compose),
           ("scan", lambda: G.scan(G.S_exact, pieces=pieces))]
    timer.run(ops, warmup, cold=False)
    cold_step, cold_op = timer.run(ops, steps, cold=True)
    warm_step, warm_op = timer.run(ops, steps, cold=False)
    T = w.online.n_tok
    cold = {k: stats(v) for k, v in cold_op.items()}
    warm = {k: stats(v) for k, v in warm_op.items()}
    med = {k: v["median_us"] * 1e-3 for k, v in cold.items()}   # ms
    work = work_model(w)
    # the Gated DeltaNet fold sits at the ridge (404 GFLOP over 1.32 GB at 32K) and its
    # time goes to matrix-core work (the hi/lo passes double it): priced against MFMA
    bounds = {"fold": "mfma"} if w.layer.family == 0 else {}
    roofs = {name: roofline(name, work[name], med[name], bounds.get(name)) for name in med}
    for op, tb in traffic_table(w).items():
        roofs[op]["traffic"] = tb
    step_med = stats(cold_step)["median_us"] * 1e-3
    return dict(
        step_cold=stats(cold_step), step_warm=stats(warm_step), ops_cold=cold, ops_warm=warm,
        roofline_by_kernel=roofs, dominant=max(med, key=med.get),
        tokens_per_s=round(T / (step_med * 1e-3), 1),
        lb_tokens_per_s=round(T / ((med["init_single"] + med["scan"]) * 1e-3), 1),
        ex_tokens_per_s=round(T / ((med["fold"] + med["compose"] + med["scan"]) * 1e-3), 1),
        composition_latency_us=round(med["compose"] * 1e3, 2),
        fold_plus_compose_latency_us=round((med["fold"] + med["compose"]) * 1e3, 2),
        single_init_latency_us=round(med["init_single"] * 1e3, 2),
        scan_us=round(med["scan"] * 1e3, 2),
        scan_pieces=pieces)


def workload_desc(w):
    from paper_2608_11231_amd import inputs as I
    L = w.layer
    T = w.online.n_tok
    return (f"{w.name}: {'Gated DeltaNet' if L.family == I.GDN else 'Mamba-2 SSD'} layer, "
            f"{w.n_req} requests, {T} online tokens, {L.h_v} heads"
            f"{f' ({L.h_qk} q/k)' if L.h_qk != L.h_v and L.family == I.GDN else ''}, dk={L.dk}, dv={L.dv}, "
            f"chunk {L.chunk}, {w.n_blk} cached blocks ({w.cached.n_tok} tokens), bf16 inputs, fp32 state")


# ---------------------------------------------------------------- main
def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50, help="timed steps (cold and warm each); medians reported")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=3,
                    help="workload index (default 3: Gated DeltaNet, 32K context, 4 requests)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of CPU-oracle work")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the timings outside the step (decode, gather, staging, probe)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (8K Gated DeltaNet, 8K Mamba-2, ragged 16K)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured-peak probes")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after timing, run a plain 512 MiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures one GPU only (the hot path is per-GPU; see the "
              "sharding note in the design document); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_11231_amd import gpu_io
    from paper_2608_11231_amd import inputs as I

    torch.cuda.set_device(0)
    timer = Timer()
    tic = time.perf_counter()
    w = I.config(args.config, workers=16)
    log(f"[bench] workload {w.name}: {w.online.n_tok} online tokens, {w.cached.n_tok} cached tokens in "
        f"{w.n_blk} blocks, generated in {time.perf_counter() - tic:.1f} s")
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=False)        # the cache content: per-block states
    torch.cuda.synchronize()
    log("[bench] inputs resident in HBM; block states built")
    m = measure(w, G, args.steps, args.warmup, timer)
    log("[bench] cold medians: " + ", ".join(f"{k} {v['median_us']:.1f} us" for k, v in m["ops_cold"].items())
        + f"; step {m['step_cold']['median_us']:.1f} us (warm {m['step_warm']['median_us']:.1f} us)")

    # LinearKV's path as one launch: the scan starting from the cached pool row
    from paper_2608_11231_amd import lkv
    fused = lambda: lkv.chunk_scan_from_pool(G.layer, G.online.struct, w.scale, G.B_pool, w.n_blk, G.last_blk,
                                             G.out, G.S_final)
    timer.run([("fused", fused)], 3, cold=False)
    _, f_op = timer.run([("fused", fused)], args.steps, cold=True)
    fused_us = stats(f_op["fused"])["median_us"]
    log(f"[bench] LinearKV path in one launch (scan from the pool row): {fused_us:.1f} us")

    decode = None if args.no_decode else decode_bench(w, G.S_final, args.steps)
    gather = None if args.no_decode else gather_bench(w, G, args.steps)
    staging = None if (args.no_decode or w.layer.family != I.GDN) else staging_bench(w, G, args.steps)
    diag = None
    if not args.no_decode:
        diag = dict(default_gates=diag_bench(w, G, args.steps))
        wm = I.config(args.config, mild=True, workers=16)
        Gm = gpu_io.GpuWorkload(wm)
        Gm.block_summary(B=True, M=False)
        diag["mild_gates"] = diag_bench(wm, Gm, args.steps)
        del Gm

    others = {}
    if not args.no_configs:
        for idx in (1, 2, 4):
            if idx == args.config:
                continue
            wo = I.config(idx, workers=16)
            Go = gpu_io.GpuWorkload(wo)
            Go.block_summary(B=True, M=False)
            mo = measure(wo, Go, args.steps, args.warmup, timer)
            mo["workload"] = workload_desc(wo)
            others[wo.name] = mo
            log(f"[bench] {wo.name} cold medians: " + ", ".join(
                f"{k} {v['median_us']:.1f} us" for k, v in mo["ops_cold"].items())
                + f"; step {mo['step_cold']['median_us']:.1f} us")
            del Go

    # measured denominators last, so that their heat does not slow the timings above
    peaks = None
    if not args.no_peaks:
        peaks = measured_peaks()
        log(f"[bench] measured peaks: HBM {peaks['hbm_GBs']:.0f} GB/s, bf16 matmul {peaks['bf16_TFLOPs']:.0f} "
            f"TFLOP/s")
        for r in [*m["roofline_by_kernel"].values(),
                  *(x for o in others.values() for x in o["roofline_by_kernel"].values())]:
            meas = peaks["hbm_GBs"] if r["bound"] == "hbm" else peaks["bf16_TFLOPs"]
            r["frac_of_measured_peak"] = round(r["achieved"] / meas, 4)

    if args.copy_probe:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    T = w.online.n_tok
    L = w.layer
    roofs = m["roofline_by_kernel"]
    result = {
        "metric": "online linear-layer prefill tokens/s at 8K/32K; K-way composition latency (us)",
        "value": m["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(m["step_cold"]["median_us"] * 1e-3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": workload_desc(w),
            "online_tokens": T,
            "cached_tokens": w.cached.n_tok,
            "cached_blocks": w.n_blk,
            "requests": w.n_req,
            "parallelism": "single GPU",
        },
        "timing": ("cold: each timed step preceded by an untimed 512 MiB buffer write (Infinity Cache "
                   "evicted); value and per-kernel figures are medians over the cold steps; warm "
                   "(back-to-back) figures alongside"),
        "composition_latency_us": m["composition_latency_us"],
        "fold_plus_compose_latency_us": m["fold_plus_compose_latency_us"],
        "single_init_latency_us": m["single_init_latency_us"],
        "scan_us": m["scan_us"],
        "lb_tokens_per_s": m["lb_tokens_per_s"],
        "lb_fused_us": round(fused_us, 2),
        "lb_fused_tokens_per_s": round(T / (fused_us * 1e-6), 1),
        "ex_tokens_per_s": m["ex_tokens_per_s"],
        "step_cold": m["step_cold"],
        "step_warm": m["step_warm"],
        "ops_cold": m["ops_cold"],
        "ops_warm": m["ops_warm"],
        "measured_peaks": peaks,
        "roofline": roofs[m["dominant"]],
        "roofline_by_kernel": roofs,
        "other_workloads": others,
        "decode_step": decode,
        "gather_selected": gather,
        "bf16_pool_staging": staging,
        "relative_error_probe": diag,
        "cpu_baseline": None,
    }
    if args.copy_probe:
        result["copy_probe_bytes"] = 2 * (512 << 20)
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
