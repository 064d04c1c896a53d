"""GPU parity of every call of liblkv.so against the CPU oracle, on seeded inputs.

Bars: index/gather work bit-exact; every fp32 state-valued output (B, M,
Lambda, S_init, S_final) within 1e-4 normwise relative error per (segment,
head) slice; bf16 outputs within 2e-2 absolute error; fp32-io outputs within
1e-4 relative.  Shapes span several chunks, ragged tails, empty segments and
grouped heads.
"""
import numpy as np
import pytest

from paper_2608_11231_amd import inputs as I

from oracle_ref import max_abs, rel_slices
import oracle_ref as R

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_11231_amd import gpu_io, lkv  # noqa: E402

STATE_TOL = 1e-4
OUT_ABS = 2e-2


def _np(t):
    return t.detach().float().cpu().numpy()


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


GDN_CASES = [
    # (dk, dv, chunk, io, h_qk, h_v, blocks, online)
    (16, 16, 16, "f32", 1, 1, ((64, 64),), (32,)),
    (32, 32, 16, "bf16", 2, 4, ((40, 23), (17, 0, 5)), (37, 70)),
    (64, 64, 64, "bf16", 2, 2, ((130, 64), (1,)), (150, 64)),
    (128, 128, 64, "bf16", 2, 2, ((200, 77),), (193,)),
    (64, 64, 64, "f32", 1, 2, ((90,), (65, 3)), (129, 0)),
    (64, 48, 16, "bf16", 1, 1, ((33,),), (47,)),
    # the largest supported state (dk = 128, dv = 512): eight row tiles per head
    (128, 512, 64, "bf16", 1, 2, ((70, 33),), (90,)),
]

SSD_CASES = [
    # (N, P, chunk, io, G, H, blocks, online)
    (16, 16, 16, "f32", 1, 2, ((40, 23),), (37,)),
    (128, 64, 64, "bf16", 1, 4, ((130, 64), (1, 70)), (150, 64)),
    (64, 32, 16, "bf16", 2, 4, ((50,),), (77,)),
    (64, 64, 16, "f32", 1, 2, ((20,),), (33,)),
    # other state widths with 64-token chunks: grouped B / C, ragged and empty segments
    (32, 64, 64, "bf16", 2, 4, ((100, 0, 65),), (129,)),
    (64, 128, 64, "bf16", 1, 2, ((64, 128), (3,)), (0, 191)),
    # the largest supported state (N = 128, P = 512); kept last (the pinned-geometry test takes it)
    (128, 512, 64, "bf16", 1, 2, ((70,),), (90,)),
]


def _work(fam, case, seed=11):
    dk, dv, chunk, io, hq, hv, blocks, online = case
    layer = I.Layer(fam, hq, hv, dk, dv, chunk, io, io if fam == I.GDN else "f32")
    if fam == I.GDN:
        law = I.GateLaw(x_mu=-3.0, beta_mu=0.0)
    else:
        law = I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0, a_hi=4.0)
    return I.build_workload(f"case{case}", layer, [list(b) for b in blocks], list(online), law, seed,
                            scale=0.75 if fam == I.GDN else 1.0)


@pytest.mark.parametrize("case", GDN_CASES, ids=[f"gdn{c[:4]}" for c in GDN_CASES])
def test_gdn_block_summary(case):
    w = _work(I.GDN, case)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    torch.cuda.synchronize()
    B, M = R.summaries(w)
    assert rel_slices(_np(G.B_pool), B) < STATE_TOL
    assert rel_slices(_np(G.M_pool), M) < STATE_TOL


@pytest.mark.parametrize("case", SSD_CASES, ids=[f"ssd{c[:4]}" for c in SSD_CASES])
def test_ssd_block_summary(case):
    w = _work(I.SSD, case)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    torch.cuda.synchronize()
    B, Lam = R.summaries(w)
    assert rel_slices(_np(G.B_pool), B) < STATE_TOL
    assert np.max(np.abs(_np(G.M_pool) - Lam) / np.maximum(np.abs(Lam), 1e-30)) < STATE_TOL


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_init_single_bit_exact(fam):
    w = _work(fam, GDN_CASES[1] if fam == I.GDN else SSD_CASES[1])
    G = gpu_io.GpuWorkload(w)
    pool = np.random.default_rng(5).standard_normal(tuple(G.B_pool.shape)).astype(np.float32)
    G.B_pool.copy_(_dev(pool))
    src = np.array([w.n_blk - 1, -1, 0, w.n_blk + 3, -7, 1], np.int32)
    S = torch.empty((len(src),) + tuple(G.B_pool.shape[1:]), device="cuda")
    lkv.init_single(G.layer, w.n_blk, G.B_pool, torch.from_numpy(src).cuda(), S)
    torch.cuda.synchronize()
    got = _np(S)
    for r, b in enumerate(src):
        if 0 <= b < w.n_blk:
            assert np.array_equal(got[r].view(np.uint32), pool[b].view(np.uint32))
        elif b == -1:
            assert np.array_equal(got[r], np.zeros_like(got[r]))
        else:
            assert np.isnan(got[r]).all()


def _orth_pool(rng, n, h, d, scale=0.9):
    q, _ = np.linalg.qr(rng.standard_normal((n * h, d, d)))
    return (scale * q).reshape(n, h, d, d)


@pytest.mark.parametrize("dk,dv", [(16, 16), (64, 48), (128, 128), (128, 512)])
def test_gdn_compose_o1_transitions(dk, dv):
    """Composition on O(1)-norm transitions (0.9 x orthogonal), so every block matters."""
    rng = np.random.default_rng(dk + dv)
    n_blk, h = 9, 2
    B = rng.standard_normal((n_blk, h, dv, dk)).astype(np.float32)
    M = _orth_pool(rng, n_blk, h, dk).astype(np.float32)
    blk_cu = np.array([0, 4, 4, 5, 9], np.int32)             # K = 4, 0, 1, 4
    ids = np.array([3, 0, 7, 1, 8, 2, 6, 5, 4], np.int32)
    layer = lkv.make_layer(I.GDN, 1, h, dk, dv, 64)
    S = torch.empty((4, h, dv, dk), device="cuda")
    lkv.init_compose(layer, n_blk, _dev(B), _dev(M), torch.from_numpy(ids).cuda(),
                     torch.from_numpy(blk_cu).cuda(), len(ids), S)
    torch.cuda.synchronize()
    import oracle
    ref = oracle.compose_gdn(blk_cu, ids, B, M)
    got = _np(S)
    assert rel_slices(got[[0, 3]], ref[[0, 3]]) < STATE_TOL
    assert np.array_equal(got[1], np.zeros_like(got[1]))
    assert np.array_equal(got[2].view(np.uint32), B[8].view(np.uint32))   # K = 1: the cached state


def test_compose_invalid_id_gives_nan():
    rng = np.random.default_rng(1)
    B = rng.standard_normal((3, 1, 16, 16)).astype(np.float32)
    M = rng.standard_normal((3, 1, 16, 16)).astype(np.float32)
    layer = lkv.make_layer(I.GDN, 1, 1, 16, 16, 16)
    S = torch.empty((2, 1, 16, 16), device="cuda")
    lkv.init_compose(layer, 3, _dev(B), _dev(M), torch.tensor([0, 5, 1, 2], dtype=torch.int32, device="cuda"),
                     torch.tensor([0, 2, 4], dtype=torch.int32, device="cuda"), 4, S)
    torch.cuda.synchronize()
    got = _np(S)
    assert np.isnan(got[0]).all() and np.isfinite(got[1]).all()


def test_ssd_compose():
    rng = np.random.default_rng(3)
    n_blk, H, P, N = 7, 3, 32, 64
    B = rng.standard_normal((n_blk, H, P, N)).astype(np.float32)
    Lam = (-rng.uniform(0.0, 3.0, (n_blk, H))).astype(np.float32)
    blk_cu = np.array([0, 3, 7], np.int32)
    ids = np.array([6, 0, 2, 1, 3, 4, 5], np.int32)
    layer = lkv.make_layer(I.SSD, 1, H, N, P, 64, gate_dtype=torch.float32)
    S = torch.empty((2, H, P, N), device="cuda")
    lkv.init_compose(layer, n_blk, _dev(B), _dev(Lam), torch.from_numpy(ids).cuda(),
                     torch.from_numpy(blk_cu).cuda(), len(ids), S)
    torch.cuda.synchronize()
    import oracle
    assert rel_slices(_np(S), oracle.compose_ssd(blk_cu, ids, B, Lam)) < STATE_TOL


def _scan_check(w, G, S0_ref):
    o_ref, S_ref = R.scan(w, S0_ref)
    G.scan(_dev(S0_ref))
    torch.cuda.synchronize()
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    if w.layer.io_dtype == "f32":
        assert rel_slices(_np(G.out)[None], o_ref[None], lead=1) < STATE_TOL
    else:
        assert max_abs(_np(G.out), o_ref) < OUT_ABS


@pytest.mark.parametrize("case", GDN_CASES, ids=[f"gdn{c[:4]}" for c in GDN_CASES])
def test_gdn_scan_from_composed_state(case):
    w = _work(I.GDN, case)
    B, M = R.summaries(w)
    S0 = R.init_compose(w, B, M)
    _scan_check(w, gpu_io.GpuWorkload(w, with_cached=False), S0)


@pytest.mark.parametrize("case", SSD_CASES, ids=[f"ssd{c[:4]}" for c in SSD_CASES])
def test_ssd_scan_from_composed_state(case):
    w = _work(I.SSD, case)
    B, M = R.summaries(w)
    S0 = R.init_compose(w, B, M)
    _scan_check(w, gpu_io.GpuWorkload(w, with_cached=False), S0)


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_scan_zero_start_and_in_place(fam):
    case = GDN_CASES[2] if fam == I.GDN else SSD_CASES[1]
    w = _work(fam, case)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    o_ref, S_ref = R.scan(w, None)
    G.scan(None)
    torch.cuda.synchronize()
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    # in place: S_init aliases S_final
    rng = np.random.default_rng(2)
    S0 = (0.3 * rng.standard_normal(tuple(G.S_final.shape))).astype(np.float32)
    o_ref, S_ref = R.scan(w, S0)
    G.S_final.copy_(_dev(S0))
    G.scan(G.S_final)
    torch.cuda.synchronize()
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    assert max_abs(_np(G.out), o_ref) < OUT_ABS


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_deterministic(fam):
    case = GDN_CASES[3] if fam == I.GDN else SSD_CASES[1]
    w = _work(fam, case)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    G.init_compose()
    G.scan(G.S_exact)
    torch.cuda.synchronize()
    first = [t.clone() for t in (G.B_pool, G.M_pool, G.S_exact, G.S_final, G.out)]
    G.block_summary()
    G.init_compose()
    G.scan(G.S_exact)
    torch.cuda.synchronize()
    for a, b in zip(first, (G.B_pool, G.M_pool, G.S_exact, G.S_final, G.out)):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))


def test_fp32_io_needs_dk_at_most_64():
    w = _work(I.GDN, (128, 32, 64, "f32", 1, 1, ((20,),), (20,)))
    G = gpu_io.GpuWorkload(w, with_cached=False)
    with pytest.raises(lkv.LkvError, match="UNSUPPORTED"):
        G.scan(None)


def test_tiny_config_end_to_end():
    """The 1-head fp32 workload: block summaries, both init modes and the scan."""
    w = I.config(0)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    G.init_single()
    G.init_compose()
    torch.cuda.synchronize()
    B, M = R.summaries(w)
    assert rel_slices(_np(G.B_pool), B) < STATE_TOL and rel_slices(_np(G.M_pool), M) < STATE_TOL
    S1 = R.init_single(w, B)
    SX = R.init_compose(w, B, M)
    assert rel_slices(_np(G.S_single), S1) < STATE_TOL
    assert rel_slices(_np(G.S_exact), SX) < STATE_TOL
    for S_dev, S_ref in ((G.S_single, S1), (G.S_exact, SX)):
        o_ref, Sf_ref = R.scan(w, S_ref)
        G.scan(S_dev)
        torch.cuda.synchronize()
        assert rel_slices(_np(G.S_final), Sf_ref) < STATE_TOL
        assert rel_slices(_np(G.out)[None], o_ref[None], lead=1) < STATE_TOL


@pytest.mark.parametrize("fam,bf", [(I.GDN, False), (I.GDN, True), (I.SSD, False), (I.SSD, True)])
def test_scan_from_pool_matches_init_then_scan(fam, bf):
    """LinearKV's one-launch path (the scan reading its start from the pool row) is
    bit-identical to the single-block initialisation followed by the scan; -1 starts
    from zero and an invalid id gives NaN."""
    case = GDN_CASES[1] if fam == I.GDN else SSD_CASES[2]
    w = _work(fam, case)
    # four requests: reuse the workload's online stream by repeating its segments
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=False)
    pool = G.B_pool.to(torch.bfloat16) if bf else G.B_pool
    n_req = w.n_req
    src = np.array([w.n_blk - 1, -1][:n_req] + [0] * max(0, n_req - 2), np.int32)
    src_d = torch.from_numpy(src).cuda()
    S_ref = torch.empty_like(G.S_single)
    if bf:
        lkv.init_single_bf16(G.layer, w.n_blk, pool, src_d, S_ref)
    else:
        lkv.init_single(G.layer, w.n_blk, pool, src_d, S_ref)
    G.scan(S_ref)
    torch.cuda.synchronize()
    out_ref, SF_ref = G.out.clone(), G.S_final.clone()
    G.out.zero_()
    G.S_final.zero_()
    lkv.chunk_scan_from_pool(G.layer, G.online.struct, w.scale, pool, w.n_blk, src_d, G.out, G.S_final)
    torch.cuda.synchronize()
    ob = (lambda t: t.view(torch.int16)) if G.out.dtype == torch.bfloat16 else (lambda t: t.view(torch.int32))
    assert torch.equal(ob(G.out), ob(out_ref))
    assert torch.equal(G.S_final.view(torch.int32), SF_ref.view(torch.int32))
    # an invalid id: that request's state and outputs are NaN, the others unchanged
    src_bad = src.copy()
    src_bad[0] = w.n_blk + 5
    lkv.chunk_scan_from_pool(G.layer, G.online.struct, w.scale, pool, w.n_blk, torch.from_numpy(src_bad).cuda(),
                             G.out, G.S_final)
    torch.cuda.synchronize()
    assert torch.isnan(G.S_final[0]).all()
    if n_req > 1:
        assert torch.equal(G.S_final[1:].view(torch.int32), SF_ref[1:].view(torch.int32))


@pytest.mark.parametrize("case", SSD_CASES, ids=[f"ssd{c[:4]}" for c in SSD_CASES])
def test_ssd_lambda_only(case):
    """Mamba-2 transitions alone (no B_out): the segmented dt sum, from dt and A only
    (k and v may be absent), against the oracle and the combined summary."""
    w = _work(I.SSD, case)
    G = gpu_io.GpuWorkload(w)
    c = G.cached
    blocks = lkv.make_tokens(c.cu, c.n_tok, None, None, None, c.g, None, c.A)
    lam = torch.empty((w.n_blk, w.layer.h_v), device="cuda")
    lkv.block_summary(G.layer, blocks, None, lam)
    G.block_summary(B=True, M=True)
    torch.cuda.synchronize()
    _, ref = R.summaries(w)
    got = _np(lam)
    assert np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)) < STATE_TOL
    assert np.max(np.abs(got - _np(G.M_pool)) / np.maximum(np.abs(ref), 1e-30)) < STATE_TOL


# The method's degenerate gates, on the online scan:
#   Gated DeltaNet alpha = 1, beta = 0: every update term is an exact zero and
#   b_C = 1, so the state passes through bit for bit and o = scale * S_0 q;
#   alpha = 1, beta = 1 (the plain delta rule); strong forgetting (log alpha = -30
#   per token, so a chunk's decay underflows); Mamba-2 with vanishing dt and
#   with dt = 4 (per-token decay e^-4 .. e^-16; larger dt would only grow the
#   outputs past what bf16 rounding keeps within the absolute output bar).
DEGENERATE = [
    (I.GDN, 0.0, 0.0, True),
    (I.GDN, 0.0, 1.0, False),
    (I.GDN, -30.0, 0.5, False),
    (I.SSD, 1e-6, None, False),
    (I.SSD, 4.0, None, False),
]


@pytest.mark.parametrize("fam,gate,beta,identity", DEGENERATE,
                         ids=["gdn_a1_b0", "gdn_a1_b1", "gdn_forget", "ssd_dt_tiny", "ssd_dt_large"])
def test_degenerate_gates(fam, gate, beta, identity):
    case = (64, 64, 64, "bf16", 2, 2, ((130, 64), (1,), (40,)), (150, 64, 1)) if fam == I.GDN \
        else (128, 64, 64, "bf16", 1, 4, ((130, 64), (1,), (40,)), (150, 64, 1))
    w = _work(fam, case)
    w.online.g[...] = gate
    if beta is not None:
        w.online.beta[...] = beta
    rng = np.random.default_rng(5)
    L = w.layer
    S0 = (0.5 * rng.standard_normal((w.n_req, L.h_v, L.dv, L.dk))).astype(np.float32)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    if identity:
        G.scan(_dev(S0))
        torch.cuda.synchronize()
        assert np.array_equal(_np(G.S_final).view(np.uint32), S0.view(np.uint32))
    _scan_check(w, G, S0)


@pytest.mark.parametrize("chunk", [16, 64])
def test_wait_that_gives_up_makes_nan(chunk):
    """The solver's bounded wait, forced from the host to give up at once (0
    polls): every Gated DeltaNet chunk kernel still ends, its states,
    transitions and outputs come out NaN on every non-empty segment instead of
    plausible values, and with the default bound back the same calls match the
    oracle again."""
    case = (64, 64, chunk, "bf16", 2, 2, ((130, 64), (0, 9), (5,)), (150, 0, 64))
    w = _work(I.GDN, case)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()                      # a valid pool for the scan from the pool
    torch.cuda.synchronize()
    pool = _np(G.B_pool)
    prev = lkv.set_wait_limit(0)
    try:
        G.scan(None)
        lkv.chunk_scan_from_pool(G.layer, G.online.struct, w.scale, G.B_pool, w.n_blk, G.last_blk, G.out,
                                 G.S_exact)
        G.block_summary()
        torch.cuda.synchronize()
    finally:
        lkv.set_wait_limit(prev)
    blens = np.diff(w.cached.cu)
    olens = np.diff(w.online.cu)
    B, M = _np(G.B_pool), _np(G.M_pool)
    for b, n in enumerate(blens):
        assert np.isnan(B[b]).all() == (n > 0) and np.isnan(M[b]).all() == (n > 0), b
        if n == 0:
            assert np.array_equal(B[b], np.zeros_like(B[b]))
            assert np.array_equal(M[b], np.broadcast_to(np.eye(w.layer.dk, dtype=np.float32), M[b].shape))
    SF, SP = _np(G.S_final), _np(G.S_exact)
    for r, n in enumerate(olens):
        assert np.isnan(SF[r]).all() == (n > 0) and np.isnan(SP[r]).all() == (n > 0), r
        if n == 0:
            assert np.array_equal(SF[r], np.zeros_like(SF[r]))
            assert np.array_equal(SP[r].view(np.uint32), pool[w.last_blk[r]].view(np.uint32))
    assert np.isnan(_np(G.out)).all()
    # default bound restored: normal results
    G.block_summary()
    G.scan(None)
    torch.cuda.synchronize()
    Bo, Mo = R.summaries(w)
    assert rel_slices(_np(G.B_pool), Bo) < STATE_TOL and rel_slices(_np(G.M_pool), Mo) < STATE_TOL
    o_ref, S_ref = R.scan(w, None)
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    assert max_abs(_np(G.out), o_ref) < OUT_ABS


@pytest.mark.parametrize("scale", [0.9, 0.99])
def test_gdn_compose_32_blocks(scale):
    """Exact composition at the 32K workload's depth and width (K = 32 chained
    products, dk = dv = 128) on O(1)-norm transitions (scale x orthogonal), so
    every block contributes; shorter requests (K = 16, 8, 4, 2) reuse pool rows
    in other orders.  The error per K is printed for the design notes."""
    rng = np.random.default_rng(3200)
    n_blk, h, d = 40, 4, 128
    B = rng.standard_normal((n_blk, h, d, d)).astype(np.float32)
    M = _orth_pool(rng, n_blk, h, d, scale).astype(np.float32)
    Ks = [32, 16, 8, 4, 2]
    ids = np.concatenate([rng.permutation(n_blk)[:k] for k in Ks]).astype(np.int32)
    blk_cu = np.concatenate([[0], np.cumsum(Ks)]).astype(np.int32)
    layer = lkv.make_layer(I.GDN, 1, h, d, d, 64)
    S = torch.empty((len(Ks), h, d, d), device="cuda")
    lkv.init_compose(layer, n_blk, _dev(B), _dev(M), torch.from_numpy(ids).cuda(),
                     torch.from_numpy(blk_cu).cuda(), len(ids), S)
    torch.cuda.synchronize()
    import oracle
    ref = oracle.compose_gdn(blk_cu, ids, B, M)
    got = _np(S)
    errs = {k: rel_slices(got[[r]], ref[[r]]) for r, k in enumerate(Ks)}
    print(f"compose K-chain error at scale {scale}: " + ", ".join(f"K={k} {e:.2e}" for k, e in errs.items()))
    assert max(errs.values()) < STATE_TOL, errs


@pytest.mark.parametrize("nb", [1, 2, 4, 8])
@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_dv512_pinned_geometry(fam, nb, monkeypatch):
    """The largest state (dk = 128, dv = 512) in every launch geometry the chunk
    kernels have: 16 nb state rows per workgroup (nb = 8: four waves of two row
    tiles, block summaries only), i.e. 32 / nb row tiles per head; the scan takes
    nb up to 4 (eight row tiles per head at dv = 512)."""
    case = GDN_CASES[-1] if fam == I.GDN else SSD_CASES[-1]
    w = _work(fam, case)
    G = gpu_io.GpuWorkload(w)
    monkeypatch.setenv("LKV_SCAN_NB", str(nb))
    G.block_summary()
    torch.cuda.synchronize()
    B, M = R.summaries(w)
    assert rel_slices(_np(G.B_pool), B) < STATE_TOL
    if fam == I.GDN:
        assert rel_slices(_np(G.M_pool), M) < STATE_TOL
    else:
        assert np.max(np.abs(_np(G.M_pool) - M) / np.maximum(np.abs(M), 1e-30)) < STATE_TOL
    monkeypatch.setenv("LKV_SCAN_NB", str(min(nb, 4)))
    S0 = R.init_compose(w, B, M)
    _scan_check(w, gpu_io.GpuWorkload(w, with_cached=False), S0)


def test_fold_view_keeps_blocks_reused_later():
    """Position-independent caching reuses a cached block in any position: a
    block that is one request's first block and a later block of another keeps
    its transition in the fold over blocks 2..K; only blocks whose transition
    no request reads are emptied.  The composed states match the oracle."""
    import dataclasses
    w = _work(I.GDN, (64, 64, 64, "bf16", 2, 2, ((70, 90, 40), (130, 20)), (64, 80)))
    # pool rows 0..4; request 0 = [0, 1, 2], request 1 = [3, 4], request 2 = [2, 0, 4]
    ids = np.array([0, 1, 2, 3, 4, 2, 0, 4], np.int32)
    blk_cu = np.array([0, 3, 5, 8], np.int32)
    w = dataclasses.replace(w, blk_ids=ids, blk_cu=blk_cu, last_blk=np.array([2, 4, 4], np.int32),
                            online=w.online.__class__(np.array([0, 64, 100, 144], np.int32),
                                                      *[None if a is None else a[:144] for a in
                                                        (w.online.q, w.online.k, w.online.v, w.online.g,
                                                         w.online.beta)]))
    assert gpu_io.fold_dropped_blocks(w) == [3]
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=False)
    G.fold_transitions()
    G.init_compose()
    torch.cuda.synchronize()
    B, M = R.summaries(w)
    got_M = _np(G.M_pool)
    assert rel_slices(got_M[[0, 1, 2, 4]], M[[0, 1, 2, 4]]) < STATE_TOL
    assert np.array_equal(got_M[3], np.broadcast_to(np.eye(64, dtype=np.float32), got_M[3].shape))
    assert rel_slices(_np(G.S_exact), R.init_compose(w, B, M)) < STATE_TOL


@pytest.mark.parametrize("x_mu", [-3.0, 0.0], ids=["rescale-every-few-chunks", "rescale-every-chunk"])
def test_gdn_state_rescale(x_mu):
    """The state waves hold S / e^lam and rescale once lam would drop below
    -32 (the chunk decays of Eq. 3 moved into the gate rows).  With log-decays
    of about -5 per 64-token chunk the rescale comes about every seventh chunk
    (once in each 12-chunk block, twice in the 15-chunk online stream) and the
    blocks' transitions stay near e^-60, inside fp32's range; with about -50
    per chunk it comes in every chunk.  Summaries and the scan are checked
    against the oracle; at -50 per chunk a block's transition (about e^-600)
    is below fp32's range, so only its state, the outputs and the final state
    are compared."""
    layer = I.Layer(I.GDN, 1, 2, 128, 128, 64, "bf16", "bf16")
    w = I.build_workload(f"rescale{x_mu}", layer, [[768, 700]], [900], I.GateLaw(x_mu=x_mu, beta_mu=0.0), 31,
                         scale=0.75)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    torch.cuda.synchronize()
    B, M = R.summaries(w)
    assert rel_slices(_np(G.B_pool), B) < STATE_TOL
    if x_mu < -1.0:
        assert rel_slices(_np(G.M_pool), M) < STATE_TOL
    _scan_check(w, G, R.init_compose(w, B, M))
