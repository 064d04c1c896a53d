"""GPU parity of the selected-position gather (bit-exact against the oracle's
row-by-row definition) and of the scan over the gathered stream; the
random-block single-source initial state is a bit-exact pool row."""
import numpy as np
import pytest

from paper_2608_11231_amd import inputs as I

from oracle_ref import max_abs, rel_slices
import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_11231_amd import gpu_io, lkv  # noqa: E402

STATE_TOL = 1e-4
OUT_ABS = 2e-2


def _bits(t):
    """uint32 bit patterns of a device tensor widened to fp32 (bf16 widening is exact)."""
    return t.detach().float().cpu().numpy().view(np.uint32)


def _context(fam, dk, dv, io, hq, hv, ctx_lens, seed=31):
    layer = I.Layer(fam, hq, hv, dk, dv, 64, io, io if fam == I.GDN else "f32")
    law = I.GateLaw(x_mu=-3.0, beta_mu=0.0) if fam == I.GDN else I.GateLaw(dt_mu=-3.0, dt_bias=-1.0,
                                                                             a_lo=1.0, a_hi=4.0)
    # the context streams are drawn as the "online" streams of a workload without cached blocks
    return I.build_workload("ctx", layer, [[] for _ in ctx_lens], list(ctx_lens), law, seed,
                            scale=0.75 if fam == I.GDN else 1.0)


def _selection(ctx_lens, seed):
    rng = np.random.default_rng(seed)
    per = []
    for r, n in enumerate(ctx_lens):
        kind = r % 4
        if kind == 0:
            per.append(I.select_uniform(rng, n, 0.2))
        elif kind == 1:
            cuts = sorted(rng.choice(np.arange(1, n), size=3, replace=False)) if n > 3 else []
            lens = np.diff([0, *cuts, n])
            per.append(I.select_seams(lens, 8))
        elif kind == 2:
            per.append(np.arange(n, dtype=np.int32))
        else:
            per.append(np.zeros(0, np.int32))
    return per


CASES = [
    # (family, dk, dv, io, h_qk, h_v, context lengths)
    (I.GDN, 32, 48, "bf16", 2, 4, (130, 77, 300, 50, 0, 64)),
    (I.GDN, 16, 16, "f32", 1, 1, (33, 20, 5, 9)),
    (I.SSD, 64, 32, "bf16", 2, 4, (150, 41, 90, 12)),
    # more requests than a workgroup has threads: the request search takes two
    # passes and reads the offsets past the first 256 from global memory
    (I.GDN, 16, 16, "bf16", 1, 2, tuple((7 * r + 3) % 13 for r in range(300))),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{'gdn' if c[0] == I.GDN else 'ssd'}{c[1:6]}" for c in CASES])
def test_gather_bit_exact(case):
    fam, dk, dv, io, hq, hv, ctx_lens = case
    w = _context(fam, dk, dv, io, hq, hv, ctx_lens)
    per = _selection(ctx_lens, seed=len(ctx_lens))
    # out-of-range positions give NaN rows: one past the end, one negative, one in an empty context
    per[1] = np.concatenate([per[1], [ctx_lens[1], -1]]).astype(np.int32)
    if 0 in ctx_lens:
        per[ctx_lens.index(0)] = np.array([0], np.int32)
    sel_cu, pos = I.pack_selection(per)
    ctx = gpu_io.GpuTokens(w.online, w.layer, w.A)
    sel = gpu_io.GpuSelection(ctx, w.online.cu, sel_cu, pos, w.layer)
    sel.gather()
    torch.cuda.synchronize()
    o = w.online
    ref = oracle.gather_selected(o.cu, sel_cu, pos, o.q, o.k, o.v, o.g, o.beta)
    for name, got, want in zip("q k v g beta".split(), (sel.q, sel.k, sel.v, sel.g, sel.beta), ref):
        if want is None:
            assert got is None
            continue
        assert np.array_equal(_bits(got), want.astype(np.float32).view(np.uint32)), name
    assert np.isnan(ref[1][oracle.gather_rows(o.cu, sel_cu, pos) < 0]).all()


def test_gather_subset_of_arrays_leaves_the_rest():
    w = _context(I.GDN, 32, 32, "bf16", 1, 2, (40, 60))
    sel_cu, pos = I.pack_selection(_selection((40, 60), 1))
    ctx = gpu_io.GpuTokens(w.online, w.layer, w.A)
    sel = gpu_io.GpuSelection(ctx, w.online.cu, sel_cu, pos, w.layer)
    sel.q.fill_(3.0)
    lkv.gather_selected(sel.layer, sel.ctx_struct, sel.pos, sel.sel_cu, sel.n_sel, None, sel.k, None,
                        None, None)
    torch.cuda.synchronize()
    assert bool((sel.q == 3.0).all())
    (k,) = oracle.gather_selected(w.online.cu, sel_cu, pos, w.online.k)
    assert np.array_equal(_bits(sel.k), k.view(np.uint32))


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_scan_over_gathered_stream(fam):
    """GPU gather then GPU chunk scan from a random state equal the oracle scan over
    the oracle's gathered stream (Alg. 1's recompute over U only)."""
    ctx_lens = (700, 260, 1000)
    dk, dv = (128, 128) if fam == I.GDN else (128, 64)
    w = _context(fam, dk, dv, "bf16", 2 if fam == I.GDN else 1, 4, ctx_lens, seed=8)
    rng = np.random.default_rng(8)
    per = [I.select_uniform(rng, 700, 0.25), I.select_seams([100, 60, 100], 16),
           I.select_uniform(rng, 1000, 0.2)]
    sel_cu, pos = I.pack_selection(per)
    ctx = gpu_io.GpuTokens(w.online, w.layer, w.A)
    sel = gpu_io.GpuSelection(ctx, w.online.cu, sel_cu, pos, w.layer)
    S0 = (0.3 * rng.standard_normal((3, 4, dv, dk))).astype(np.float32)
    S = torch.from_numpy(S0).cuda()
    out = torch.empty((sel.n_sel, 4, dv), device="cuda", dtype=torch.bfloat16)
    sel.gather()
    if fam == I.GDN:
        lkv.gdn_chunk_scan(sel.layer, sel.struct, w.scale, S, out, S)
    else:
        lkv.ssd_chunk_scan(sel.layer, sel.struct, S, out, S)
    torch.cuda.synchronize()
    o = w.online
    q, k, v, g, beta = oracle.gather_selected(o.cu, sel_cu, pos, o.q, o.k, o.v, o.g, o.beta)
    if fam == I.GDN:
        o_ref, S_ref = oracle.gdn_scan(sel_cu, q, k, v, g, beta, scale=w.scale, S0=S0)
    else:
        o_ref, S_ref = oracle.ssd_scan(sel_cu, q, k, v, g, w.A, S0=S0)
    assert rel_slices(S.cpu().numpy(), S_ref) < STATE_TOL
    assert max_abs(out.float().cpu().numpy(), o_ref) < OUT_ABS


def test_gather_full_size_random_bits():
    """The 32K-context workload's shape (4 requests x 32768 context tokens, 32 heads,
    d = 128, bf16) with a 1/8 budget, 4096 positions per request: the launch the
    benchmark times.  Random bit patterns (NaN payloads included) must come
    through unchanged."""
    n_req, n_ctx, h, d = 4, 32768, 32, 128
    layer = I.Layer(I.GDN, h, h, d, d, 64)
    gen = torch.Generator(device="cuda").manual_seed(5)

    def bits(*shape):
        return torch.randint(-32768, 32768, shape, device="cuda", dtype=torch.int32,
                             generator=gen).to(torch.int16).view(torch.bfloat16)
    N = n_req * n_ctx
    ctx_cu = (np.arange(n_req + 1) * n_ctx).astype(np.int32)
    cu_dev = torch.from_numpy(ctx_cu).cuda()
    arrs = dict(q=bits(N, h, d), k=bits(N, h, d), v=bits(N, h, d), g=bits(N, h), beta=bits(N, h))
    rng = np.random.default_rng(12)
    sel_cu, pos = I.pack_selection([I.select_uniform(rng, n_ctx, 0.125) for _ in range(n_req)])
    assert sel_cu[-1] == n_req * 4096
    L = gpu_io.layer_struct(layer)
    ctx = lkv.make_tokens(cu_dev, N, arrs["q"], arrs["k"], arrs["v"], arrs["g"], arrs["beta"])
    outs = {k: torch.empty((int(sel_cu[-1]),) + tuple(x.shape[1:]), device="cuda", dtype=x.dtype)
            for k, x in arrs.items()}
    lkv.gather_selected(L, ctx, torch.from_numpy(pos).cuda(), torch.from_numpy(sel_cu).cuda(), int(sel_cu[-1]),
                        outs["q"], outs["k"], outs["v"], outs["g"], outs["beta"])
    torch.cuda.synchronize()
    for name, x in arrs.items():
        (want,) = oracle.gather_selected(ctx_cu, sel_cu, pos, x.view(torch.int16).cpu().numpy())
        assert np.array_equal(outs[name].view(torch.int16).cpu().numpy(), want), name


def test_random_block_single_source():
    """App. A's random-block initialiser: each request starts from one uniformly
    drawn matched block's cached state, a bit-exact pool row."""
    w = I.small(I.GDN, n_req=2, blocks=((40, 23, 17), (30, 50)), online=(37, 70))
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=False)
    src = I.random_block_src(np.random.default_rng(4), w)
    S = torch.empty_like(G.S_single)
    lkv.init_single(G.layer, w.n_blk, G.B_pool, torch.from_numpy(src).cuda(), S)
    torch.cuda.synchronize()
    pool = G.B_pool.cpu().numpy()
    got = S.cpu().numpy()
    for r, b in enumerate(src):
        assert w.blk_cu[r] <= np.nonzero(w.blk_ids == b)[0][0] < w.blk_cu[r + 1]
        assert np.array_equal(got[r].view(np.uint32), pool[b].view(np.uint32))
    c = w.cached
    sl = slice(int(c.cu[src[0]]), int(c.cu[src[0] + 1]))
    _, B = oracle.gdn_scan(np.array([0, sl.stop - sl.start], np.int32), None, c.k[sl], c.v[sl], c.g[sl],
                           c.beta[sl], want_o=False)
    assert rel_slices(got[0][None], B) < STATE_TOL
