"""GPU parity of the bf16 cached-state pool: rounding to bf16 (bit-exact against
the oracle's round-to-nearest-even), the bf16-pool initialisations (exact
widening; composition within 1e-4), host-to-device staging of cache rows
(bit-exact), and the staged serving flow end to end."""
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


def _u32(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def _round_on_gpu(x):
    src = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    dst = torch.empty(src.shape, dtype=torch.bfloat16, device="cuda")
    lkv.round_bf16(src, dst)
    torch.cuda.synchronize()
    return dst.float().cpu().numpy()


def test_round_bf16_bit_exact():
    rng = np.random.default_rng(1)
    n = 100003                                   # not a multiple of 8: the tail path runs too
    x = (rng.standard_normal(n) * np.exp(rng.uniform(-60, 60, n))).astype(np.float32)
    special = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.3895314e38, 3.3961776e38, 3.4e38,
                        -3.4e38, np.inf, -np.inf, 0.0, -0.0, np.nan], np.float32)
    x[:len(special)] = special
    got = _round_on_gpu(x)
    want = oracle.round_bf16(x)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)            # NaN stays NaN (payload not compared)
    assert np.array_equal(_u32(got)[~nan], _u32(want)[~nan])


def test_round_bf16_subnormals():
    """fp32 subnormals round like any other value (bf16 shares fp32's exponent range)."""
    x = np.array([2 ** -133, 3 * 2 ** -134, 2 ** -149, 5 * 2 ** -140, -7 * 2 ** -138, 1.1754942e-38],
                 np.float32)
    assert np.array_equal(_u32(_round_on_gpu(x)), _u32(oracle.round_bf16(x)))


def _bf16_pool(rng, shape):
    return I.to_storage(rng.standard_normal(shape), "bf16")     # fp32 arrays holding bf16 values


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_init_single_bf16_exact_widening(fam):
    rng = np.random.default_rng(2)
    n_blk, h, dv, dk = 6, 3, 32, 64
    pool = _bf16_pool(rng, (n_blk, h, dv, dk))
    layer = lkv.make_layer(fam, 1, h, dk, dv, 64, gate_dtype=torch.float32)
    src = np.array([5, -1, 0, 9, 2], np.int32)
    S = torch.empty((len(src), h, dv, dk), device="cuda")
    lkv.init_single_bf16(layer, n_blk, torch.from_numpy(pool).to("cuda", torch.bfloat16),
                         torch.from_numpy(src).cuda(), S)
    torch.cuda.synchronize()
    got = S.cpu().numpy()
    want = oracle.init_single(pool, np.where(src < n_blk, src, -1))
    for r, b in enumerate(src):
        if b < n_blk:
            assert np.array_equal(_u32(got[r]), _u32(want[r].astype(np.float32)))
        else:
            assert np.isnan(got[r]).all()


@pytest.mark.parametrize("dk,dv", [(16, 16), (64, 48), (128, 128)])
def test_init_compose_bf16_gdn(dk, dv):
    rng = np.random.default_rng(dk)
    n_blk, h = 7, 2
    B = _bf16_pool(rng, (n_blk, h, dv, dk))
    q, _ = np.linalg.qr(rng.standard_normal((n_blk * h, dk, dk)))
    M = (0.9 * q).reshape(n_blk, h, dk, dk).astype(np.float32)
    blk_cu = np.array([0, 4, 4, 5, 7], np.int32)
    ids = np.array([3, 0, 6, 1, 2, 5, 4], np.int32)
    layer = lkv.make_layer(I.GDN, 1, h, dk, dv, 64)
    S = torch.empty((4, h, dv, dk), device="cuda")
    lkv.init_compose_bf16(layer, n_blk, torch.from_numpy(B).to("cuda", torch.bfloat16), torch.from_numpy(M).cuda(),
                          torch.from_numpy(ids).cuda(), torch.from_numpy(blk_cu).cuda(), len(ids), S)
    torch.cuda.synchronize()
    ref = oracle.compose_gdn(blk_cu, ids, B, M)
    got = S.cpu().numpy()
    assert rel_slices(got[[0, 3]], ref[[0, 3]]) < STATE_TOL
    assert np.array_equal(got[1], np.zeros_like(got[1]))
    assert np.array_equal(_u32(got[2]), _u32(B[2]))     # K = 1: the widened cached state


def test_init_compose_bf16_ssd():
    rng = np.random.default_rng(3)
    n_blk, H, P, N = 5, 4, 32, 64
    B = _bf16_pool(rng, (n_blk, H, P, N))
    Lam = (-rng.uniform(0.0, 2.0, (n_blk, H))).astype(np.float32)
    blk_cu = np.array([0, 3, 5], np.int32)
    ids = np.array([4, 0, 2, 1, 3], np.int32)
    layer = lkv.make_layer(I.SSD, 1, H, N, P, 64, gate_dtype=torch.float32)
    S = torch.empty((2, H, P, N), device="cuda")
    lkv.init_compose_bf16(layer, n_blk, torch.from_numpy(B).to("cuda", torch.bfloat16), torch.from_numpy(Lam).cuda(),
                          torch.from_numpy(ids).cuda(), torch.from_numpy(blk_cu).cuda(), len(ids), S)
    torch.cuda.synchronize()
    assert rel_slices(S.cpu().numpy(), oracle.compose_ssd(blk_cu, ids, B, Lam)) < STATE_TOL


def test_stage_rows_bit_exact_on_a_side_stream():
    rng = np.random.default_rng(4)
    pool = torch.empty((12, 3, 16, 32), dtype=torch.bfloat16, pin_memory=True)
    pool.copy_(torch.from_numpy(_bf16_pool(rng, (12, 3, 16, 32))))
    rows = np.array([5, 6, 7, 2, 2, 11, 0], np.int32)           # runs, a repeat, the last row
    dst = torch.full((len(rows), 3, 16, 32), 7.0, device="cuda", dtype=torch.bfloat16)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    lkv.stage_rows(dst, pool, rows, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    S = torch.empty((len(rows), 3, 16, 32), device="cuda")
    layer = lkv.make_layer(I.GDN, 1, 3, 32, 16, 64)
    lkv.init_single_bf16(layer, len(rows), dst, torch.arange(len(rows), dtype=torch.int32, device="cuda"), S)
    torch.cuda.synchronize()
    want = pool.float().numpy()[rows]
    assert np.array_equal(_u32(dst.float().cpu().numpy()), _u32(want))
    assert np.array_equal(_u32(S.cpu().numpy()), _u32(want))
    with pytest.raises(ValueError):
        lkv.stage_rows(dst, pool, np.array([12], np.int32))


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_staged_serving_flow(fam):
    """The cache as stored (oracle block states rounded to bf16 by the oracle, plus the
    cached key/gate streams) in pinned host memory; a batch that uses a subset of the
    blocks stages its rows, folds its transitions, composes and scans.  Both
    initialisations are checked against the oracle fed the same bf16 states."""
    dk, dv = (64, 64) if fam == I.GDN else (64, 32)
    w = I.small(fam, n_req=2, dk=dk, dv=dv, chunk=64, blocks=((40, 23, 70, 17, 33, 90), (30,)),
                online=(37, 70), h_qk=2 if fam == I.GDN else 1, h_v=4)
    c = w.cached
    if fam == I.GDN:
        _, B = oracle.gdn_scan(c.cu, None, c.k, c.v, c.g, c.beta, want_o=False)
        M = oracle.gdn_transition(c.cu, c.k, c.g, c.beta)
    else:
        _, B = oracle.ssd_scan(c.cu, None, c.k, c.v, c.g, w.A, want_y=False)
        M = oracle.ssd_log_decay(c.cu, c.g, w.A)
    Bq = oracle.round_bf16(B.astype(np.float32))
    hc = gpu_io.HostCache(w, Bq)
    # the batch: request 0 uses blocks 4, 1, 6 (in that context order), request 1 uses 3
    blk_ids = np.array([4, 1, 6, 3], np.int32)
    blk_cu = np.array([0, 3, 4], np.int32)
    last = np.array([6, 3], np.int32)
    sb = gpu_io.StagedBatch(hc, blk_ids, blk_cu, last)
    assert sb.rows.tolist() == [1, 3, 4, 6]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    sb.stage_single(side)
    sb.stage_exact(side)
    torch.cuda.current_stream().wait_stream(side)
    S1 = torch.empty((2, 4, dv, dk), device="cuda")
    SX = torch.empty_like(S1)
    sb.init_single(S1)
    sb.init_compose(SX)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    G.scan(SX)
    torch.cuda.synchronize()
    assert np.array_equal(_u32(S1.cpu().numpy()), _u32(Bq[last]))
    if fam == I.GDN:
        SX_ref = oracle.compose_gdn(blk_cu, blk_ids, Bq, M)
    else:
        SX_ref = oracle.compose_ssd(blk_cu, blk_ids, Bq, M)
    assert rel_slices(SX.cpu().numpy(), SX_ref) < STATE_TOL
    o = w.online
    if fam == I.GDN:
        o_ref, SF_ref = oracle.gdn_scan(o.cu, o.q, o.k, o.v, o.g, o.beta, scale=w.scale, S0=SX_ref)
    else:
        o_ref, SF_ref = oracle.ssd_scan(o.cu, o.q, o.k, o.v, o.g, w.A, S0=SX_ref)
    assert rel_slices(G.S_final.cpu().numpy(), SF_ref) < STATE_TOL
    assert max_abs(G.out.float().cpu().numpy(), o_ref) < OUT_ABS
