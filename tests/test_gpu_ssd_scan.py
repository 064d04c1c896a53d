"""The Mamba-2 scan kernel (four symmetric state waves) against the shared chunk
kernel, which computes the same chunkwise form (Eq. 2 decay, Eq. 5 state
passing) with the same products in the same order: scans, block summaries
(B and Lambda), starts from a pool row (fp32 and bf16), and the sequence-
parallel form must agree bit for bit.  Parity with the oracle is in
test_gpu_parity.py; this pins the two GPU paths to each other on every mode.
"""
import os

import numpy as np
import pytest

from paper_2608_11231_amd import inputs as I

import oracle_ref as R
from oracle_ref import max_abs, rel_slices

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_11231_amd import gpu_io, lkv  # noqa: E402

CASES = [
    # (N, P, G, H, blocks, online)
    (128, 64, 1, 4, ((130, 64), (1, 70)), (150, 64)),
    (32, 64, 2, 4, ((100, 0, 65),), (129,)),
    (64, 128, 1, 2, ((64, 128), (3,)), (0, 191)),
    (128, 192, 1, 2, ((65,), (200,), (7,)), (63, 1, 256)),
]


def _work(case, seed=23):
    dk, dv, hq, hv, blocks, online = case
    layer = I.Layer(I.SSD, hq, hv, dk, dv, 64, "bf16", "f32")
    law = I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0, a_hi=4.0)
    return I.build_workload(f"ssd{case[:4]}", layer, [list(b) for b in blocks], list(online), law, seed)


class _ChunkKernel:
    """Selects the shared chunk kernel for Mamba-2 while active (read per call);
    outside it, the tests select ssd_scan_kernel."""

    def __enter__(self):
        os.environ.pop("LKV_SSD_SCAN_KERNEL", None)

    def __exit__(self, *exc):
        os.environ["LKV_SSD_SCAN_KERNEL"] = "1"


@pytest.fixture(autouse=True)
def _scan_kernel():
    os.environ["LKV_SSD_SCAN_KERNEL"] = "1"
    yield
    os.environ.pop("LKV_SSD_SCAN_KERNEL", None)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _same(a, b):
    """bit-identical, NaN payloads aside (NaN where the other is NaN)"""
    torch.cuda.synchronize()
    na, nb = a.isnan(), b.isnan()
    if not torch.equal(na, nb):
        return False
    return torch.equal(_bits(a.masked_fill(na, 0)), _bits(b.masked_fill(nb, 0)))


@pytest.mark.parametrize("case", CASES, ids=[f"ssd{c[:4]}" for c in CASES])
def test_scan_matches_chunk_kernel(case):
    w = _work(case)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    rng = np.random.default_rng(4)
    S0 = torch.from_numpy((0.5 * rng.standard_normal(tuple(G.S_final.shape))).astype(np.float32)).cuda()
    G.scan(S0)
    out, S = G.out.clone(), G.S_final.clone()
    with _ChunkKernel():
        G.scan(S0)
    assert _same(out, G.out) and _same(S, G.S_final)
    # and the oracle, at the parity bars
    o_ref, S_ref = R.scan(w, S0.cpu().numpy())
    assert rel_slices(S.cpu().numpy(), S_ref) < 1e-4
    assert max_abs(out.float().cpu().numpy(), o_ref) < 2e-2


@pytest.mark.parametrize("case", CASES, ids=[f"ssd{c[:4]}" for c in CASES])
def test_block_summary_matches_chunk_kernel(case):
    w = _work(case)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    B, M = G.B_pool.clone(), G.M_pool.clone()
    with _ChunkKernel():
        G.block_summary()
    assert _same(B, G.B_pool) and _same(M, G.M_pool)
    # B only, then Lambda only
    G.B_pool.zero_()
    G.block_summary(M=False)
    assert _same(B, G.B_pool)
    G.M_pool.zero_()
    G.block_summary(B=False)
    torch.cuda.synchronize()
    B_ref, L_ref = R.summaries(w)
    assert rel_slices(B.cpu().numpy(), B_ref) < 1e-4
    assert np.max(np.abs(G.M_pool.cpu().numpy() - L_ref) / np.maximum(np.abs(L_ref), 1e-30)) < 1e-4


@pytest.mark.parametrize("bf16_pool", [False, True])
def test_scan_from_pool_matches_chunk_kernel(bf16_pool):
    w = _work(CASES[3])
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    pool = G.B_pool.to(torch.bfloat16) if bf16_pool else G.B_pool
    # a cached row, the zero state (-1) and an id outside the pool (NaN state)
    assert w.n_req == 3
    src = torch.tensor([w.n_blk - 1, -1, w.n_blk + 5], dtype=torch.int32, device="cuda")
    lkv.chunk_scan_from_pool(G.layer, G.online.struct, 1.0, pool, w.n_blk, src, G.out, G.S_final)
    out, S = G.out.clone(), G.S_final.clone()
    with _ChunkKernel():
        lkv.chunk_scan_from_pool(G.layer, G.online.struct, 1.0, pool, w.n_blk, src, G.out, G.S_final)
    assert _same(out, G.out) and _same(S, G.S_final)
    assert torch.isfinite(S[:2]).all() and S[2].isnan().all()


@pytest.mark.parametrize("pieces", [2, 4])
def test_sequence_parallel_matches_chunk_kernel(pieces, monkeypatch):
    """The summary / composition / rescan form of the sequence-parallel scan,
    on either kernel."""
    monkeypatch.setenv("LKV_SSD_SP_CORRECT", "0")
    w = _work(CASES[3])
    G = gpu_io.GpuWorkload(w, with_cached=False)
    rng = np.random.default_rng(9)
    S0 = torch.from_numpy((0.5 * rng.standard_normal(tuple(G.S_final.shape))).astype(np.float32)).cuda()
    G.scan(S0, pieces=pieces)
    out, S = G.out.clone(), G.S_final.clone()
    with _ChunkKernel():
        G.scan(S0, pieces=pieces)
    assert _same(out, G.out) and _same(S, G.S_final)
    o_ref, S_ref = R.scan(w, S0.cpu().numpy())
    assert rel_slices(S.cpu().numpy(), S_ref) < 1e-4
    assert max_abs(out.float().cpu().numpy(), o_ref) < 2e-2


SP_CASES = [
    # (N, P, G, H, online lengths): ragged, empty, one-token and chunk-multiple requests
    (128, 64, 1, 4, (450, 63, 0, 200)),
    (64, 128, 2, 4, (333, 64, 1, 640)),
    (32, 192, 1, 2, (1000,)),
]


@pytest.mark.parametrize("with_out", [True, False])
@pytest.mark.parametrize("with_init", [True, False])
@pytest.mark.parametrize("pieces", [2, 3, 4, 8])
@pytest.mark.parametrize("case", SP_CASES, ids=[f"ssd{c[:4]}" for c in SP_CASES])
def test_sequence_parallel_correction(case, pieces, with_init, with_out):
    """The one-pass form: pieces scanned once (piece 0 from the initial state,
    the rest from zero), outputs corrected by exp(L_t) C_t S_p^T, final state
    composed.  Checked against the oracle and against the rescan form."""
    dk, dv, hq, hv, online = case
    layer = I.Layer(I.SSD, hq, hv, dk, dv, 64, "bf16", "f32")
    law = I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0, a_hi=4.0)
    w = I.build_workload("sp", layer, [[] for _ in online], list(online), law, 7)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    rng = np.random.default_rng(3)
    S0_np = (0.5 * rng.standard_normal(tuple(G.S_final.shape))).astype(np.float32) if with_init else None
    S0 = torch.from_numpy(S0_np).cuda() if with_init else None
    o_ref, S_ref = R.scan(w, S0_np)
    G.out.fill_(7.0)
    ws = torch.empty(lkv.chunk_scan_sp_workspace(G.layer, w.n_req, pieces), dtype=torch.uint8, device="cuda")
    lkv.chunk_scan_sp(G.layer, G.online.struct, 1.0, S0, G.out if with_out else None, G.S_final, pieces, ws)
    torch.cuda.synchronize()
    assert rel_slices(G.S_final.cpu().numpy(), S_ref) < 1e-4
    if with_out:
        assert max_abs(G.out.float().cpu().numpy(), o_ref) < 2e-2
        out = G.out.clone()
        os.environ["LKV_SSD_SP_CORRECT"] = "0"
        try:
            G.scan(S0, pieces=pieces)
        finally:
            os.environ.pop("LKV_SSD_SP_CORRECT", None)
        torch.cuda.synchronize()
        assert (out.float() - G.out.float()).abs().max().item() < 2e-2
    else:
        assert bool((G.out == 7.0).all())  # no outputs written
