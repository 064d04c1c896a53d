"""GPU parity of the sequence-parallel chunk scan (lkv_chunk_scan_sp) against the
CPU oracle: each request's stream cut into pieces, the pieces' (transition,
state) pairs composed (Eq. 5 applied piece after piece, Eq. 6) into start
states, every piece scanned from its start.  Same bars as the serial scan:
fp32 states within 1e-4 normwise relative error per (request, head) slice,
bf16 outputs within 2e-2 absolute, fp32-io outputs within 1e-4 relative."""
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


def _work(fam, dk, dv, chunk, io, hq, hv, online, seed=5):
    layer = I.Layer(fam, hq, hv, dk, dv, chunk, io, io if fam == I.GDN else "f32")
    law = I.GateLaw(x_mu=-3.0, beta_mu=0.0) if fam == I.GDN else I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0,
                                                                             a_hi=4.0)
    return I.build_workload("sp", layer, [[] for _ in online], list(online), law, seed,
                            scale=0.75 if fam == I.GDN else 1.0)


CASES = [
    # (family, dk, dv, chunk, io, h_qk, h_v, online lengths)
    (I.GDN, 64, 64, 64, "bf16", 2, 2, (300, 0, 64, 129, 5)),
    (I.GDN, 128, 128, 64, "bf16", 1, 2, (700, 191)),
    (I.GDN, 32, 32, 16, "bf16", 2, 4, (97, 40, 0)),
    (I.GDN, 16, 16, 16, "f32", 1, 1, (130, 17)),
    (I.SSD, 128, 64, 64, "bf16", 1, 4, (450, 63, 0, 200)),
    (I.SSD, 64, 32, 16, "bf16", 2, 4, (77, 160)),
    (I.SSD, 16, 16, 16, "f32", 1, 2, (90,)),
]


@pytest.mark.parametrize("pieces", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("case", CASES, ids=[f"{'gdn' if c[0] == I.GDN else 'ssd'}{c[1:5]}" for c in CASES])
@pytest.mark.parametrize("with_init", [False, True])
def test_sp_scan_matches_oracle(case, pieces, with_init):
    fam, dk, dv, chunk, io, hq, hv, online = case
    w = _work(fam, dk, dv, chunk, io, hq, hv, online)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    S0 = None
    if with_init:
        S0 = (0.3 * np.random.default_rng(9).standard_normal(tuple(G.S_final.shape))).astype(np.float32)
    o_ref, S_ref = R.scan(w, S0)
    G.out.fill_(float("nan"))
    G.S_final.fill_(float("nan"))
    G.scan(None if S0 is None else _dev(S0), pieces=pieces)
    torch.cuda.synchronize()
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    if io == "f32":
        assert rel_slices(_np(G.out)[None], o_ref[None], lead=1) < STATE_TOL
    else:
        assert max_abs(_np(G.out), o_ref) < OUT_ABS


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_sp_state_only_and_null_final(fam):
    """Outputs NULL: only the pieces' pairs and the composition run; S_final NULL:
    the final state goes to the workspace and the outputs still match."""
    case = CASES[0] if fam == I.GDN else CASES[4]
    w = _work(*case)
    G = gpu_io.GpuWorkload(w, with_cached=False)
    o_ref, S_ref = R.scan(w, None)
    ws = torch.empty(lkv.chunk_scan_sp_workspace(G.layer, w.n_req, 4), dtype=torch.uint8, device="cuda")
    lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, None, None, G.S_final, 4, ws)
    lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, None, G.out, None, 4, ws)
    torch.cuda.synchronize()
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    assert max_abs(_np(G.out), o_ref) < OUT_ABS


def test_sp_rejects_small_or_misaligned_workspace():
    w = _work(*CASES[0])
    G = gpu_io.GpuWorkload(w, with_cached=False)
    need = lkv.chunk_scan_sp_workspace(G.layer, w.n_req, 3)
    ws = torch.empty(need + 512, dtype=torch.uint8, device="cuda")
    with pytest.raises(lkv.LkvError, match="SHAPE"):
        lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, None, G.out, G.S_final, 3, ws[:need - 256])
    with pytest.raises(lkv.LkvError, match="ALIGN"):
        lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, None, G.out, G.S_final, 3, ws[16:])
    with pytest.raises(lkv.LkvError, match="SHAPE"):
        lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, None, G.out, G.S_final, 0, ws)


@pytest.mark.parametrize("index,pieces", [(1, 4), (1, 8), (2, 4), (2, 8), (2, 12)])
def test_sp_full_size_8k(index, pieces):
    """The 8K workloads (one request) in the piece count the benchmark uses
    (gpu_io.sp_pieces: 4) and others, against the oracle on every head, from the
    exact-composition initial state."""
    w = I.config(index, workers=16)
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=False)
    G.fold_transitions()
    G.init_compose()
    G.scan(G.S_exact, pieces=pieces)
    torch.cuda.synchronize()
    SX = _np(G.S_exact).astype(np.float64)
    o_ref, S_ref = R.scan(w, SX)
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    assert max_abs(_np(G.out), o_ref) < OUT_ABS
