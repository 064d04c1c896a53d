"""GPU parity of the relative-error diagnostic, of the Eq. 7 mismatch recursion
as the library's composition realises it, and of the layer-0 probe (exact
composition reproduces the full-prefix state; the single block misses the
earlier blocks' share)."""
import numpy as np
import pytest

from paper_2608_11231_amd import inputs as I

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_11231_amd import gpu_io, lkv  # noqa: E402


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def test_rel_error_parity():
    rng = np.random.default_rng(0)
    R = rng.standard_normal((3, 5, 64, 48)).astype(np.float32)
    S = (R + 0.1 * rng.standard_normal(R.shape)).astype(np.float32)
    S[0, 0] = R[0, 0]                 # exact slice
    R[2, 4] = 0.0                     # zero reference: inf
    sq, rel, rg = lkv.state_rel_error(_dev(S), _dev(R), group=5)
    torch.cuda.synchronize()
    want, want_g = oracle.rel_error(S, R, group=5)
    got = rel.cpu().numpy()
    fin = np.isfinite(want)
    assert np.array_equal(np.isinf(got), np.isinf(want))
    assert np.all(np.abs(got[fin] - want[fin]) <= 1e-12 * np.maximum(want[fin], 1e-300))
    assert got[0] == 0.0
    assert np.allclose(rg.cpu().numpy(), want_g, rtol=1e-12, atol=0)
    d2 = ((S.astype(np.float64) - R) ** 2).reshape(15, -1).sum(1)
    assert np.allclose(sq.cpu().numpy()[:, 0], d2, rtol=1e-12, atol=0)


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_eq7_recursion_on_gpu(fam):
    """Perturb every cached state by delta_j: the GPU-composed gap equals the
    recursion e_j = e_{j-1} M_j + delta_j, and the diagnostic reports its norm."""
    rng = np.random.default_rng(7)
    K, h, dv, dk = 6, 3, 64, 64
    B = rng.standard_normal((K, h, dv, dk)).astype(np.float32)
    d = (0.3 * rng.standard_normal((K, h, dv, dk))).astype(np.float32)
    if fam == I.GDN:
        q, _ = np.linalg.qr(rng.standard_normal((K * h, dk, dk)))
        M = (0.95 * q).reshape(K, h, dk, dk).astype(np.float32)
        layer = lkv.make_layer(I.GDN, 1, h, dk, dv, 64)
    else:
        M = (-rng.uniform(0.0, 0.3, (K, h))).astype(np.float32)
        layer = lkv.make_layer(I.SSD, 1, h, dk, dv, 64, gate_dtype=torch.float32)
    ids = torch.arange(K, dtype=torch.int32, device="cuda")
    cu = torch.tensor([0, K], dtype=torch.int32, device="cuda")
    S_true = torch.empty((1, h, dv, dk), device="cuda")
    S_pert = torch.empty_like(S_true)
    lkv.init_compose(layer, K, _dev(B), _dev(M), ids, cu, K, S_true)
    lkv.init_compose(layer, K, _dev(B + d), _dev(M), ids, cu, K, S_pert)
    _, rel, rg = lkv.state_rel_error(S_pert, S_true, group=h)
    torch.cuda.synchronize()
    e = (S_pert - S_true).cpu().numpy()[0].astype(np.float64)
    e_ref = oracle.mismatch_recursion(d, M=M) if fam == I.GDN else oracle.mismatch_recursion(d, Lam=M)
    assert np.max(np.abs(e - e_ref)) < 1e-3 * np.max(np.abs(e_ref))
    kc = np.array([0, K], np.int32)
    kid = np.arange(K, dtype=np.int32)
    S_ref = (oracle.compose_gdn(kc, kid, B, M) if fam == I.GDN else oracle.compose_ssd(kc, kid, B, M))[0]
    rel_ref, rg_ref = oracle.rel_error(S_ref + e_ref, S_ref, group=h)
    assert np.allclose(rel.cpu().numpy(), rel_ref, rtol=1e-3, atol=0)
    assert np.allclose(rg.cpu().numpy(), rg_ref, rtol=1e-3, atol=0)


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_layer0_probe(fam):
    """On first-layer-like inputs (every block's tokens are the same whether prefilled
    alone or in context) exact composition reproduces S* (the scan of the whole
    context from zero) to the fp32 floor, while the last block alone misses the
    earlier blocks' share; both figures match the oracle's."""
    dk, dv = (64, 64) if fam == I.GDN else (64, 32)
    w = I.small(fam, n_req=2, dk=dk, dv=dv, chunk=64, blocks=((40, 23, 70, 17), (30, 90)), online=(1, 1),
                h_qk=2 if fam == I.GDN else 1, h_v=4)
    G = gpu_io.GpuWorkload(w)
    G.block_summary()
    G.init_single()
    G.init_compose()
    ctx_cu = I.context_cu(w)
    cu = torch.from_numpy(ctx_cu).cuda()
    c = G.cached
    full = lkv.make_tokens(cu, int(ctx_cu[-1]), None, c.k, c.v, c.g, c.beta, c.A)
    S_star = torch.empty_like(G.S_exact)
    if fam == I.GDN:
        lkv.gdn_chunk_scan(G.layer, full, 1.0, None, None, S_star)
    else:
        lkv.ssd_chunk_scan(G.layer, full, None, None, S_star)
    _, rel_x, rg_x = lkv.state_rel_error(G.S_exact, S_star, group=4)
    _, rel_1, rg_1 = lkv.state_rel_error(G.S_single, S_star, group=4)
    torch.cuda.synchronize()
    cc = w.cached
    if fam == I.GDN:
        _, S_ref = oracle.gdn_scan(ctx_cu, None, cc.k, cc.v, cc.g, cc.beta, want_o=False)
        _, B = oracle.gdn_scan(cc.cu, None, cc.k, cc.v, cc.g, cc.beta, want_o=False)
    else:
        _, S_ref = oracle.ssd_scan(ctx_cu, None, cc.k, cc.v, cc.g, w.A, want_y=False)
        _, B = oracle.ssd_scan(cc.cu, None, cc.k, cc.v, cc.g, w.A, want_y=False)
    _, want_1 = oracle.rel_error(B[w.last_blk], S_ref, group=4)
    assert np.all(rg_x.cpu().numpy() < 1e-4)
    assert np.allclose(rg_1.cpu().numpy(), want_1, rtol=1e-3, atol=1e-5)
    assert np.all(want_1 > 1e-3)       # the earlier blocks do matter at these gates
