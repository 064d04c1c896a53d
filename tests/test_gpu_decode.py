"""GPU parity of the decode step (one token per request after the prefill)
against the CPU oracle's token recurrence.

Bars as for the scan: the fp32 state within 1e-4 normwise relative error per
(request, head) slice; bf16 outputs within 2e-2 absolute error; fp32-io
outputs within 1e-4 relative.  Steps are chained so that the state the kernel
writes is the one it reads next, and the last case continues a GPU prefill.
"""
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


def _np(t):
    return t.detach().float().cpu().numpy()


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def _work(fam, dk, dv, io, hq, hv, lens, seed=21):
    layer = I.Layer(fam, hq, hv, dk, dv, 64, io, io if fam == I.GDN else "f32")
    if fam == I.GDN:
        law = I.GateLaw(x_mu=-3.0, beta_mu=0.0)
    else:
        law = I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0, a_hi=4.0)
    return I.build_workload("decode", layer, [[] for _ in lens], list(lens), law, seed,
                            scale=0.75 if fam == I.GDN else 1.0)


def _oracle_scan(w, S0):
    o = w.online
    if w.layer.family == I.GDN:
        return oracle.gdn_scan(o.cu, o.q, o.k, o.v, o.g, o.beta, scale=w.scale, S0=S0)
    return oracle.ssd_scan(o.cu, o.q, o.k, o.v, o.g, w.A, S0=S0)


def _check_out(got, ref, io):
    if io == "f32":
        assert rel_slices(got[None], ref[None], lead=1) < STATE_TOL
    else:
        assert max_abs(got, ref) < OUT_ABS


CASES = [
    # (family, dk, dv, io, h_qk, h_v, n_req, steps)
    (I.GDN, 16, 16, "f32", 1, 1, 3, 4),
    (I.GDN, 32, 48, "bf16", 2, 4, 5, 3),
    (I.GDN, 64, 64, "f32", 1, 2, 2, 3),
    (I.GDN, 128, 128, "bf16", 2, 4, 3, 3),
    (I.GDN, 128, 512, "bf16", 1, 1, 2, 2),
    (I.SSD, 16, 16, "f32", 1, 2, 3, 4),
    (I.SSD, 128, 64, "bf16", 1, 4, 3, 3),
    (I.SSD, 64, 32, "bf16", 2, 4, 2, 3),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{'gdn' if c[0] == I.GDN else 'ssd'}{c[1:6]}" for c in CASES])
def test_decode_steps_chain(case):
    """``steps`` decode steps from a random state equal one oracle scan over the
    steps' tokens; every step's outputs are checked."""
    fam, dk, dv, io, hq, hv, n_req, T = case
    w = _work(fam, dk, dv, io, hq, hv, [T] * n_req)
    rng = np.random.default_rng(dk + dv + T)
    S0 = (0.3 * rng.standard_normal((n_req, hv, dv, dk))).astype(np.float32)
    o_ref, S_ref = _oracle_scan(w, S0)
    S = _dev(S0)
    for t in range(T):
        idx = w.online.cu[:-1] + t
        step = gpu_io.GpuStep(w.online, idx, w.layer, w.A, w.scale)
        step.decode(S)
        torch.cuda.synchronize()
        _check_out(_np(step.out), o_ref[idx], io)
    assert rel_slices(_np(S), S_ref) < STATE_TOL


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_decode_continues_prefill(fam):
    """GPU chunk scan over each request's first L tokens, then one GPU decode
    step: the state and the last outputs equal the oracle's scan over L + 1."""
    dk, dv = (128, 128) if fam == I.GDN else (128, 64)
    lens = [130, 65, 1, 200]
    w = _work(fam, dk, dv, "bf16", 2 if fam == I.GDN else 1, 4, [L + 1 for L in lens], seed=5)
    full = w.online
    cu_p = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    keep = np.concatenate([np.arange(full.cu[r], full.cu[r + 1] - 1) for r in range(len(lens))])
    pre = I.Tokens(cu=cu_p, q=full.q[keep], k=full.k[keep], v=full.v[keep], g=full.g[keep],
                   beta=None if full.beta is None else full.beta[keep])
    wp = I.Workload(name="prefix", layer=w.layer, cached=w.cached, online=pre, blk_cu=w.blk_cu,
                    blk_ids=w.blk_ids, last_blk=w.last_blk, A=w.A, scale=w.scale)
    rng = np.random.default_rng(9)
    S0 = (0.3 * rng.standard_normal((len(lens), 4, dv, dk))).astype(np.float32)
    G = gpu_io.GpuWorkload(wp, with_cached=False)
    G.scan(_dev(S0))
    last = full.cu[1:] - 1
    step = gpu_io.GpuStep(full, last, w.layer, w.A, w.scale)
    step.decode(G.S_final)
    torch.cuda.synchronize()
    o_ref, S_ref = _oracle_scan(w, S0)
    assert rel_slices(_np(G.S_final), S_ref) < STATE_TOL
    assert max_abs(_np(step.out), o_ref[last]) < OUT_ABS


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_decode_state_only_matches_and_empty_batch(fam):
    """A NULL output pointer updates the state bit-identically; zero requests is a no-op."""
    w = _work(fam, 64, 64, "bf16", 1, 2, [1, 1, 1])
    step = gpu_io.GpuStep(w.online, w.online.cu[:-1], w.layer, w.A, w.scale)
    S0 = _dev(0.3 * np.random.default_rng(4).standard_normal((3, 2, 64, 64)))
    S1, S2 = S0.clone(), S0.clone()
    step.decode(S1, with_out=True)
    step.decode(S2, with_out=False)
    torch.cuda.synchronize()
    assert torch.equal(S1.view(torch.int32), S2.view(torch.int32))
    e = torch.empty(0, device="cuda")
    if fam == I.GDN:
        lkv.gdn_decode(step.layer, e, e, e, e, e, 1.0, e, None)
    else:
        lkv.ssd_decode(step.layer, e, e, e, e, step.A, e, None)
    torch.cuda.synchronize()


def test_decode_family_mismatch_is_an_error():
    w = _work(I.SSD, 16, 16, "f32", 1, 1, [1])
    step = gpu_io.GpuStep(w.online, w.online.cu[:-1], w.layer, w.A, w.scale)
    S = torch.zeros((1, 1, 16, 16), device="cuda")
    with pytest.raises(lkv.LkvError):
        lkv.gdn_decode(step.layer, step.q, step.k, step.v, step.g, step.g, 1.0, S, None)


@pytest.mark.parametrize("n_req", [4, 256])
def test_decode_full_size(n_req):
    """The 32-head, 128 x 128 Gated DeltaNet state of the 32K-context workload, at its
    4 requests and at a 256-request decode batch (512 MiB of state, the launch the
    benchmark times); sampled requests are checked against the oracle."""
    L = I.Layer(I.GDN, 32, 32, 128, 128, 64)
    w = _work(I.GDN, L.dk, L.dv, L.io_dtype, L.h_qk, L.h_v, [1] * n_req, seed=n_req)
    rng = np.random.default_rng(n_req)
    S0 = (0.3 * rng.standard_normal((n_req, L.h_v, L.dv, L.dk))).astype(np.float32)
    step = gpu_io.GpuStep(w.online, w.online.cu[:-1], w.layer, w.A, w.scale)
    S = _dev(S0)
    step.decode(S)
    torch.cuda.synchronize()
    got_S, got_o = _np(S), _np(step.out)
    reqs = sorted(set([0, n_req - 1, int(rng.integers(0, n_req))]))
    o = w.online
    o_ref, S_ref = oracle.gdn_decode(o.q[reqs], o.k[reqs], o.v[reqs], o.g[reqs], o.beta[reqs],
                                     S0[reqs], scale=w.scale)
    assert rel_slices(got_S[reqs], S_ref) < STATE_TOL
    assert max_abs(got_o[reqs], o_ref) < OUT_ABS
