"""Full-size parity: the reference workloads at their real shapes, run through the
same calls (and so the same launch geometry) the benchmark times, checked
against the CPU oracle on sampled (request, head) slices.

Each sampled slice checks every stage: the per-block states B_k and
transitions M_k (Lambda_k) of all the request's cached blocks, both initial
states, and the scan's outputs and final state.  Mild-gate variants (slowly
decaying gates) make every cached block visible in the composed state.
"""
import numpy as np
import pytest

import oracle
from paper_2608_11231_amd import inputs as I

from oracle_ref import max_abs, rel_slices

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_11231_amd import gpu_io  # noqa: E402

STATE_TOL = 1e-4
OUT_ABS = 2e-2


def _np(t):
    return t.detach().float().cpu().numpy()


def _oracle_slice(w, r, h):
    """Oracle results for request r, value head h (one head, fp64)."""
    L = w.layer
    hq = h // (L.h_v // L.h_qk)
    c, o = w.cached, w.online
    ids = w.blk_ids[w.blk_cu[r]:w.blk_cu[r + 1]]
    Bs, Ms = [], []
    for b in ids:
        sl = slice(int(c.cu[b]), int(c.cu[b + 1]))
        cu = np.array([0, sl.stop - sl.start], np.int32)
        if L.family == I.GDN:
            _, Bb = oracle.gdn_scan(cu, None, c.k[sl, hq:hq + 1], c.v[sl, h:h + 1], c.g[sl, h:h + 1],
                                    c.beta[sl, h:h + 1], want_o=False)
            Mb = oracle.gdn_transition(cu, c.k[sl, hq:hq + 1], c.g[sl, h:h + 1], c.beta[sl, h:h + 1])
        else:
            _, Bb = oracle.ssd_scan(cu, None, c.k[sl, hq:hq + 1], c.v[sl, h:h + 1], c.g[sl, h:h + 1],
                                    w.A[h:h + 1], want_y=False)
            Mb = oracle.ssd_log_decay(cu, c.g[sl, h:h + 1], w.A[h:h + 1])
        Bs.append(Bb[0, 0])
        Ms.append(Mb[0, 0])
    B = np.stack(Bs)
    M = np.stack(Ms)
    K = len(ids)
    kcu = np.array([0, K], np.int32)
    kid = np.arange(K, dtype=np.int32)
    if L.family == I.GDN:
        SX = oracle.compose_gdn(kcu, kid, B[:, None], M[:, None])
    else:
        SX = oracle.compose_ssd(kcu, kid, B[:, None], M[:, None])
    S1 = B[-1]
    sl = slice(int(o.cu[r]), int(o.cu[r + 1]))
    cu = np.array([0, sl.stop - sl.start], np.int32)
    if L.family == I.GDN:
        out, SF = oracle.gdn_scan(cu, o.q[sl, hq:hq + 1], o.k[sl, hq:hq + 1], o.v[sl, h:h + 1],
                                  o.g[sl, h:h + 1], o.beta[sl, h:h + 1], scale=w.scale, S0=SX)
    else:
        out, SF = oracle.ssd_scan(cu, o.q[sl, hq:hq + 1], o.k[sl, hq:hq + 1], o.v[sl, h:h + 1],
                                  o.g[sl, h:h + 1], w.A[h:h + 1], S0=SX)
    return dict(ids=ids, B=B, M=M, S1=S1, SX=SX[0, 0], out=out[:, 0], SF=SF[0, 0], sl=sl)


CASES = [(1, False), (1, True), (2, False), (2, True), (3, False), (4, False), (4, True)]


@pytest.mark.parametrize("index,mild", CASES, ids=[f"{I.CONFIG_NAMES[i]}{'_mild' if m else ''}"
                                                     for i, m in CASES])
def test_full_size_config(index, mild):
    w = I.config(index, mild=mild, workers=16)
    L = w.layer
    G = gpu_io.GpuWorkload(w)
    G.block_summary(B=True, M=True)
    G.init_single()
    G.init_compose()
    G.scan(G.S_exact)
    torch.cuda.synchronize()
    B_pool, M_pool = _np(G.B_pool), _np(G.M_pool)
    S1, SX, SF, out = _np(G.S_single), _np(G.S_exact), _np(G.S_final), _np(G.out)
    # the benchmark's fold asks for the transitions only (Mamba-2: the segmented dt sum)
    G.block_summary(B=False, M=True)
    G.init_compose()
    torch.cuda.synchronize()
    M_only, SX_only = _np(G.M_pool), _np(G.S_exact)
    if L.family == I.GDN:
        assert np.array_equal(M_only.view(np.uint32), M_pool.view(np.uint32))
    else:
        assert np.max(np.abs(M_only - M_pool) / np.maximum(np.abs(M_pool), 1e-30)) < 1e-5
    # ... over blocks 2..K only (each request's first block an empty segment): the
    # same transitions bit for bit, identity (Lambda = 0) rows for the first
    # blocks, and the same composed state, bit for bit
    G.fold_transitions()
    G.init_compose()
    torch.cuda.synchronize()
    M_fold, SX_fold = _np(G.M_pool), _np(G.S_exact)
    first = sorted({int(w.blk_ids[w.blk_cu[r]]) for r in range(w.n_req) if w.blk_cu[r + 1] > w.blk_cu[r]})
    rest = [b for b in range(w.n_blk) if b not in first]
    assert np.array_equal(M_fold[rest].view(np.uint32), M_only[rest].view(np.uint32))
    if L.family == I.GDN:
        eye = np.broadcast_to(np.eye(L.dk, dtype=np.float32), M_fold[first].shape)
        assert np.array_equal(M_fold[first], eye)
    else:
        assert np.all(M_fold[first] == 0)
    assert np.array_equal(SX_fold.view(np.uint32), SX_only.view(np.uint32))
    # the single-block state is a bit-exact copy of the pool row
    assert np.array_equal(S1.view(np.uint32), B_pool[w.last_blk].view(np.uint32))
    rng = np.random.default_rng(index)
    reqs = sorted(set([0, w.n_req - 1, int(rng.integers(0, w.n_req))]))
    heads = sorted(set([0, L.h_v - 1, int(rng.integers(0, L.h_v))]))
    for r in reqs[:2]:
        for h in heads[:2]:
            ref = _oracle_slice(w, r, h)
            ids = ref["ids"]
            assert rel_slices(B_pool[ids, h], ref["B"], lead=1) < STATE_TOL, (r, h, "B")
            if L.family == I.GDN:
                assert rel_slices(M_pool[ids, h], ref["M"], lead=1) < STATE_TOL, (r, h, "M")
            else:
                for lam in (M_pool[ids, h], M_only[ids, h]):
                    assert np.max(np.abs(lam - ref["M"]) / np.maximum(np.abs(ref["M"]), 1e-30)) < STATE_TOL
            assert rel_slices(S1[r, h][None, None], ref["S1"][None, None]) < STATE_TOL, (r, h, "S1")
            assert rel_slices(SX[r, h][None, None], ref["SX"][None, None]) < STATE_TOL, (r, h, "SX")
            assert rel_slices(SF[r, h][None, None], ref["SF"][None, None]) < STATE_TOL, (r, h, "SF")
            assert max_abs(out[ref["sl"], h], ref["out"]) < OUT_ABS, (r, h, "out")
