"""Full-size parity: the reference workloads at their real shapes, run through the
same calls (and so the same launch geometry) the benchmark times, checked
against the CPU oracle on every value head of request 0 and on head 0 of every
other request.

Each checked (request, head) pair covers every stage: the per-block states B_k
and transitions M_k (Lambda_k) of all the request's cached blocks, both initial
states, and the scan's outputs and final state.  Mild-gate variants (slowly
decaying gates) make every cached block visible in the composed state: at the
32K Gated DeltaNet workload that is the 32-block composition with transitions
that matter.
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


def _oracle_request(w, r, heads):
    """Oracle results for request r on the value heads ``heads`` (``"all"`` or
    ``"first"``), fp64: the states and transitions of every cached block of the
    request, both initial states, the outputs and the final state."""
    L = w.layer
    hr = L.h_v // L.h_qk
    hv = slice(0, L.h_v) if heads == "all" else slice(0, 1)
    hq = slice(0, L.h_qk) if heads == "all" else slice(0, 1)
    c, o = w.cached, w.online
    ids = w.blk_ids[w.blk_cu[r]:w.blk_cu[r + 1]]
    # the request's blocks in context order, packed as one stream of segments
    rows = np.concatenate([np.arange(int(c.cu[b]), int(c.cu[b + 1])) for b in ids]) if len(ids) else \
        np.zeros(0, np.int64)
    cu = np.concatenate([[0], np.cumsum([int(c.cu[b + 1] - c.cu[b]) for b in ids])]).astype(np.int32)
    assert hr >= 1
    if L.family == I.GDN:
        _, B = oracle.gdn_scan(cu, None, c.k[rows, hq], c.v[rows, hv], c.g[rows, hv], c.beta[rows, hv],
                               want_o=False)
        M = oracle.gdn_transition(cu, c.k[rows, hq], c.g[rows, hv], c.beta[rows, hv])
    else:
        _, B = oracle.ssd_scan(cu, None, c.k[rows, hq], c.v[rows, hv], c.g[rows, hv], w.A[hv], want_y=False)
        M = oracle.ssd_log_decay(cu, c.g[rows, hv], w.A[hv])
    K = len(ids)
    kcu = np.array([0, K], np.int32)
    kid = np.arange(K, dtype=np.int32)
    SX = (oracle.compose_gdn if L.family == I.GDN else oracle.compose_ssd)(kcu, kid, B, M)
    S1 = B[-1]
    sl = slice(int(o.cu[r]), int(o.cu[r + 1]))
    ocu = np.array([0, sl.stop - sl.start], np.int32)
    if L.family == I.GDN:
        out, SF = oracle.gdn_scan(ocu, o.q[sl, hq], o.k[sl, hq], o.v[sl, hv], o.g[sl, hv], o.beta[sl, hv],
                                  scale=w.scale, S0=SX)
    else:
        out, SF = oracle.ssd_scan(ocu, o.q[sl, hq], o.k[sl, hq], o.v[sl, hv], o.g[sl, hv], w.A[hv], S0=SX)
    return dict(ids=ids, hv=hv, B=B, M=M, S1=S1, SX=SX[0], out=out, SF=SF[0], sl=sl)


CASES = [(1, False), (1, True), (2, False), (2, True), (3, False), (3, True), (4, False), (4, True)]


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
    # ... over the transitions the composition reads (blocks 2..K; every other
    # block an empty segment): the same transitions bit for bit, identity
    # (Lambda = 0) rows for the dropped blocks, and the same composed state, bit
    # for bit
    G.fold_transitions()
    G.init_compose()
    torch.cuda.synchronize()
    M_fold, SX_fold = _np(G.M_pool), _np(G.S_exact)
    first = gpu_io.fold_dropped_blocks(w)
    assert first, "every workload here has first blocks to drop"
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
    # every value head of request 0 and head 0 of every other request, each
    # against the oracle run over the request's whole cached context
    for r in range(w.n_req):
        ref = _oracle_request(w, r, "all" if r == 0 else "first")
        ids, hv = ref["ids"], ref["hv"]
        tag = (r, "all heads" if r == 0 else "head 0")
        assert rel_slices(B_pool[ids, hv], ref["B"]) < STATE_TOL, tag + ("B",)
        if L.family == I.GDN:
            assert rel_slices(M_pool[ids, hv], ref["M"]) < STATE_TOL, tag + ("M",)
        else:
            for lam in (M_pool[ids, hv], M_only[ids, hv]):
                assert np.max(np.abs(lam - ref["M"]) / np.maximum(np.abs(ref["M"]), 1e-30)) < STATE_TOL, tag
        assert rel_slices(S1[r, hv], ref["S1"], lead=1) < STATE_TOL, tag + ("S1",)
        assert rel_slices(SX[r, hv], ref["SX"], lead=1) < STATE_TOL, tag + ("SX",)
        assert rel_slices(SF[r, hv], ref["SF"], lead=1) < STATE_TOL, tag + ("SF",)
        assert max_abs(out[ref["sl"], hv], ref["out"]) < OUT_ABS, tag + ("out",)
