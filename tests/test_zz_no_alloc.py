"""The allocation-free entry point lkv_chunk_scan_sp_noalloc, called through the
C ABI, against lkv_chunk_scan_sp with a caller workspace: the same kernels on
the same inputs, so outputs and final states must agree bit for bit (and both
with the CPU oracle within the usual bars).  Two calls in a row per family, the
second on a smaller input: the fixed per-GPU scratch keeps the first call's
contents, which the second must not depend on.  A call whose workspace exceeds
the fixed scratch is rejected before anything is launched."""
import ctypes

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


def _work(fam, online, hv, dv, seed):
    layer = I.Layer(fam, 1 if fam == I.SSD else hv // 2, hv, 128, dv, 64, "bf16", "bf16" if fam == I.GDN else "f32")
    law = I.GateLaw(x_mu=-3.0, beta_mu=0.0) if fam == I.GDN else I.GateLaw(dt_mu=-3.0, dt_bias=-1.0, a_lo=1.0,
                                                                             a_hi=4.0)
    return I.build_workload("noalloc", layer, [[] for _ in online], list(online), law, seed,
                            scale=0.75 if fam == I.GDN else 1.0)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("fam", [I.GDN, I.SSD])
def test_noalloc_matches_workspace_variant(fam):
    runs = [(_work(fam, (900, 333), 8, 128, 11), 4), (_work(fam, (150,), 4, 64, 12), 3)]
    for w, pieces in runs:  # the second call is smaller than the first
        G = gpu_io.GpuWorkload(w, with_cached=False)
        S0 = (0.3 * np.random.default_rng(4).standard_normal(tuple(G.S_final.shape))).astype(np.float32)
        S0_d = torch.from_numpy(S0).cuda()
        ws = torch.empty(lkv.chunk_scan_sp_workspace(G.layer, w.n_req, pieces), dtype=torch.uint8, device="cuda")
        out_ref, S_ref = torch.empty_like(G.out), torch.empty_like(G.S_final)
        lkv.chunk_scan_sp(G.layer, G.online.struct, w.scale, S0_d, out_ref, S_ref, pieces, ws)
        G.out.fill_(float("nan"))
        G.S_final.fill_(float("nan"))
        lkv.chunk_scan_sp_noalloc(G.layer, G.online.struct, w.scale, S0_d, G.out, G.S_final, pieces)
        torch.cuda.synchronize()
        assert torch.equal(_bits(G.out), _bits(out_ref))
        assert torch.equal(_bits(G.S_final), _bits(S_ref))
        o_ora, S_ora = R.scan(w, S0)
        assert rel_slices(_np(G.S_final), S_ora) < STATE_TOL
        assert max_abs(_np(G.out), o_ora) < OUT_ABS


def test_noalloc_rejects_beyond_scratch():
    lib = lkv.load()
    L = lkv.make_layer(I.GDN, 16, 32, 128, 128, 64)
    need = lkv.chunk_scan_sp_workspace(L, 8, 8)
    assert need > 64 << 20
    t = lkv.Tokens()
    t.n_seq, t.n_tok = 8, 0
    st = lib.lkv_chunk_scan_sp_noalloc(ctypes.byref(L), ctypes.byref(t), ctypes.c_float(1.0), None, None, None, 8,
                                       None)
    assert st == 6  # LKV_E_WORKSPACE
    assert b"64 MiB" in lib.lkv_status_string(6)
