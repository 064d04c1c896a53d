"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments synchronously (no GPU needed: all
of these return before any HIP call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lkv.h")
LIB = os.path.join(ROOT, "paper_2608_11231_amd", "liblkv.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="liblkv.so not built")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lkv_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2608_11231_amd import lkv
    return lkv.load()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"lkv_block_summary", "lkv_init_single", "lkv_init_compose", "lkv_gdn_chunk_scan",
            "lkv_ssd_chunk_scan"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    from paper_2608_11231_amd import lkv
    assert set(names) == set(lkv.EXPORTS)


def test_version_and_strings(lib):
    assert lib.lkv_abi_version() == 9
    assert lib.lkv_status_string(0) == b"ok"
    assert b"NULL" in lib.lkv_status_string(1)


def test_wait_limit_setter(lib):
    """The bound of the chunk kernels' inter-wave wait is host state: the setter
    returns the previous bound, and a negative value restores the default."""
    default = lib.lkv_set_wait_limit(-1)
    assert default == 1 << 14
    assert lib.lkv_set_wait_limit(0) == default
    assert lib.lkv_set_wait_limit(5) == 0
    assert lib.lkv_set_wait_limit(-3) == 5
    assert lib.lkv_set_wait_limit(-1) == default


def test_sp_workspace_size(lib):
    """The sequence-parallel scan's workspace: every region of the documented
    layout, each 256-byte aligned; piece counts outside 1..64 are rejected."""
    from paper_2608_11231_amd import lkv
    up = lambda x: (x + 255) // 256 * 256
    for fam, hq, hv, dk, dv, n_req, P in ((0, 2, 4, 128, 128, 3, 4), (1, 1, 64, 128, 64, 1, 8)):
        L = _layer(family=fam, h_qk=hq, h_v=hv, dk=dk, dv=dv, gate_dtype=0 if fam else 1)
        n = ctypes.c_size_t(0)
        assert lib.lkv_chunk_scan_sp_workspace(ctypes.byref(L), n_req, P, ctypes.byref(n)) == 0
        seg, state = n_req * P, hv * dv * dk * 4
        trans = hv * dk * dk * 4 if fam == 0 else hv * 4
        want = (up((seg + 1) * 4) + up(n_req * (P + 1) * 4) + up((n_req + 1) * 4) + up((seg + n_req) * state)
                + up((seg + n_req) * trans) + up(seg * state) + up(n_req * state))
        assert n.value == want
        assert lkv.chunk_scan_sp_workspace(L, n_req, P) == want
        for bad in (0, 65):
            assert lib.lkv_chunk_scan_sp_workspace(ctypes.byref(L), n_req, bad, ctypes.byref(n)) == 2


def _layer(**kw):
    from paper_2608_11231_amd import lkv
    d = dict(family=0, h_qk=2, h_v=4, dk=128, dv=128, chunk=64, io_dtype=1, gate_dtype=1)
    d.update(kw)
    return lkv.Layer(**d)


def _tokens(n_seq=0, n_tok=0):
    from paper_2608_11231_amd import lkv
    t = lkv.Tokens()
    t.n_seq, t.n_tok = n_seq, n_tok
    return t


def test_argument_validation(lib):
    by = ctypes.byref
    T = _tokens()
    assert lib.lkv_gdn_chunk_scan(None, by(T), ctypes.c_float(1.0), None, None, None, None) == 1
    assert lib.lkv_gdn_chunk_scan(by(_layer(dk=96)), by(T), ctypes.c_float(1.0), None, None, None, None) == 5
    assert lib.lkv_gdn_chunk_scan(by(_layer(dv=40)), by(T), ctypes.c_float(1.0), None, None, None, None) == 5
    assert lib.lkv_gdn_chunk_scan(by(_layer(chunk=48)), by(T), ctypes.c_float(1.0), None, None, None, None) == 5
    assert lib.lkv_gdn_chunk_scan(by(_layer(h_v=3)), by(T), ctypes.c_float(1.0), None, None, None, None) == 2
    assert lib.lkv_gdn_chunk_scan(by(_layer(io_dtype=7)), by(T), ctypes.c_float(1.0), None, None, None, None) == 3
    # family mismatch
    assert lib.lkv_ssd_chunk_scan(by(_layer()), by(T), None, None, None, None) == 2
    assert lib.lkv_ssd_chunk_scan(by(_layer(family=1, gate_dtype=1)), by(T), None, None, None, None) == 3
    # empty batch: nothing to launch
    assert lib.lkv_gdn_chunk_scan(by(_layer()), by(T), ctypes.c_float(1.0), None, None, None, None) == 0
    # missing token tensors
    T2 = _tokens(1, 10)
    T2.cu = ctypes.c_void_p(0x1000)
    assert lib.lkv_gdn_chunk_scan(by(_layer()), by(T2), ctypes.c_float(1.0), None, None, None, None) == 1
    # misaligned tensor
    T3 = _tokens(1, 10)
    T3.cu = T3.k = T3.v = T3.g = T3.beta = T3.q = ctypes.c_void_p(0x1008)
    assert lib.lkv_gdn_chunk_scan(by(_layer()), by(T3), ctypes.c_float(1.0), None, None, None, None) == 4
    # summaries need at least one output
    assert lib.lkv_block_summary(by(_layer()), by(T), None, None, None) == 1
    # init calls
    assert lib.lkv_init_single(by(_layer()), -1, 1, None, None, None, None) == 2
    assert lib.lkv_init_single(by(_layer()), 0, 1, None, None, None, None) == 0
    assert lib.lkv_init_single(by(_layer()), 2, 1, None, None, None, None) == 1
    assert lib.lkv_init_compose(by(_layer()), 1, 1, None, None, None, None, 0, None, None) == 1
    assert lib.lkv_init_compose(by(_layer()), 0, 0, None, None, None, None, 0, None, None) == 0



def test_decode_and_gather_validation(lib):
    by = ctypes.byref
    vp = ctypes.c_void_p
    # decode: family checked per call, empty batch is a no-op, missing tensors
    assert lib.lkv_ssd_decode(by(_layer()), 1, *([None] * 7), None) == 2
    assert lib.lkv_gdn_decode(by(_layer()), 0, *([None] * 5), ctypes.c_float(1.0), None, None, None) == 0
    assert lib.lkv_gdn_decode(by(_layer()), 1, *([None] * 5), ctypes.c_float(1.0), None, None, None) == 1
    assert lib.lkv_gdn_decode(by(_layer()), -1, *([None] * 5), ctypes.c_float(1.0), None, None, None) == 2
    a = vp(0x1000)
    assert lib.lkv_gdn_decode(by(_layer()), 1, a, a, vp(0x1008), a, a, ctypes.c_float(1.0), a, None,
                              None) == 4
    # gather: nothing selected is a no-op; a requested array needs its source
    C = _tokens(1, 10)
    C.cu = a
    assert lib.lkv_gather_selected(by(_layer()), by(C), None, None, ctypes.c_int64(0), a, a, a, a, a,
                                   None) == 0
    assert lib.lkv_gather_selected(by(_layer()), by(C), a, a, ctypes.c_int64(-1), None, None, None,
                                   None, None, None) == 2
    assert lib.lkv_gather_selected(by(_layer()), by(C), a, a, ctypes.c_int64(4), a, None, None, None,
                                   None, None) == 1
    C.q = vp(0x1008)
    assert lib.lkv_gather_selected(by(_layer()), by(C), a, a, ctypes.c_int64(4), a, None, None, None,
                                   None, None) == 4
    assert lib.lkv_gather_selected(by(_layer()), by(C), a, a, ctypes.c_int64(4), None, None, None, None,
                                   None, None) == 0
    assert lib.lkv_gather_selected(by(_layer()), None, a, a, ctypes.c_int64(4), None, None, None, None,
                                   None, None) == 1



def test_pool_calls_validation(lib):
    by = ctypes.byref
    vp = ctypes.c_void_p
    a = vp(0x1000)
    assert lib.lkv_round_bf16(None, None, ctypes.c_int64(0), None) == 0
    assert lib.lkv_round_bf16(a, a, ctypes.c_int64(-1), None) == 2
    assert lib.lkv_round_bf16(None, a, ctypes.c_int64(8), None) == 1
    assert lib.lkv_round_bf16(a, vp(0x1002), ctypes.c_int64(8), None) == 4
    assert lib.lkv_stage_rows(None, None, None, 0, ctypes.c_int64(64), None) == 0
    assert lib.lkv_stage_rows(a, a, None, 2, ctypes.c_int64(64), None) == 1
    bad = (ctypes.c_int32 * 2)(0, -3)
    assert lib.lkv_stage_rows(a, a, bad, 2, ctypes.c_int64(64), None) == 2
    assert lib.lkv_init_single_bf16(by(_layer()), 0, 1, None, None, None, None) == 0
    assert lib.lkv_init_single_bf16(by(_layer()), 2, 1, None, None, None, None) == 1
    assert lib.lkv_init_compose_bf16(by(_layer()), 1, 1, None, None, None, None, 0, None, None) == 1



def test_rel_error_validation(lib):
    vp = ctypes.c_void_p
    a = vp(0x1000)
    i64 = ctypes.c_int64
    assert lib.lkv_state_rel_error(None, None, 0, i64(16), 1, None, None, None, None) == 0
    assert lib.lkv_state_rel_error(a, a, -1, i64(16), 1, a, a, None, None) == 2
    assert lib.lkv_state_rel_error(a, None, 2, i64(16), 1, a, a, None, None) == 1
    assert lib.lkv_state_rel_error(a, a, 2, i64(18), 1, a, a, None, None) == 2
    assert lib.lkv_state_rel_error(a, a, 3, i64(16), 2, a, a, a, None) == 2
    assert lib.lkv_state_rel_error(a, vp(0x1004), 2, i64(16), 1, a, a, None, None) == 4



def test_scan_from_pool_validation(lib):
    by = ctypes.byref
    vp = ctypes.c_void_p
    T = _tokens()
    f = ctypes.c_float(1.0)
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T), f, None, 0, 0, None, None, None, None) == 0
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T), f, None, 7, 0, None, None, None, None) == 3
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T), f, None, 0, -1, None, None, None, None) == 2
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T), f, None, 0, 2, None, None, None, None) == 1
    T1 = _tokens(1, 10)
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T1), f, None, 0, 0, None, None, None, None) == 1
    assert lib.lkv_chunk_scan_from_pool(by(_layer()), by(T), f, vp(0x1008), 0, 1, None, None, None, None) == 4
