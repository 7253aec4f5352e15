"""The C-ABI library without a GPU: it loads, exports every entry point the
header declares, sizes workspaces, and rejects bad arguments before any HIP
call (no call here reaches a kernel launch)."""

import ctypes as C
import os
import re

import pytest

from paper_2608_16305_amd import mtgnn as M

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mtgnn.h")

pytestmark = pytest.mark.skipif(not os.path.exists(M.LIB_PATH), reason="libmtgnn.so not built")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(mtgnn_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = M.lib()
    declared = _declared()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(M.ENTRY_POINTS) == declared
    assert L.mtgnn_version() == 100


def test_status_strings():
    L = M.lib()
    assert L.mtgnn_status_string(0) == b"ok"
    assert L.mtgnn_status_string(-3) == b"workspace too small"
    assert L.mtgnn_status_string(7) == b"unknown status"


def _dims(**kw):
    base = dict(n_nodes=1000, d_mem=32, d_time=32, d_edge=16, d_attn=32, n_heads=1, k=5, dtype=M.F32)
    base.update(kw)
    return M.Dims(*[base[f] for f, _ in M.Dims._fields_])


def test_workspace_sizes_are_monotone_and_positive():
    d = _dims()
    for op in (M.OP_AGGREGATE_LAST, M.OP_GRU_UPDATE, M.OP_TEMPORAL_ATTN_BWD, M.OP_GRU_UPDATE_BWD, M.OP_BUILD_CSR):
        a = M.workspace_bytes(op, d, 100, 150)
        b = M.workspace_bytes(op, d, 10000, 15000)
        assert 0 < a <= b, op
    assert M.save_bytes(M.OP_GRU_UPDATE, d, 400, 0) >= 5 * 400 * 32 * 4
    assert M.save_bytes(M.OP_TEMPORAL_ATTN, d, 0, 600) >= 600 * 5 * (32 + 16 + 32) * 4
    # invalid dims -> 0
    assert M.workspace_bytes(M.OP_GRU_UPDATE, _dims(n_heads=3), 10, 0) == 0


@pytest.mark.parametrize("bad,code", [
    (dict(n_heads=3), M.MtgnnError), (dict(k=0), M.MtgnnError), (dict(k=65), M.MtgnnError),
    (dict(dtype=7), M.MtgnnError), (dict(d_mem=0), M.MtgnnError), (dict(d_attn=400, n_heads=2), M.MtgnnError),
])
def test_dims_validation(bad, code):
    L = M.lib()
    d = _dims(**bad)
    b = M.Batch(0, None, None, None, None, None)
    st = L.mtgnn_build_messages(C.byref(b), C.c_void_p(8), C.c_void_p(8), None, 4, C.c_void_p(8), C.c_void_p(8),
                                C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), C.byref(d), C.c_void_p(8),
                                C.c_void_p(8), None)
    assert st in (-1, -2)
    assert L.mtgnn_last_error()


def test_null_and_size_checks_return_before_hip():
    L = M.lib()
    d = _dims()
    # NULL batch
    assert L.mtgnn_aggregate_last(None, 10, None, None, None, None, 0, None) == -1
    # a batch with n > 0 but NULL arrays
    b = M.Batch(5, None, None, None, None, None)
    assert L.mtgnn_aggregate_last(C.byref(b), 10, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), 1 << 20,
                                  None) == -1
    # too small a workspace -> EWORKSPACE, checked before any launch
    b = M.Batch(5, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), None)
    assert L.mtgnn_aggregate_last(C.byref(b), 10, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), C.c_void_p(8), 16,
                                  None) == -3
    # sampling: k out of range, NULL CSR
    assert L.mtgnn_sample_recent(None, None, None, None, 10, None, None, None, 4, 3, None, None, None, None) == -1
    p = C.c_void_p(8)
    assert L.mtgnn_sample_recent(p, p, p, p, 10, p, p, None, 4, 99, p, p, p, None) == -2
    # edge features must be given iff d_edge > 0
    b0 = M.Batch(0, None, None, None, None, None)
    assert L.mtgnn_build_messages(C.byref(b0), p, p, None, 4, p, p, None, p, p, C.byref(d), p, p, None) == -1
    # attention backward with no query is rejected (nothing to differentiate)
    g = M.AttnGrads(*([p] * 12))
    ap = M.AttnParams(*([p] * 12))
    assert L.mtgnn_temporal_attn_bwd(p, p, None, 0, p, p, p, p, p, None, 4, p, p, C.byref(ap), C.byref(d), C.byref(g),
                                     p, p, p, p, 1 << 30, None) == -1
    # CSR build: bad sizes
    assert L.mtgnn_build_temporal_csr(p, p, p, -1, 10, p, p, p, p, p, 0, None) == -1
    assert L.mtgnn_build_temporal_csr(p, p, p, 10, 0, p, p, p, p, p, 0, None) == -1
    # decoder weight copies: NULL params, a max_q that is not a multiple of 3, too small a workspace
    lp = M.LinkParams(p, p, p, p)
    assert L.mtgnn_link_prepare_weights(None, C.byref(d), 6, p, 1 << 30, None) == -1
    assert L.mtgnn_link_prepare_weights(C.byref(lp), C.byref(d), 5, p, 1 << 30, None) == -1
    assert L.mtgnn_link_prepare_weights(C.byref(lp), C.byref(d), 6, p, 16, None) == -3
    # the attention's and the decoder's copies in one call: NULL decoder parameters, a bad max_q
    assert L.mtgnn_temporal_attn_prepare_weights_link(C.byref(ap), p, p, C.byref(d), p, None, 6, p, 1 << 30,
                                                      None) == -1
    assert L.mtgnn_temporal_attn_prepare_weights_link(C.byref(ap), p, p, C.byref(d), p, C.byref(lp), 7, p, 1 << 30,
                                                      None) == -1
    # prepared loss: the second stream without its fork event (or the reverse) is rejected
    lg = M.LinkGrads(p, p, p, p)
    assert L.mtgnn_link_loss_prepared(p, p, 6, C.byref(lp), C.byref(d), p, p, p, C.byref(lg), p, 1 << 30, None, p,
                                      None) == -1
    assert L.mtgnn_link_loss_prepared(p, p, 6, C.byref(lp), C.byref(d), p, p, p, C.byref(lg), p, 1 << 30, None, None,
                                      p) == -1


def test_binding_refuses_host_tensors():
    import torch
    with pytest.raises(M.MtgnnError):
        M.batch(torch.zeros(3, dtype=torch.int32), torch.zeros(3, dtype=torch.int32), torch.zeros(3))
