"""ctypes binding of libmtgnn.so.

Argument marshalling only: every function checks that its tensors live on the
GPU with the expected dtype and layout, passes their device pointers and the
current HIP stream to the C entry point of the same name, and raises
``MtgnnError`` on a non-zero status.  No computation happens here, and there
is no fallback: if the library is missing, the first call raises.
"""

import ctypes as C
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmtgnn.so")

F32, BF16 = 0, 1
OP_BUILD_QUERIES, OP_AGGREGATE_LAST, OP_BUILD_MESSAGES, OP_GRU_UPDATE, OP_SAMPLE_RECENT = 0, 1, 2, 3, 4
OP_TEMPORAL_ATTN, OP_TEMPORAL_ATTN_BWD, OP_GRU_UPDATE_BWD, OP_BUILD_MESSAGES_BWD, OP_BUILD_CSR = 5, 6, 7, 8, 9
OP_LINK_LOSS, OP_MIXED_BATCHES, OP_RNN_UPDATE, OP_RNN_UPDATE_BWD, OP_TIME_PROJECTION_BWD = 10, 11, 12, 13, 14

ENTRY_POINTS = (
    "mtgnn_build_queries", "mtgnn_aggregate_last", "mtgnn_build_messages", "mtgnn_gru_update",
    "mtgnn_sample_recent", "mtgnn_temporal_attn", "mtgnn_temporal_attn_prepare", "mtgnn_temporal_attn_prepare_weights",
    "mtgnn_temporal_attn_prepare_weights_link",
    "mtgnn_temporal_attn_prepare_slots", "mtgnn_temporal_attn_prepared",
    "mtgnn_temporal_attn_bwd", "mtgnn_temporal_attn_bwd_overlap", "mtgnn_temporal_attn_bwd_group",
    "mtgnn_temporal_attn_bwd_grouped",
    "mtgnn_gru_update_bwd", "mtgnn_link_loss", "mtgnn_link_loss_overlap", "mtgnn_link_prepare_weights",
    "mtgnn_link_loss_prepared",
    "mtgnn_build_messages_bwd", "mtgnn_build_messages_bwd_noalloc", "mtgnn_build_temporal_csr",
    "mtgnn_dependency_scan", "mtgnn_mixed_batches", "mtgnn_rnn_update", "mtgnn_rnn_update_bwd",
    "mtgnn_time_projection", "mtgnn_time_projection_bwd", "mtgnn_controller_create", "mtgnn_controller_destroy",
    "mtgnn_controller_decide", "mtgnn_controller_observe", "mtgnn_controller_state", "mtgnn_grad_norm_ws_bytes",
    "mtgnn_grad_norm", "mtgnn_prune_aux", "mtgnn_cache_refresh", "mtgnn_adam_step", "mtgnn_workspace_bytes", "mtgnn_save_bytes",
    "mtgnn_status_string", "mtgnn_last_error", "mtgnn_version", "mtgnn_timer_start", "mtgnn_timer_stop",
)


class MtgnnError(RuntimeError):
    pass


class Dims(C.Structure):
    _fields_ = [("n_nodes", C.c_int64), ("d_mem", C.c_int32), ("d_time", C.c_int32), ("d_edge", C.c_int32),
                ("d_attn", C.c_int32), ("n_heads", C.c_int32), ("k", C.c_int32), ("dtype", C.c_int32)]


class Batch(C.Structure):
    _fields_ = [("n", C.c_int64), ("src", C.c_void_p), ("dst", C.c_void_p), ("eid", C.c_void_p),
                ("t", C.c_void_p), ("flags", C.c_void_p)]


_ATTN = ("W_q", "W_k", "W_v", "W_o", "W_1", "W_2", "b_q", "b_k", "b_v", "b_o", "b_1", "b_2")


class AttnParams(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _ATTN]


class AttnGrads(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _ATTN]


_LINK = ("W_d1", "b_d1", "W_d2", "b_d2")


class ControllerConfig(C.Structure):
    _fields_ = [("alpha", C.c_double), ("beta", C.c_double), ("tau_g", C.c_double), ("tau_c", C.c_double),
                ("interval", C.c_int32)]


class AdamConfig(C.Structure):
    _fields_ = [("lr", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
                ("t", C.c_int32)]


class LinkParams(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _LINK]


class LinkGrads(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _LINK]


_P = C.c_void_p
_I64 = C.c_int64
_I32 = C.c_int32
_SZ = C.c_size_t
_SIGS = {
    "mtgnn_build_queries": [C.POINTER(Batch), _P, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_aggregate_last": [C.POINTER(Batch), _I64, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_build_messages": [C.POINTER(Batch), _P, _P, _P, _I64, _P, _P, _P, _P, _P, C.POINTER(Dims), _P, _P, _P],
    "mtgnn_gru_update": [C.POINTER(Batch), _P, _P, _P, _I64, _P, _P, _P, _P, _P, C.POINTER(Dims), _P, _P, _P, _P, _SZ,
                         _P],
    "mtgnn_sample_recent": [_P, _P, _P, _P, _I64, _P, _P, _P, _I64, _I32, _P, _P, _P, _P],
    "mtgnn_temporal_attn": [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _P, C.POINTER(AttnParams), C.POINTER(Dims), _P,
                            _P, _P, _SZ, _P],
    "mtgnn_temporal_attn_prepare": [_P, _P, _I64, C.POINTER(AttnParams), _P, _P, C.POINTER(Dims), _P, _P, _SZ, _P],
    "mtgnn_temporal_attn_prepare_weights": [C.POINTER(AttnParams), _P, _P, C.POINTER(Dims), _P, _P],
    "mtgnn_temporal_attn_prepare_weights_link": [C.POINTER(AttnParams), _P, _P, C.POINTER(Dims), _P,
                                                 C.POINTER(LinkParams), _I64, _P, _SZ, _P],
    "mtgnn_temporal_attn_prepare_slots": [_P, _P, _I64, C.POINTER(Dims), _P, _P, _SZ, _P],
    "mtgnn_temporal_attn_prepared": [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _P, C.POINTER(AttnParams),
                                     C.POINTER(Dims), _P, _P, _P],
    "mtgnn_temporal_attn_bwd": [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _I64, _P, _P, C.POINTER(AttnParams),
                                C.POINTER(Dims), C.POINTER(AttnGrads), _P, _P, _P, _P, _SZ, _P],
    "mtgnn_temporal_attn_bwd_overlap": [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _I64, _P, _P,
                                        C.POINTER(AttnParams), C.POINTER(Dims), C.POINTER(AttnGrads), _P, _P, _P, _P,
                                        _SZ, _P, _P, _P, _P],
    "mtgnn_temporal_attn_bwd_group": [_P, _P, _I64, _P, _P, _P, _P, _I64, C.POINTER(Dims), _P, _SZ, _P],
    "mtgnn_temporal_attn_bwd_grouped": [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _I64, _P, _P,
                                        C.POINTER(AttnParams), C.POINTER(Dims), C.POINTER(AttnGrads), _P, _P, _P, _P,
                                        _SZ, _P, _P, _P, _P],
    "mtgnn_gru_update_bwd": [_P, _P, _P, _P, _I64, _P, _P, C.POINTER(Dims), _P, _P, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_link_loss": [_P, _P, _I64, C.POINTER(LinkParams), C.POINTER(Dims), _P, _P, _P, C.POINTER(LinkGrads), _P,
                        _SZ, _P],
    "mtgnn_link_loss_overlap": [_P, _P, _I64, C.POINTER(LinkParams), C.POINTER(Dims), _P, _P, _P,
                                C.POINTER(LinkGrads), _P, _SZ, _P, _P, _P],
    "mtgnn_link_prepare_weights": [C.POINTER(LinkParams), C.POINTER(Dims), _I64, _P, _SZ, _P],
    "mtgnn_link_loss_prepared": [_P, _P, _I64, C.POINTER(LinkParams), C.POINTER(Dims), _P, _P, _P,
                                 C.POINTER(LinkGrads), _P, _SZ, _P, _P, _P],
    "mtgnn_build_messages_bwd": [_P, _P, _P, _I64, _P, _P, C.POINTER(Dims), _P, _P, _P, _SZ, _P],
    "mtgnn_build_messages_bwd_noalloc": [_P, _P, _P, _I64, _P, _P, C.POINTER(Dims), _P, _P, _P],
    "mtgnn_build_temporal_csr": [_P, _P, _P, _I64, _I64, _P, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_dependency_scan": [_P, _P, _I64, _P, _I64, _I32, _I64, _I32, _P, _P, _P],
    "mtgnn_rnn_update": [C.POINTER(Batch), _P, _P, _P, _I64, _P, _P, _P, _P, _P, C.POINTER(Dims), _P, _P, _P, _P, _SZ,
                         _P],
    "mtgnn_rnn_update_bwd": [_P, _P, _P, _P, _I64, _P, _P, C.POINTER(Dims), _P, _P, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_time_projection": [_P, _P, _P, _I64, _P, _P, _P, _P, C.c_float, C.POINTER(Dims), _P, _P],
    "mtgnn_time_projection_bwd": [_P, _P, _P, _I64, _P, _P, _P, _P, C.c_float, _P, _P, _P, _I64, C.POINTER(Dims),
                                  _P, _P, _P, _P, _SZ, _P],
    "mtgnn_controller_create": [C.POINTER(ControllerConfig), C.POINTER(C.c_void_p)],
    "mtgnn_controller_destroy": [_P],
    "mtgnn_controller_decide": [_P, _I64, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32)],
    "mtgnn_controller_observe": [_P, C.c_double, C.c_double],
    "mtgnn_controller_state": [_P] + [C.POINTER(C.c_double)] * 4,
    "mtgnn_grad_norm_ws_bytes": [C.POINTER(C.c_int64), _I32],
    "mtgnn_grad_norm": [C.POINTER(C.c_void_p), C.POINTER(C.c_int64), _I32, _P, _P, _SZ, _P],
    "mtgnn_prune_aux": [_P, _I64, _I32, _P],
    "mtgnn_cache_refresh": [_P, _I64, _P, _P, C.POINTER(Dims), _P, _P, _P],
    "mtgnn_adam_step": [C.POINTER(C.c_void_p)] * 5 + [C.POINTER(C.c_int64), _I32, C.POINTER(AdamConfig), _P],
    "mtgnn_mixed_batches": [_P, _I64, _I64, _P, _P, _P, _P, _SZ, _P],
    "mtgnn_workspace_bytes": [C.c_int, C.POINTER(Dims), _I64, _I64],
    "mtgnn_save_bytes": [C.c_int, C.POINTER(Dims), _I64, _I64],
    "mtgnn_status_string": [C.c_int],
    "mtgnn_last_error": [],
    "mtgnn_version": [],
    "mtgnn_timer_start": [C.c_char_p, C.c_int],
    "mtgnn_timer_stop": [C.POINTER(C.c_double), C.POINTER(C.c_int)],
}
_RES = {"mtgnn_workspace_bytes": _SZ, "mtgnn_save_bytes": _SZ, "mtgnn_grad_norm_ws_bytes": _SZ,
        "mtgnn_controller_destroy": None, "mtgnn_status_string": C.c_char_p,
        "mtgnn_last_error": C.c_char_p, "mtgnn_version": C.c_int}

_lib = None


def lib() -> C.CDLL:
    """Load the in-tree libmtgnn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MtgnnError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = _RES.get(name, C.c_int)
        _lib = L
    return _lib


def _check(status: int, name: str):
    if status != 0:
        L = lib()
        raise MtgnnError(f"{name}: {L.mtgnn_status_string(status).decode()} "
                         f"({L.mtgnn_last_error().decode()})")


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


_DT = {F32: torch.float32, BF16: torch.bfloat16}


def _ptr(t, dtype=None, name="tensor", optional=False):
    if t is None:
        if optional:
            return None
        raise MtgnnError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise MtgnnError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise MtgnnError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise MtgnnError(f"{name} must be contiguous")
    return C.c_void_p(t.data_ptr())


def _ws(ws):
    if ws is None:
        return None, 0
    return _ptr(ws, torch.uint8, "ws"), ws.numel()


def dims(n_nodes, d_mem, d_time, d_edge, d_attn, n_heads, k, dtype=F32) -> Dims:
    return Dims(int(n_nodes), int(d_mem), int(d_time), int(d_edge), int(d_attn), int(n_heads), int(k), int(dtype))


def batch(src, dst, t, eid=None, flags=None) -> Batch:
    n = int(src.numel())
    return Batch(n, _ptr(src, torch.int32, "src"), _ptr(dst, torch.int32, "dst"),
                 _ptr(eid, torch.int32, "eid", optional=True), _ptr(t, torch.float32, "t"),
                 _ptr(flags, torch.uint8, "flags", optional=True))


def workspace_bytes(op, d: Dims = None, max_rows=0, max_q=0) -> int:
    return int(lib().mtgnn_workspace_bytes(op, C.byref(d) if d is not None else None, int(max_rows), int(max_q)))


def save_bytes(op, d: Dims, max_rows=0, max_q=0) -> int:
    return int(lib().mtgnn_save_bytes(op, C.byref(d), int(max_rows), int(max_q)))


def alloc_bytes(n, device="cuda"):
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------- entry points

def mtgnn_build_queries(b: Batch, neg, q_node, q_t, n_q, ws=None, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_build_queries(C.byref(b), _ptr(neg, torch.int32, "neg"), _ptr(q_node, torch.int32, "q_node"),
                                     _ptr(q_t, torch.float32, "q_t"), _ptr(n_q, torch.int32, "n_q"), wp, wb,
                                     _stream(stream)), "mtgnn_build_queries")


def mtgnn_aggregate_last(b: Batch, n_nodes, uniq, winner, n_uniq, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_aggregate_last(C.byref(b), int(n_nodes), _ptr(uniq, torch.int32, "uniq"),
                                      _ptr(winner, torch.int32, "winner"), _ptr(n_uniq, torch.int32, "n_uniq"), wp, wb,
                                      _stream(stream)), "mtgnn_aggregate_last")


def mtgnn_build_messages(b: Batch, uniq, winner, n_rows, max_rows, memory, last_update, edge_feat, time_w, time_b,
                         d: Dims, msg, dt, stream=None):
    md = _DT[d.dtype]
    _check(lib().mtgnn_build_messages(C.byref(b), _ptr(uniq, torch.int32, "uniq"), _ptr(winner, torch.int32, "winner"),
                                      _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows),
                                      _ptr(memory, md, "memory"), _ptr(last_update, torch.float32, "last_update"),
                                      _ptr(edge_feat, torch.float32, "edge_feat", True),
                                      _ptr(time_w, torch.float32, "time_w"), _ptr(time_b, torch.float32, "time_b"),
                                      C.byref(d), _ptr(msg, md, "msg"), _ptr(dt, torch.float32, "dt"),
                                      _stream(stream)), "mtgnn_build_messages")


def mtgnn_gru_update(b: Batch, uniq, winner, n_rows, max_rows, msg, W_ih, W_hh, b_ih, b_hh, d: Dims, memory,
                     last_update, save, ws, stream=None):
    md = _DT[d.dtype]
    wp, wb = _ws(ws)
    _check(lib().mtgnn_gru_update(C.byref(b), _ptr(uniq, torch.int32, "uniq"), _ptr(winner, torch.int32, "winner"),
                                  _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows), _ptr(msg, md, "msg"),
                                  _ptr(W_ih, md, "W_ih"), _ptr(W_hh, md, "W_hh"), _ptr(b_ih, torch.float32, "b_ih"),
                                  _ptr(b_hh, torch.float32, "b_hh"), C.byref(d), _ptr(memory, md, "memory"),
                                  _ptr(last_update, torch.float32, "last_update"),
                                  _ptr(save, torch.uint8, "save", True), wp, wb, _stream(stream)), "mtgnn_gru_update")


def mtgnn_sample_recent(csr_off, csr_nbr, csr_t, csr_eid, n_nodes, q_node, q_t, n_q, max_q, k, out_nbr, out_t,
                        out_eid, stream=None):
    _check(lib().mtgnn_sample_recent(_ptr(csr_off, torch.int64, "csr_off"), _ptr(csr_nbr, torch.int32, "csr_nbr"),
                                     _ptr(csr_t, torch.float32, "csr_t"), _ptr(csr_eid, torch.int32, "csr_eid"),
                                     int(n_nodes), _ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"),
                                     _ptr(n_q, torch.int32, "n_q", True), int(max_q), int(k),
                                     _ptr(out_nbr, torch.int32, "out_nbr"), _ptr(out_t, torch.float32, "out_t"),
                                     _ptr(out_eid, torch.int32, "out_eid"), _stream(stream)), "mtgnn_sample_recent")


def attn_params(p: dict, d: Dims) -> AttnParams:
    md = _DT[d.dtype]
    return AttnParams(*[_ptr(p[n], md if n.startswith("W") else torch.float32, n) for n in _ATTN])


def attn_grads(g: dict) -> AttnGrads:
    return AttnGrads(*[_ptr(g[n], torch.float32, "d" + n) for n in _ATTN])


def mtgnn_temporal_attn(q_node, q_t, n_q, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b,
                        params: AttnParams, d: Dims, z, save, ws=None, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_temporal_attn(_ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"),
                                     _ptr(n_q, torch.int32, "n_q", True), int(max_q), _ptr(nbr, torch.int32, "nbr"),
                                     _ptr(nt, torch.float32, "nt"), _ptr(neid, torch.int32, "neid"),
                                     _ptr(memory, _DT[d.dtype], "memory"),
                                     _ptr(edge_feat, torch.float32, "edge_feat", True),
                                     _ptr(time_w, torch.float32, "time_w"), _ptr(time_b, torch.float32, "time_b"),
                                     C.byref(params), C.byref(d), _ptr(z, torch.float32, "z"),
                                     _ptr(save, torch.uint8, "save"), wp, wb, _stream(stream)), "mtgnn_temporal_attn")


def mtgnn_temporal_attn_prepare(nbr, n_q, max_q, params: AttnParams, time_w, time_b, d: Dims, save, ws=None,
                                stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_temporal_attn_prepare(_ptr(nbr, torch.int32, "nbr"), _ptr(n_q, torch.int32, "n_q", True),
                                             int(max_q), C.byref(params), _ptr(time_w, torch.float32, "time_w"),
                                             _ptr(time_b, torch.float32, "time_b"), C.byref(d),
                                             _ptr(save, torch.uint8, "save"), wp, wb, _stream(stream)),
           "mtgnn_temporal_attn_prepare")


def mtgnn_temporal_attn_prepare_weights(params: AttnParams, time_w, time_b, d: Dims, save, stream=None):
    _check(lib().mtgnn_temporal_attn_prepare_weights(C.byref(params), _ptr(time_w, torch.float32, "time_w"),
                                                     _ptr(time_b, torch.float32, "time_b"), C.byref(d),
                                                     _ptr(save, torch.uint8, "save"), _stream(stream)),
           "mtgnn_temporal_attn_prepare_weights")


def mtgnn_temporal_attn_prepare_weights_link(params: AttnParams, time_w, time_b, d: Dims, save, link: LinkParams,
                                             max_q, link_ws, stream=None):
    wp, wb = _ws(link_ws)
    _check(lib().mtgnn_temporal_attn_prepare_weights_link(C.byref(params), _ptr(time_w, torch.float32, "time_w"),
                                                          _ptr(time_b, torch.float32, "time_b"), C.byref(d),
                                                          _ptr(save, torch.uint8, "save"), C.byref(link), int(max_q),
                                                          wp, wb, _stream(stream)),
           "mtgnn_temporal_attn_prepare_weights_link")


def mtgnn_temporal_attn_prepare_slots(nbr, n_q, max_q, d: Dims, save, ws=None, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_temporal_attn_prepare_slots(_ptr(nbr, torch.int32, "nbr"), _ptr(n_q, torch.int32, "n_q", True),
                                                   int(max_q), C.byref(d), _ptr(save, torch.uint8, "save"), wp, wb,
                                                   _stream(stream)), "mtgnn_temporal_attn_prepare_slots")


def mtgnn_temporal_attn_prepared(q_node, q_t, n_q, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b,
                                 params: AttnParams, d: Dims, z, save, stream=None):
    _check(lib().mtgnn_temporal_attn_prepared(_ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"),
                                              _ptr(n_q, torch.int32, "n_q", True), int(max_q),
                                              _ptr(nbr, torch.int32, "nbr"), _ptr(nt, torch.float32, "nt"),
                                              _ptr(neid, torch.int32, "neid"), _ptr(memory, _DT[d.dtype], "memory"),
                                              _ptr(edge_feat, torch.float32, "edge_feat", True),
                                              _ptr(time_w, torch.float32, "time_w"),
                                              _ptr(time_b, torch.float32, "time_b"), C.byref(params), C.byref(d),
                                              _ptr(z, torch.float32, "z"), _ptr(save, torch.uint8, "save"),
                                              _stream(stream)), "mtgnn_temporal_attn_prepared")


def mtgnn_temporal_attn_bwd(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w, time_b,
                            params: AttnParams, d: Dims, grads: AttnGrads, d_mem, d_time_w, d_time_b, ws,
                            stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_temporal_attn_bwd(_ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"),
                                         _ptr(n_q, torch.int32, "n_q", True), int(max_q),
                                         _ptr(nbr, torch.int32, "nbr"), _ptr(nt, torch.float32, "nt"),
                                         _ptr(dz, torch.float32, "dz"), _ptr(save, torch.uint8, "save"),
                                         _ptr(uniq, torch.int32, "uniq", True), _ptr(n_rows, torch.int32, "n_rows", True),
                                         int(max_rows), _ptr(time_w, torch.float32, "time_w"),
                                         _ptr(time_b, torch.float32, "time_b"), C.byref(params), C.byref(d),
                                         C.byref(grads), _ptr(d_mem, torch.float32, "d_mem", True),
                                         _ptr(d_time_w, torch.float32, "d_time_w"),
                                         _ptr(d_time_b, torch.float32, "d_time_b"), wp, wb, _stream(stream)),
           "mtgnn_temporal_attn_bwd")


_hip = None


def _hip_rt():
    # the HIP runtime already loaded in this process (torch's, which the library resolves to as well)
    global _hip
    if _hip is None:
        _hip = C.CDLL("libamdhip64.so.7", mode=C.RTLD_GLOBAL)
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipStreamWaitEvent", "hipEventDestroy"):
            getattr(_hip, f).restype = C.c_int
    return _hip


def _hip_check(rc, what):
    if rc != 0:
        raise MtgnnError(f"{what} failed with HIP error {rc}")


class DeviceEvent:
    """An event that orders work between two streams of the current device.

    No timing, and a device-scope release when it is recorded (hipEventDisableSystemFence): both streams
    run on one GPU, so the system-scope fence of a default event, a cache write-back and invalidate that
    costs several microseconds per record, is not needed.  Methods follow torch.cuda.Event's:
    record(stream) and wait(stream) (the stream waits for the event)."""

    _FLAGS = 0x2 | 0x20000000   # hipEventDisableTiming | hipEventDisableSystemFence

    def __init__(self):
        self._rt = _hip_rt()
        h = C.c_void_p()
        _hip_check(self._rt.hipEventCreateWithFlags(C.byref(h), C.c_uint(self._FLAGS)), "hipEventCreateWithFlags")
        self.handle = h

    def record(self, stream=None):
        _hip_check(self._rt.hipEventRecord(self.handle, _stream(stream)), "hipEventRecord")

    def wait(self, stream=None):
        _hip_check(self._rt.hipStreamWaitEvent(_stream(stream), self.handle, C.c_uint(0)), "hipStreamWaitEvent")

    def __del__(self):
        try:   # may run at interpreter exit, after the runtime (or this module's globals) are gone
            if getattr(self, "handle", None) and self.handle.value:
                self._rt.hipEventDestroy(self.handle)
                self.handle = None
        except Exception:
            pass


def _event(e, name):
    if isinstance(e, DeviceEvent):
        return e.handle
    h = e.cuda_event if isinstance(e, torch.cuda.Event) else 0
    if not h:
        raise MtgnnError(f"{name}: a torch.cuda.Event that has been recorded once (so that it exists) is required")
    return C.c_void_p(h)


def mtgnn_temporal_attn_bwd_group(q_node, n_q, max_q, nbr, save, uniq, n_rows, max_rows, d: Dims, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_temporal_attn_bwd_group(
        _ptr(q_node, torch.int32, "q_node"), _ptr(n_q, torch.int32, "n_q", True), int(max_q),
        _ptr(nbr, torch.int32, "nbr"), _ptr(save, torch.uint8, "save"), _ptr(uniq, torch.int32, "uniq", True),
        _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows), C.byref(d), wp, wb, _stream(stream)),
        "mtgnn_temporal_attn_bwd_group")


def mtgnn_temporal_attn_bwd_overlap(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w,
                                    time_b, params: AttnParams, d: Dims, grads: AttnGrads, d_mem, d_time_w, d_time_b,
                                    ws, dmem_stream, fork, join, stream=None, grouped=False):
    """grouped=True calls mtgnn_temporal_attn_bwd_grouped (the grouping left in ws by
    mtgnn_temporal_attn_bwd_group on dmem_stream); there join may be None (the caller joins)."""
    wp, wb = _ws(ws)
    name = "mtgnn_temporal_attn_bwd_grouped" if grouped else "mtgnn_temporal_attn_bwd_overlap"
    _check(getattr(lib(), name)(
        _ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"), _ptr(n_q, torch.int32, "n_q", True),
        int(max_q), _ptr(nbr, torch.int32, "nbr"), _ptr(nt, torch.float32, "nt"), _ptr(dz, torch.float32, "dz"),
        _ptr(save, torch.uint8, "save"), _ptr(uniq, torch.int32, "uniq", True),
        _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows), _ptr(time_w, torch.float32, "time_w"),
        _ptr(time_b, torch.float32, "time_b"), C.byref(params), C.byref(d), C.byref(grads),
        _ptr(d_mem, torch.float32, "d_mem", True), _ptr(d_time_w, torch.float32, "d_time_w"),
        _ptr(d_time_b, torch.float32, "d_time_b"), wp, wb, _stream(stream), _stream(dmem_stream),
        _event(fork, "fork"), None if (grouped and join is None) else _event(join, "join")), name)


def mtgnn_gru_update_bwd(d_mem, save, msg, n_rows, max_rows, W_ih, W_hh, d: Dims, dW_ih, dW_hh, db_ih, db_hh,
                         dmsg_time, ws, stream=None):
    md = _DT[d.dtype]
    wp, wb = _ws(ws)
    _check(lib().mtgnn_gru_update_bwd(_ptr(d_mem, torch.float32, "d_mem"), _ptr(save, torch.uint8, "save"),
                                      _ptr(msg, md, "msg"), _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows),
                                      _ptr(W_ih, md, "W_ih"), _ptr(W_hh, md, "W_hh"), C.byref(d),
                                      _ptr(dW_ih, torch.float32, "dW_ih"), _ptr(dW_hh, torch.float32, "dW_hh"),
                                      _ptr(db_ih, torch.float32, "db_ih"), _ptr(db_hh, torch.float32, "db_hh"),
                                      _ptr(dmsg_time, torch.float32, "dmsg_time", True), wp, wb, _stream(stream)),
           "mtgnn_gru_update_bwd")


def link_params(p: dict) -> LinkParams:
    return LinkParams(*[_ptr(p[n], torch.float32, n) for n in _LINK])


def link_grads(g: dict) -> LinkGrads:
    return LinkGrads(*[_ptr(g[n], torch.float32, "d" + n) for n in _LINK])


def mtgnn_link_prepare_weights(params: LinkParams, d: Dims, max_q, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_link_prepare_weights(C.byref(params), C.byref(d), int(max_q), wp, wb, _stream(stream)),
           "mtgnn_link_prepare_weights")


def mtgnn_link_loss(z, n_q, max_q, params: LinkParams, d: Dims, loss, scores, dz, grads: LinkGrads, ws, stream=None,
                    dw_stream=None, fork=None, prepared=False):
    """dw_stream and fork given: mtgnn_link_loss_overlap (W_d1's gradient on dw_stream after fork).
    prepared: mtgnn_link_loss_prepared (ws holds mtgnn_link_prepare_weights' copies of params' W_d1)."""
    wp, wb = _ws(ws)
    args = (_ptr(z, torch.float32, "z"), _ptr(n_q, torch.int32, "n_q", True), int(max_q), C.byref(params), C.byref(d),
            _ptr(loss, torch.float32, "loss"), _ptr(scores, torch.float32, "scores", True), _ptr(dz, torch.float32, "dz"),
            C.byref(grads), wp, wb, _stream(stream))
    if prepared:
        ov = dw_stream is not None
        _check(lib().mtgnn_link_loss_prepared(*args, _stream(dw_stream) if ov else None,
                                              _event(fork, "fork") if ov else None), "mtgnn_link_loss_prepared")
    elif dw_stream is None:
        _check(lib().mtgnn_link_loss(*args), "mtgnn_link_loss")
    else:
        _check(lib().mtgnn_link_loss_overlap(*args, _stream(dw_stream), _event(fork, "fork")),
               "mtgnn_link_loss_overlap")


def mtgnn_build_messages_bwd(dmsg_time, dt, n_rows, max_rows, time_w, time_b, d: Dims, d_time_w, d_time_b, ws,
                             stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_build_messages_bwd(_ptr(dmsg_time, torch.float32, "dmsg_time"), _ptr(dt, torch.float32, "dt"),
                                          _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows),
                                          _ptr(time_w, torch.float32, "time_w"), _ptr(time_b, torch.float32, "time_b"),
                                          C.byref(d), _ptr(d_time_w, torch.float32, "d_time_w"),
                                          _ptr(d_time_b, torch.float32, "d_time_b"), wp, wb, _stream(stream)),
           "mtgnn_build_messages_bwd")


def mtgnn_build_messages_bwd_noalloc(dmsg_time, dt, n_rows, max_rows, time_w, time_b, d: Dims, d_time_w, d_time_b,
                                     stream=None):
    _check(lib().mtgnn_build_messages_bwd_noalloc(
        _ptr(dmsg_time, torch.float32, "dmsg_time"), _ptr(dt, torch.float32, "dt"),
        _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows), _ptr(time_w, torch.float32, "time_w"),
        _ptr(time_b, torch.float32, "time_b"), C.byref(d), _ptr(d_time_w, torch.float32, "d_time_w"),
        _ptr(d_time_b, torch.float32, "d_time_b"), _stream(stream)), "mtgnn_build_messages_bwd_noalloc")


def mtgnn_build_temporal_csr(src, dst, t, n_nodes, csr_off, csr_nbr, csr_t, csr_eid, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_build_temporal_csr(_ptr(src, torch.int32, "src"), _ptr(dst, torch.int32, "dst"),
                                          _ptr(t, torch.float32, "t"), int(src.numel()), int(n_nodes),
                                          _ptr(csr_off, torch.int64, "csr_off"), _ptr(csr_nbr, torch.int32, "csr_nbr"),
                                          _ptr(csr_t, torch.float32, "csr_t"), _ptr(csr_eid, torch.int32, "csr_eid"),
                                          wp, wb, _stream(stream)), "mtgnn_build_temporal_csr")


def mtgnn_dependency_scan(src, dst, owner, n_workers, batch, window, role, sync_bits, stream=None):
    _check(lib().mtgnn_dependency_scan(_ptr(src, torch.int32, "src"), _ptr(dst, torch.int32, "dst"), int(src.numel()),
                                       _ptr(owner, torch.int32, "owner"), int(owner.numel()), int(n_workers),
                                       int(batch), int(window), _ptr(role, torch.uint8, "role"),
                                       _ptr(sync_bits, torch.int32, "sync_bits"), _stream(stream)),
           "mtgnn_dependency_scan")


def mtgnn_mixed_batches(role, batch, eid_out, flags_out, batch_off, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_mixed_batches(_ptr(role, torch.uint8, "role"), int(role.numel()), int(batch),
                                     _ptr(eid_out, torch.int32, "eid_out"), _ptr(flags_out, torch.uint8, "flags_out"),
                                     _ptr(batch_off, torch.int32, "batch_off"), wp, wb, _stream(stream)),
           "mtgnn_mixed_batches")


def mtgnn_rnn_update(b: Batch, uniq, winner, n_rows, max_rows, msg, W_ih, W_hh, b_ih, b_hh, d: Dims, memory,
                     last_update, save, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_rnn_update(C.byref(b), _ptr(uniq, torch.int32, "uniq"), _ptr(winner, torch.int32, "winner"),
                                  _ptr(n_rows, torch.int32, "n_rows", True), int(max_rows), _ptr(msg, _DT[d.dtype], "msg"),
                                  _ptr(W_ih, _DT[d.dtype], "W_ih"), _ptr(W_hh, _DT[d.dtype], "W_hh"),
                                  _ptr(b_ih, torch.float32, "b_ih"), _ptr(b_hh, torch.float32, "b_hh"), C.byref(d),
                                  _ptr(memory, _DT[d.dtype], "memory"), _ptr(last_update, torch.float32, "last_update"),
                                  _ptr(save, torch.uint8, "save", True), wp, wb, _stream(stream)), "mtgnn_rnn_update")


def mtgnn_rnn_update_bwd(d_mem, save, msg, n_rows, max_rows, W_ih, W_hh, d: Dims, dW_ih, dW_hh, db_ih, db_hh,
                         dmsg_time, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_rnn_update_bwd(_ptr(d_mem, torch.float32, "d_mem"), _ptr(save, torch.uint8, "save"),
                                      _ptr(msg, _DT[d.dtype], "msg"), _ptr(n_rows, torch.int32, "n_rows", True),
                                      int(max_rows), _ptr(W_ih, _DT[d.dtype], "W_ih"), _ptr(W_hh, _DT[d.dtype], "W_hh"),
                                      C.byref(d), _ptr(dW_ih, torch.float32, "dW_ih"),
                                      _ptr(dW_hh, torch.float32, "dW_hh"), _ptr(db_ih, torch.float32, "db_ih"),
                                      _ptr(db_hh, torch.float32, "db_hh"),
                                      _ptr(dmsg_time, torch.float32, "dmsg_time", True), wp, wb, _stream(stream)),
           "mtgnn_rnn_update_bwd")


def mtgnn_time_projection(q_node, q_t, n_q, max_q, memory, last_update, W_p, b_p, time_scale, d: Dims, z,
                          stream=None):
    _check(lib().mtgnn_time_projection(_ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"),
                                       _ptr(n_q, torch.int32, "n_q", True), int(max_q),
                                       _ptr(memory, _DT[d.dtype], "memory"),
                                       _ptr(last_update, torch.float32, "last_update"), _ptr(W_p, torch.float32, "W_p"),
                                       _ptr(b_p, torch.float32, "b_p"), float(time_scale), C.byref(d),
                                       _ptr(z, torch.float32, "z"), _stream(stream)), "mtgnn_time_projection")


def mtgnn_time_projection_bwd(q_node, q_t, n_q, max_q, memory, last_update, W_p, b_p, time_scale, dz, uniq, n_rows,
                              max_rows, d: Dims, dW_p, db_p, d_mem, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_time_projection_bwd(
        _ptr(q_node, torch.int32, "q_node"), _ptr(q_t, torch.float32, "q_t"), _ptr(n_q, torch.int32, "n_q", True),
        int(max_q), _ptr(memory, _DT[d.dtype], "memory"), _ptr(last_update, torch.float32, "last_update"),
        _ptr(W_p, torch.float32, "W_p"), _ptr(b_p, torch.float32, "b_p"), float(time_scale),
        _ptr(dz, torch.float32, "dz"), _ptr(uniq, torch.int32, "uniq"), _ptr(n_rows, torch.int32, "n_rows", True),
        int(max_rows), C.byref(d), _ptr(dW_p, torch.float32, "dW_p"), _ptr(db_p, torch.float32, "db_p"),
        _ptr(d_mem, torch.float32, "d_mem"), wp, wb, _stream(stream)), "mtgnn_time_projection_bwd")


class Controller:
    """The library's host-side runtime controller (Eq. 6-9): decisions before a batch, observations after."""

    def __init__(self, alpha, beta, tau_g, tau_c, interval):
        h = C.c_void_p()
        _check(lib().mtgnn_controller_create(C.byref(ControllerConfig(alpha, beta, tau_g, tau_c, int(interval))),
                                             C.byref(h)), "mtgnn_controller_create")
        self._h = h

    def decide(self, r):
        """(boundary, S_r, H_r) before batch r."""
        b, sy, hv = C.c_int32(), C.c_int32(), C.c_int32()
        _check(lib().mtgnn_controller_decide(self._h, int(r), C.byref(b), C.byref(sy), C.byref(hv)),
               "mtgnn_controller_decide")
        return b.value, sy.value, hv.value

    def observe(self, grad_norm, batch_time):
        _check(lib().mtgnn_controller_observe(self._h, float(grad_norm), float(batch_time)),
               "mtgnn_controller_observe")

    def state(self):
        v = [C.c_double() for _ in range(4)]
        _check(lib().mtgnn_controller_state(self._h, *[C.byref(x) for x in v]), "mtgnn_controller_state")
        return tuple(x.value for x in v)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.mtgnn_controller_destroy(h)
            self._h = None


def _ptr_array(ts, dtype, name):
    arr = (C.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = _ptr(t, dtype, name).value
    return arr


def _sizes(ts):
    return (C.c_int64 * len(ts))(*[int(t.numel()) for t in ts])


def grad_norm_ws_bytes(tensors) -> int:
    return int(lib().mtgnn_grad_norm_ws_bytes(_sizes(tensors), len(tensors)))


def mtgnn_grad_norm(grads, norm, ws, stream=None):
    wp, wb = _ws(ws)
    _check(lib().mtgnn_grad_norm(_ptr_array(grads, torch.float32, "grad"), _sizes(grads), len(grads),
                                 _ptr(norm, torch.float64, "norm"), wp, wb, _stream(stream)), "mtgnn_grad_norm")


def mtgnn_prune_aux(flags, heavy, stream=None):
    _check(lib().mtgnn_prune_aux(_ptr(flags, torch.uint8, "flags"), int(flags.numel()), int(heavy), _stream(stream)),
           "mtgnn_prune_aux")


def mtgnn_cache_refresh(sync_bits, n_nodes, auth_memory, auth_lu, d: Dims, memory, last_update, stream=None):
    _check(lib().mtgnn_cache_refresh(_ptr(sync_bits, torch.int32, "sync_bits"), int(n_nodes),
                                     _ptr(auth_memory, None, "auth_memory"), _ptr(auth_lu, torch.float32, "auth_lu"),
                                     C.byref(d), _ptr(memory, None, "memory"),
                                     _ptr(last_update, torch.float32, "last_update"), _stream(stream)),
           "mtgnn_cache_refresh")


def mtgnn_adam_step(params, grads, m, v, shadow, lr, beta1, beta2, eps, t, stream=None):
    """params, grads, m, v: lists of float32 tensors; shadow: None or a list of (None | bf16 tensor)."""
    sh = None
    if shadow is not None:
        sh = (C.c_void_p * len(shadow))()
        for i, x in enumerate(shadow):
            sh[i] = None if x is None else _ptr(x, torch.bfloat16, "shadow").value
    _check(lib().mtgnn_adam_step(_ptr_array(params, torch.float32, "param"), _ptr_array(grads, torch.float32, "grad"),
                                 _ptr_array(m, torch.float32, "m"), _ptr_array(v, torch.float32, "v"), sh,
                                 _sizes(params), len(params), C.byref(AdamConfig(lr, beta1, beta2, eps, int(t))),
                                 _stream(stream)), "mtgnn_adam_step")


def timer_start(kernel: str, max_launches: int):
    """Arm the library's launch timer for `kernel` (instrumentation)."""
    _check(lib().mtgnn_timer_start(kernel.encode(), int(max_launches)), "mtgnn_timer_start")


def timer_stop():
    """Disarm the timer; returns (summed milliseconds, number of timed launches)."""
    ms, n = C.c_double(0.0), C.c_int(0)
    _check(lib().mtgnn_timer_stop(C.byref(ms), C.byref(n)), "mtgnn_timer_stop")
    return ms.value, n.value
