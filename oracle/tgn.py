"""The memory-based TGNN batch step, written out plainly (test infrastructure only).

The paper (Section III-A, Eq. 1-2) fixes the chronological semantics: each
event e_k = (u_k, v_k, t_k, x_k) produces one message per endpoint from the
endpoint memories just before t_k, and each endpoint memory is updated from
its message.  It leaves Message/Update abstract and names TGN as the model
(Section VII-A).  This module takes the TGN reading of those functions:

* message   = [m_node || m_partner || cos(w * dt + b) || x_k],
              dt = t_k - last_update[node];
* aggregate = the most recent message per node (largest (t, eid, role));
* update    = a GRU cell (PyTorch gate order r, z, n) writing the memory row
              and last_update[node] = t of the winning message;
* embedding = one layer of multi-head temporal attention over the k most
              recent earlier neighbours, followed by a 2-layer merge MLP.

The mixed-batch masks come from Definition 2 and Eq. 10-13: replay events
(bit 0) advance memory but get no query and no loss; pruned events (bit 1)
are removed before the step (they stay in the temporal adjacency, which is
built offline).

Precision modes (``prec``):
* ``"f64"``  -- float64 everywhere, no storage rounding (used for algebraic
                and finite-difference pins);
* ``"f32"``  -- memory stored as float32; dt and the cosine argument rounded
                to float32 exactly as the GPU computes them (fp32 multiply,
                then fp32 add, no fused multiply-add); arithmetic in float64;
* ``"bf16"`` -- as f32, plus bfloat16 storage of memory, weights and every
                matrix-product input (messages, projection inputs, the
                attention output, the merge-layer inputs).
"""

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

from .bf16 import round_bf16

F32, F64 = np.float32, np.float64

WEIGHTS = ("W_ih", "W_hh", "W_q", "W_k", "W_v", "W_o", "W_1", "W_2")
BIASES = ("b_ih", "b_hh", "b_q", "b_k", "b_v", "b_o", "b_1", "b_2")
ATTN_PARAMS = ("W_q", "b_q", "W_k", "b_k", "W_v", "b_v", "W_o", "b_o", "W_1", "b_1", "W_2", "b_2")
GRU_PARAMS = ("W_ih", "W_hh", "b_ih", "b_hh")


# --------------------------------------------------------------------------- precision

class Prec:
    """Storage and rounding rules of one precision mode."""

    def __init__(self, mode: str):
        if mode not in ("f64", "f32", "bf16"):
            raise ValueError(mode)
        self.mode = mode

    @property
    def mem_dtype(self):
        return F64 if self.mode == "f64" else F32

    def store(self, x) -> np.ndarray:
        """Round a computed value to the memory table's storage type."""
        if self.mode == "f64":
            return np.asarray(x, F64)
        x32 = np.asarray(x, F64).astype(F32)
        return round_bf16(x32) if self.mode == "bf16" else x32

    def pack(self, x) -> np.ndarray:
        """A value as it enters a matrix product (bf16 mode rounds it)."""
        if self.mode == "bf16":
            return round_bf16(np.asarray(x, F64).astype(F32)).astype(F64)
        return np.asarray(x, F64)

    def weight(self, x) -> np.ndarray:
        return self.pack(x)

    def delta(self, t, t_ref) -> np.ndarray:
        """Elapsed time t - t_ref (float32 subtraction outside f64 mode)."""
        if self.mode == "f64":
            return np.asarray(t, F64) - np.asarray(t_ref, F64)
        return (np.asarray(t, F32) - np.asarray(t_ref, F32)).astype(F32)

    def time_arg(self, dt, w, b) -> np.ndarray:
        """Cosine argument w_j * dt + b_j, broadcast over a trailing d_t axis."""
        dt = np.asarray(dt)
        if self.mode == "f64":
            return dt.astype(F64)[..., None] * np.asarray(w, F64) + np.asarray(b, F64)
        prod = dt.astype(F32)[..., None] * np.asarray(w, F32)   # one fp32 rounding
        return (prod + np.asarray(b, F32)).astype(F32)            # second fp32 rounding


def time_encode(prec: Prec, dt, w, b) -> np.ndarray:
    """phi(dt)_j = cos(w_j dt + b_j), cosine evaluated in float64 on the (rounded) argument."""
    return np.cos(prec.time_arg(dt, w, b).astype(F64))


def _sigmoid(x):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


# --------------------------------------------------------------------------- batches

def active_mask(flags, n) -> np.ndarray:
    """Events that enter the memory phase: every event not pruned (Eq. 11)."""
    if flags is None:
        return np.ones(n, bool)
    return (np.asarray(flags) & 2) == 0


def target_mask(flags, n) -> np.ndarray:
    """Target events (Eq. 12): neither replayed nor pruned."""
    if flags is None:
        return np.ones(n, bool)
    return (np.asarray(flags) & 3) == 0


# --------------------------------------------------------------------------- memory phase

def select_last(src, dst, t, eid, flags=None):
    """Most-recent message per node.

    Every non-pruned event i yields two messages: role 0 for node src[i] and
    role 1 for node dst[i].  A node's winner is its message with the largest
    key (t, eid, role), t compared as float32.  Returns ``uniq`` (touched
    nodes, ascending) and ``winner`` (2*i + role of each node's winner).
    """
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    n = src.shape[0]
    idx = np.nonzero(active_mask(flags, n))[0]
    nodes = np.concatenate([src[idx], dst[idx]])
    ev = np.concatenate([idx, idx])
    role = np.concatenate([np.zeros(idx.size, np.int64), np.ones(idx.size, np.int64)])
    tt = np.asarray(t, F32)[ev]
    ee = np.asarray(eid, np.int64)[ev]
    order = np.lexsort((role, ee, tt, nodes))      # last key is primary
    nodes_s = nodes[order]
    is_last = np.ones(nodes_s.size, bool)
    if nodes_s.size:
        is_last[:-1] = nodes_s[1:] != nodes_s[:-1]
    uniq = nodes_s[is_last]
    winner = (2 * ev + role)[order][is_last]
    return uniq.astype(np.int64), winner.astype(np.int64)


def build_messages(prec: Prec, dims, src, dst, t, eid, uniq, winner, mem, lu, x_all, time_w, time_b):
    """Messages of the winning events (Eq. 1), read from the pre-batch state.

    Row r: [M[node] || M[partner] || phi(t - LU[node]) || x_eid], node = uniq[r].
    Returns (msg float64 [U, D_msg], dt [U] in the delta type).
    """
    ev = winner // 2
    role = winner % 2
    node = np.where(role == 0, np.asarray(src)[ev], np.asarray(dst)[ev]).astype(np.int64)
    assert np.array_equal(node, uniq)
    partner = np.where(role == 0, np.asarray(dst)[ev], np.asarray(src)[ev]).astype(np.int64)
    tw = np.asarray(t, F32)[ev]
    dt = prec.delta(tw, np.asarray(lu)[node])
    parts = [np.asarray(mem[node], F64), np.asarray(mem[partner], F64),
             prec.pack(time_encode(prec, dt, time_w, time_b))]
    if dims.d_edge > 0:
        parts.append(prec.pack(np.asarray(x_all[np.asarray(eid)[ev]], F64)))
    msg = np.concatenate(parts, axis=1) if len(uniq) else np.zeros((0, dims.d_msg))
    return msg, dt


def gru_cell(x, h, W_ih, W_hh, b_ih, b_hh):
    """GRU cell, gate order (r, z, n):

    r = sigmoid(W_ir x + b_ir + W_hr h + b_hr)
    z = sigmoid(W_iz x + b_iz + W_hz h + b_hz)
    n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
    h' = (1 - z) * n + z * h
    Returns h' and the saved gates (r, z, n, W_hn h + b_hn).
    """
    dm = h.shape[1]
    gi = x @ W_ih.T + b_ih
    gh = h @ W_hh.T + b_hh
    r = _sigmoid(gi[:, :dm] + gh[:, :dm])
    z = _sigmoid(gi[:, dm:2 * dm] + gh[:, dm:2 * dm])
    ghn = gh[:, 2 * dm:]
    n = np.tanh(gi[:, 2 * dm:] + r * ghn)
    return (1.0 - z) * n + z * h, (r, z, n, ghn)


@dataclass
class MemoryPhase:
    uniq: np.ndarray
    winner: np.ndarray
    msg: np.ndarray          # float64 [U, D_msg] (as packed)
    dt: np.ndarray           # [U]
    h_old: np.ndarray        # float64 [U, d_m]
    gates: tuple             # (r, z, n, ghn) float64 [U, d_m] each
    h_new: np.ndarray        # float64 [U, d_m] before storage rounding
    mem: np.ndarray          # updated memory table (storage dtype)
    lu: np.ndarray           # updated last_update (float32)


def memory_phase(prec: Prec, dims, batch: dict, mem, lu, x_all, params) -> MemoryPhase:
    """Eq. 1-2 for one batch: select, build messages, GRU, write back."""
    src, dst, t, eid = batch["src"], batch["dst"], batch["t"], batch["eid"]
    uniq, winner = select_last(src, dst, t, eid, batch.get("flags"))
    msg, dt = build_messages(prec, dims, src, dst, t, eid, uniq, winner, mem, lu, x_all,
                             params["time_w"], params["time_b"])
    h_old = np.asarray(mem[uniq], F64)
    h_new, gates = gru_cell(msg, h_old, prec.weight(params["W_ih"]), prec.weight(params["W_hh"]),
                            np.asarray(params["b_ih"], F64), np.asarray(params["b_hh"], F64))
    mem2 = np.array(mem, copy=True)
    lu2 = np.array(lu, copy=True)
    if len(uniq):
        mem2[uniq] = prec.store(h_new)
        lu2[uniq] = np.asarray(t, F32)[winner // 2]
    return MemoryPhase(uniq, winner, msg, dt, h_old, gates, h_new, mem2, lu2)


# --------------------------------------------------------------------------- temporal adjacency + sampling

@dataclass
class Adjacency:
    """Per-node event lists sorted by (t, eid, role) ascending."""
    off: np.ndarray   # int64 [N+1]
    nbr: np.ndarray   # int64 [2E]
    t: np.ndarray     # float32 [2E]
    eid: np.ndarray   # int64 [2E]


def build_adjacency(src, dst, t, n_nodes) -> Adjacency:
    """Both directions of every event of the stream (targets, replay and pruned).

    Event e contributes (node=src, nbr=dst, role 0) and (node=dst, nbr=src,
    role 1); a self-loop therefore appears twice.  Event ids are stream
    positions.
    """
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    E = src.shape[0]
    eid = np.arange(E, dtype=np.int64)
    node = np.concatenate([src, dst])
    nbr = np.concatenate([dst, src])
    tt = np.concatenate([np.asarray(t, F32), np.asarray(t, F32)])
    ee = np.concatenate([eid, eid])
    role = np.concatenate([np.zeros(E, np.int8), np.ones(E, np.int8)])
    order = np.lexsort((role, ee, tt, node))
    counts = np.bincount(node, minlength=n_nodes)
    off = np.zeros(n_nodes + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    return Adjacency(off, nbr[order], tt[order], ee[order])


def build_adjacency_for(src, dst, t, n_nodes, nodes) -> Adjacency:
    """The lists of ``nodes`` only, as ``build_adjacency`` orders them; every other list is empty.

    Only events with an endpoint in ``nodes`` are read into the lists, so a
    few queried nodes of a very long stream are cheap to serve.
    """
    want = np.zeros(n_nodes, bool)
    want[np.asarray(nodes, np.int64)] = True
    e_src = np.nonzero(want[src])[0]
    e_dst = np.nonzero(want[dst])[0]
    node = np.concatenate([np.asarray(src)[e_src], np.asarray(dst)[e_dst]]).astype(np.int64)
    nbr = np.concatenate([np.asarray(dst)[e_src], np.asarray(src)[e_dst]]).astype(np.int64)
    tt = np.concatenate([np.asarray(t, F32)[e_src], np.asarray(t, F32)[e_dst]])
    ee = np.concatenate([e_src, e_dst]).astype(np.int64)
    role = np.concatenate([np.zeros(e_src.size, np.int8), np.ones(e_dst.size, np.int8)])
    order = np.lexsort((role, ee, tt, node))
    counts = np.bincount(node, minlength=n_nodes)
    off = np.zeros(n_nodes + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    return Adjacency(off, nbr[order], tt[order], ee[order])


def sample_recent(adj: Adjacency, q_node, q_t, k: int):
    """The k most recent neighbours strictly before each query time.

    For query (n, tau): among n's entries with t < tau (float32 compare), the
    k largest by (t, eid, role), newest first.  Missing slots are padded with
    nbr = -1, t = 0, eid = -1.
    """
    q_node = np.asarray(q_node, np.int64)
    q_t = np.asarray(q_t, F32)
    Q = q_node.shape[0]
    nbr = np.full((Q, k), -1, np.int64)
    nt = np.zeros((Q, k), F32)
    neid = np.full((Q, k), -1, np.int64)
    for qi in range(Q):
        lo, hi = adj.off[q_node[qi]], adj.off[q_node[qi] + 1]
        end = lo + np.searchsorted(adj.t[lo:hi], q_t[qi], side="left")
        start = max(lo, end - k)
        m = end - start
        if m:
            sl = slice(start, end)
            nbr[qi, :m] = adj.nbr[sl][::-1]
            nt[qi, :m] = adj.t[sl][::-1]
            neid[qi, :m] = adj.eid[sl][::-1]
    return nbr, nt, neid


def sample_recent_bruteforce(src, dst, t, q_node, q_t, k: int):
    """Sampling by direct scan of the whole stream (tiny inputs only)."""
    Q = len(q_node)
    nbr = np.full((Q, k), -1, np.int64)
    nt = np.zeros((Q, k), F32)
    neid = np.full((Q, k), -1, np.int64)
    for qi in range(Q):
        n, tau = int(q_node[qi]), F32(q_t[qi])
        cand = []
        for e in range(len(src)):
            te = F32(t[e])
            if not te < tau:
                continue
            if int(src[e]) == n:
                cand.append((te, e, 0, int(dst[e])))
            if int(dst[e]) == n:
                cand.append((te, e, 1, int(src[e])))
        cand.sort(reverse=True)
        for s, (te, e, _r, v) in enumerate(cand[:k]):
            nbr[qi, s], nt[qi, s], neid[qi, s] = v, te, e
    return nbr, nt, neid


# --------------------------------------------------------------------------- embedding

def queries(batch: dict):
    """Query list of a batch: src || dst || neg of its target events, each at the event time."""
    n = len(batch["src"])
    tar = np.nonzero(target_mask(batch.get("flags"), n))[0]
    q_node = np.concatenate([np.asarray(batch["src"])[tar], np.asarray(batch["dst"])[tar],
                             np.asarray(batch["neg"])[tar]]).astype(np.int64)
    q_t = np.tile(np.asarray(batch["t"], F32)[tar], 3)
    return q_node, q_t, int(tar.size)


@dataclass
class AttnSave:
    q_node: np.ndarray
    q_t: np.ndarray
    nbr: np.ndarray
    nt: np.ndarray
    neid: np.ndarray
    valid: np.ndarray
    hq: np.ndarray
    q_in: np.ndarray
    q: np.ndarray
    kv_in: np.ndarray
    dts: np.ndarray
    K: np.ndarray
    V: np.ndarray
    p: np.ndarray
    attn: np.ndarray
    o: np.ndarray
    m_in: np.ndarray
    m1: np.ndarray
    a1: np.ndarray
    z: np.ndarray
    relu1: np.ndarray        # the ReLU decisions of m1 (m1 > 0 unless flipped)


def attention_fwd(prec: Prec, dims, mem, x_all, params, q_node, q_t, nbr, nt, neid, flip_m1=None) -> AttnSave:
    """One layer of multi-head temporal attention over the sampled neighbours.

    q   = W_q [M[q] || phi(0)] + b_q
    K_j = W_k [M[n_j] || x_{e_j} || phi(tau - t_j)] + b_k,  V_j likewise with W_v
    per head h (d_a/H columns): p = softmax_j(q_h . K_jh / sqrt(d_a/H)) over valid j,
    attn_h = sum_j p_j V_jh (zero when no neighbour is valid)
    o = W_o attn + b_o;  z = W_2 relu(W_1 [o || M[q]] + b_1) + b_2

    ``flip_m1`` (boolean, the shape of m1) inverts chosen ReLU decisions; a caller uses it only
    where m1 lies within rounding distance of zero, where either decision is a valid result.
    """
    dm, de, da, H = dims.d_mem, dims.d_edge, dims.d_attn, dims.n_heads
    dh = da // H
    Q, k = np.shape(nbr)
    W = {n: prec.weight(params[n]) for n in ("W_q", "W_k", "W_v", "W_o", "W_1", "W_2")}
    b = {n: np.asarray(params[n], F64) for n in ("b_q", "b_k", "b_v", "b_o", "b_1", "b_2")}
    tw, tb = params["time_w"], params["time_b"]

    hq = np.asarray(mem[q_node], F64)
    phi0 = prec.pack(time_encode(prec, np.zeros(1, F32), tw, tb))[0]
    q_in = np.concatenate([hq, np.broadcast_to(phi0, (Q, phi0.size))], axis=1)
    q = q_in @ W["W_q"].T + b["b_q"]

    valid = np.asarray(nbr) >= 0
    vf = valid[..., None].astype(F64)
    hn = np.asarray(mem[np.where(valid, nbr, 0)], F64) * vf
    dts = np.where(valid, prec.delta(np.asarray(q_t, F32)[:, None], nt), 0).astype(
        F64 if prec.mode == "f64" else F32)
    phin = prec.pack(time_encode(prec, dts, tw, tb)) * vf
    parts = [hn]
    if de > 0:
        parts.append(prec.pack(np.asarray(x_all[np.where(valid, neid, 0)], F64)) * vf)
    parts.append(phin)
    kv_in = np.concatenate(parts, axis=2)
    K = kv_in @ W["W_k"].T + b["b_k"]
    V = kv_in @ W["W_v"].T + b["b_v"]

    qh = q.reshape(Q, H, dh)
    Kh = K.reshape(Q, k, H, dh)
    Vh = V.reshape(Q, k, H, dh)
    s = np.einsum("qhd,qkhd->qhk", qh, Kh) / np.sqrt(dh)
    vmask = valid[:, None, :]
    s = np.where(vmask, s, -np.inf)
    smax = np.max(s, axis=2, keepdims=True) if k else np.zeros((Q, H, 1))
    smax = np.where(np.isfinite(smax), smax, 0.0)
    e = np.where(vmask, np.exp(s - smax), 0.0)
    den = e.sum(axis=2, keepdims=True)
    p = np.where(den > 0, e / np.where(den > 0, den, 1.0), 0.0)
    attn = np.einsum("qhk,qkhd->qhd", p, Vh).reshape(Q, da)
    attn_p = prec.pack(attn)
    o = attn_p @ W["W_o"].T + b["b_o"]
    m_in = np.concatenate([prec.pack(o), hq], axis=1)
    m1 = m_in @ W["W_1"].T + b["b_1"]
    relu1 = m1 > 0
    if flip_m1 is not None:
        relu1 = relu1 ^ flip_m1
    a1 = prec.pack(np.where(relu1, m1, 0.0))
    z = a1 @ W["W_2"].T + b["b_2"]
    return AttnSave(np.asarray(q_node), np.asarray(q_t), np.asarray(nbr), np.asarray(nt),
                    np.asarray(neid), valid, hq, q_in, q, kv_in, dts, K, V, p, attn_p, o,
                    m_in, m1, a1, z, relu1)


@dataclass
class AttnGrads:
    grads: dict                  # d of every attention parameter (float64)
    dhq: np.ndarray              # [Q, d_m]  d loss / d M[q_node] per query occurrence
    dhn: np.ndarray              # [Q, k, d_m] d loss / d M[nbr] per neighbour slot
    d_time_w: np.ndarray
    d_time_b: np.ndarray


def attention_bwd(prec: Prec, dims, params, sv: AttnSave, dz) -> AttnGrads:
    """Reverse-mode derivative of ``attention_fwd`` for an output gradient dz."""
    dm, de, dt_, da, H = dims.d_mem, dims.d_edge, dims.d_time, dims.d_attn, dims.n_heads
    dh = da // H
    Q, k = sv.nbr.shape
    W = {n: prec.weight(params[n]) for n in ("W_q", "W_k", "W_v", "W_o", "W_1", "W_2")}
    tw, tb = params["time_w"], params["time_b"]
    dz = np.asarray(dz, F64)
    g = {}
    # z = a1 W_2^T + b_2
    g["W_2"] = dz.T @ sv.a1
    g["b_2"] = dz.sum(0)
    dm1 = (dz @ W["W_2"]) * sv.relu1
    # m1 = m_in W_1^T + b_1
    g["W_1"] = dm1.T @ sv.m_in
    g["b_1"] = dm1.sum(0)
    dm_in = dm1 @ W["W_1"]
    do = dm_in[:, :da]
    dhq = dm_in[:, da:].copy()
    # o = attn W_o^T + b_o
    g["W_o"] = do.T @ sv.attn
    g["b_o"] = do.sum(0)
    dattn = (do @ W["W_o"]).reshape(Q, H, dh)
    # attn_h = sum_j p_j V_jh
    Kh = sv.K.reshape(Q, k, H, dh)
    Vh = sv.V.reshape(Q, k, H, dh)
    qh = sv.q.reshape(Q, H, dh)
    dV = np.einsum("qhk,qhd->qkhd", sv.p, dattn).reshape(Q, k, da)
    dp = np.einsum("qhd,qkhd->qhk", dattn, Vh)
    ds = sv.p * (dp - (sv.p * dp).sum(axis=2, keepdims=True))
    scale = 1.0 / np.sqrt(dh)
    dq = (np.einsum("qhk,qkhd->qhd", ds, Kh) * scale).reshape(Q, da)
    dK = (np.einsum("qhk,qhd->qkhd", ds, qh) * scale).reshape(Q, k, da)
    # q = q_in W_q^T + b_q
    g["W_q"] = dq.T @ sv.q_in
    g["b_q"] = dq.sum(0)
    dq_in = dq @ W["W_q"]
    dhq += dq_in[:, :dm]
    dphi0 = dq_in[:, dm:].sum(0)
    # K, V = kv_in W^T + b over valid slots (invalid slots carry zero gradient)
    kv = sv.kv_in.reshape(Q * k, sv.kv_in.shape[-1])
    g["W_k"] = dK.reshape(Q * k, da).T @ kv
    g["b_k"] = dK.reshape(Q * k, da).sum(0)
    g["W_v"] = dV.reshape(Q * k, da).T @ kv
    g["b_v"] = dV.reshape(Q * k, da).sum(0)
    dkv = dK @ W["W_k"] + dV @ W["W_v"]
    vf = sv.valid[..., None].astype(F64)
    dhn = dkv[..., :dm] * vf
    dphin = dkv[..., dm + de:] * vf
    # phi(dt) = cos(arg), arg = w dt + b
    arg0 = prec.time_arg(np.zeros(1, F32), tw, tb).astype(F64)[0]
    argn = prec.time_arg(sv.dts, tw, tb).astype(F64)
    s0 = -np.sin(arg0)
    sn = -np.sin(argn) * vf
    d_time_b = dphi0 * s0 + (dphin * sn).sum(axis=(0, 1))
    d_time_w = (dphin * sn * np.asarray(sv.dts, F64)[..., None]).sum(axis=(0, 1))
    return AttnGrads(g, dhq, dhn, d_time_w, d_time_b)


def memory_grad(uniq, q_node, nbr, dhq, dhn) -> np.ndarray:
    """d loss / d M' for the rows updated in this step (rows aligned with ``uniq``).

    Sums the gradient of every occurrence of an updated node, as a query and
    as a valid neighbour slot.  Rows that were not updated get nothing: the
    memory table itself is not differentiated across steps.
    """
    uniq = np.asarray(uniq, np.int64)
    U = uniq.size
    dm = dhq.shape[1] if dhq.ndim == 2 else dhn.shape[-1]
    out = np.zeros((U, dm), F64)
    if U == 0:
        return out

    def rows_of(nodes):
        pos = np.searchsorted(uniq, nodes)
        pos = np.minimum(pos, U - 1)
        return np.where(uniq[pos] == nodes, pos, -1)

    rq = rows_of(np.asarray(q_node, np.int64))
    m = rq >= 0
    np.add.at(out, rq[m], dhq[m])
    nb = np.asarray(nbr, np.int64).reshape(-1)
    rn = np.where(nb >= 0, rows_of(nb), -1)
    m = rn >= 0
    np.add.at(out, rn[m], dhn.reshape(-1, dm)[m])
    return out


def gru_bwd(dh_new, x, h_old, gates, W_ih, W_hh):
    """Reverse of ``gru_cell`` w.r.t. its weights and its input x (h_old is detached)."""
    r, z, n, ghn = gates
    dn = dh_new * (1.0 - z)
    dzg = dh_new * (h_old - n)
    dn_pre = dn * (1.0 - n * n)
    dr_pre = dn_pre * ghn * r * (1.0 - r)
    dz_pre = dzg * z * (1.0 - z)
    dgi = np.concatenate([dr_pre, dz_pre, dn_pre], axis=1)
    dgh = np.concatenate([dr_pre, dz_pre, dn_pre * r], axis=1)
    grads = {"W_ih": dgi.T @ x, "W_hh": dgh.T @ h_old, "b_ih": dgi.sum(0), "b_hh": dgh.sum(0)}
    return grads, dgi @ W_ih


def message_bwd(prec: Prec, dims, dx, dt, time_w, time_b):
    """Time-encoder gradient from the phi slice of the message gradient."""
    dm, dt_ = dims.d_mem, dims.d_time
    dphi = dx[:, 2 * dm:2 * dm + dt_]
    s = -np.sin(prec.time_arg(dt, time_w, time_b).astype(F64))
    return (dphi * s * np.asarray(dt, F64)[:, None]).sum(0), (dphi * s).sum(0)


# --------------------------------------------------------------------------- link prediction and the masked loss

def _softplus(x):
    """log(1 + e^x), evaluated without overflow."""
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


@dataclass
class LinkLoss:
    loss: float              # the masked batch loss (Eq. 13)
    s_pos: np.ndarray        # [n_tar] score of (src, dst)
    s_neg: np.ndarray        # [n_tar] score of (src, neg)
    dz: np.ndarray           # [3 n_tar, d_a] d loss / d z in the query layout
    grads: dict              # W_d1, b_d1, W_d2, b_d2
    pre_pos: np.ndarray      # [n_tar, d_a] hidden pre-activations of the true edges
    pre_neg: np.ndarray      # [n_tar, d_a] ... and of the negative edges


def link_loss(params, z, n_tar: int, flip_pos=None, flip_neg=None) -> LinkLoss:
    """Masked link-prediction loss of one batch (Eq. 12-13) and its gradient.

    z holds the embeddings of the batch's queries: src of the target events,
    then their dst, then their negatives (n_tar rows each; replayed and pruned
    events have none, which is the target mask of Eq. 12).  The edge score is
    TGN's link predictor: s(a, b) = W_d2 relu(W_d1 [z_a || z_b] + b_d1) + b_d2.
    The edge prediction loss of a target event is the binary cross-entropy of
    its true edge (label 1) and of its negative edge (label 0):
        l = -log sigmoid(s(src, dst)) - log(1 - sigmoid(s(src, neg)))
          = softplus(-s_pos) + softplus(s_neg),
    and the batch loss is the mean over target events, 0 without any (Eq. 13).
    Float64 throughout; the decoder's weights are float32 values.  ``flip_pos`` / ``flip_neg``
    (boolean, [n_tar, d_a]) invert chosen ReLU decisions, as ``attention_fwd``'s ``flip_m1``.
    """
    W1 = np.asarray(params["W_d1"], F64)
    b1 = np.asarray(params["b_d1"], F64)
    W2 = np.asarray(params["W_d2"], F64)
    b2 = np.asarray(params["b_d2"], F64)
    z = np.asarray(z, F64)
    n = int(n_tar)
    da = W1.shape[0]
    zs, zd, zn = z[:n], z[n:2 * n], z[2 * n:3 * n]
    x_pos = np.concatenate([zs, zd], axis=1)
    x_neg = np.concatenate([zs, zn], axis=1)
    pre_pos = x_pos @ W1.T + b1
    pre_neg = x_neg @ W1.T + b1
    on_pos = pre_pos > 0 if flip_pos is None else (pre_pos > 0) ^ flip_pos
    on_neg = pre_neg > 0 if flip_neg is None else (pre_neg > 0) ^ flip_neg
    h_pos = np.where(on_pos, pre_pos, 0.0)
    h_neg = np.where(on_neg, pre_neg, 0.0)
    s_pos = (h_pos @ W2.T + b2)[:, 0]
    s_neg = (h_neg @ W2.T + b2)[:, 0]
    if n == 0:
        g = {"W_d1": np.zeros_like(W1), "b_d1": np.zeros_like(b1), "W_d2": np.zeros_like(W2),
             "b_d2": np.zeros_like(b2)}
        return LinkLoss(0.0, s_pos, s_neg, np.zeros((0, da)), g, pre_pos, pre_neg)
    loss = float(np.mean(_softplus(-s_pos) + _softplus(s_neg)))
    # d loss / d score: (sigmoid(s) - label) / n
    ds_pos = (_sigmoid(s_pos) - 1.0) / n
    ds_neg = _sigmoid(s_neg) / n
    dh_pos = ds_pos[:, None] * W2[0] * on_pos
    dh_neg = ds_neg[:, None] * W2[0] * on_neg
    g = {"W_d2": (ds_pos @ h_pos + ds_neg @ h_neg)[None, :],
         "b_d2": np.array([ds_pos.sum() + ds_neg.sum()]),
         "W_d1": dh_pos.T @ x_pos + dh_neg.T @ x_neg,
         "b_d1": dh_pos.sum(0) + dh_neg.sum(0)}
    dx_pos = dh_pos @ W1
    dx_neg = dh_neg @ W1
    dz = np.concatenate([dx_pos[:, :da] + dx_neg[:, :da], dx_pos[:, da:], dx_neg[:, da:]], axis=0)
    return LinkLoss(loss, s_pos, s_neg, dz, g, pre_pos, pre_neg)


# --------------------------------------------------------------------------- one step

@dataclass
class StepResult:
    mp: MemoryPhase
    q_node: np.ndarray
    q_t: np.ndarray
    n_tar: int
    nbr: np.ndarray
    nt: np.ndarray
    neid: np.ndarray
    attn: AttnSave
    dz: np.ndarray
    ag: AttnGrads
    d_mem: np.ndarray
    grads: dict = field(default_factory=dict)   # every parameter gradient (float64)
    link: Optional[LinkLoss] = None


def step(prec: Prec, dims, mem, lu, params, adj: Adjacency, x_all, mem_batch: Optional[dict],
         emb_batch: dict, noise, loss: str = "noise", flips: Optional[dict] = None) -> StepResult:
    """One training step over a mixed batch.

    The memory phase runs on ``mem_batch`` (the previous batch under the
    default lag-1 order, or the current one under lag-0), the embedding on the
    target events of ``emb_batch`` with the updated table, then the backward
    pass.  Its input dZ is the gradient of the masked loss of Eq. 13:
    ``loss="link"`` takes the link-prediction loss (``link_loss``: the decoder
    and the binary cross-entropy of each target event's true and negative
    edge, averaged over target events); ``loss="noise"`` takes a linear
    stand-in with the same masking, dZ = noise / n_tar (zero when the batch has
    no target event), which lets a test put the gradient on chosen rows.
    ``flips`` ({"m1": ..., "pos": ..., "neg": ...}, boolean arrays) inverts chosen ReLU decisions of
    the merge layer and the decoder (see ``attention_fwd``).
    """
    flips = flips or {}
    if mem_batch is None:
        mem_batch = {"src": np.zeros(0, np.int64), "dst": np.zeros(0, np.int64),
                     "t": np.zeros(0, F32), "eid": np.zeros(0, np.int64)}
    mp = memory_phase(prec, dims, mem_batch, mem, lu, x_all, params)
    q_node, q_t, n_tar = queries(emb_batch)
    nbr, nt, neid = sample_recent(adj, q_node, q_t, dims.k)
    sv = attention_fwd(prec, dims, mp.mem, x_all, params, q_node, q_t, nbr, nt, neid, flips.get("m1"))
    link = None
    if loss == "link":
        link = link_loss(params, sv.z, n_tar, flips.get("pos"), flips.get("neg"))
        dz = link.dz
    else:
        noise = np.asarray(noise, F64)[:q_node.size]
        dz = noise / n_tar if n_tar > 0 else np.zeros_like(noise)
    ag = attention_bwd(prec, dims, params, sv, dz)
    d_mem = memory_grad(mp.uniq, q_node, nbr, ag.dhq, ag.dhn)
    gg, dx = gru_bwd(d_mem, mp.msg, mp.h_old, mp.gates, prec.weight(params["W_ih"]),
                     prec.weight(params["W_hh"]))
    dtw, dtb = message_bwd(prec, dims, dx, mp.dt, params["time_w"], params["time_b"])
    grads = dict(ag.grads)
    grads.update(gg)
    grads["time_w"] = ag.d_time_w + dtw
    grads["time_b"] = ag.d_time_b + dtb
    if link is not None:
        grads.update(link.grads)
    return StepResult(mp, q_node, q_t, n_tar, nbr, nt, neid, sv, dz, ag, d_mem, grads, link)


def batch_dict(stream, lo: int, hi: int) -> dict:
    """Slice [lo, hi) of a ``synth`` stream as an oracle batch (eids = positions)."""
    d = {"src": stream.src[lo:hi], "dst": stream.dst[lo:hi], "t": stream.t[lo:hi],
         "eid": np.arange(lo, hi, dtype=np.int64), "neg": stream.neg[lo:hi]}
    if stream.flags is not None:
        d["flags"] = stream.flags[lo:hi]
    return d
