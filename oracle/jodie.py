"""The JODIE variant of the batch step -- TEST INFRASTRUCTURE ONLY.

Section VII-A evaluates a second memory-based model, JODIE, whose node
states evolve through recurrent updates and whose embeddings project a
state forward in time.  In the paper's abstract form (Eq. 1-2) it differs
from TGN only in Update and in the embedding:

* messages, most-recent aggregation and the write-back of last_update are
  those of ``tgn`` (Eq. 1-2 read the same way);
* Update is a recurrent cell: h' = tanh(W_ih x + b_ih + W_hh h + b_hh);
* the embedding of node n at time tau is the time projection
      z = M[n] * (1 + W_p Delta + b_p),   Delta = (tau - last_update[n]) * s,
  with W_p [d_m, 1], b_p [d_m] and a fixed time scale s (an input), so no
  neighbour sampling is involved;
* the masked link-prediction loss of ``tgn.link_loss`` on z.

Float64 arithmetic on the storage dtype's values (float32 here), as ``tgn``.
"""

from dataclasses import dataclass

import numpy as np

from . import tgn

F32, F64 = np.float32, np.float64


def rnn_cell(x, h, W_ih, W_hh, b_ih, b_hh):
    return np.tanh(x @ W_ih.T + b_ih + h @ W_hh.T + b_hh)


def projection_delta(prec, q_t, lu_q, scale):
    """Delta = (tau - last_update) * s: float32 operations (the subtraction, then the product) outside
    the float64 mode."""
    if prec.mode == "f64":
        return (np.asarray(q_t, F64) - np.asarray(lu_q, F64)) * float(scale)
    d = (np.asarray(q_t, F32) - np.asarray(lu_q, F32)).astype(F32)
    return (d * F32(scale)).astype(F32)


def project(mem_q, delta, W_p, b_p):
    return np.asarray(mem_q, F64) * (1.0 + np.asarray(delta, F64)[:, None] * np.asarray(W_p, F64)[:, 0]
                                     + np.asarray(b_p, F64))


@dataclass
class JodieStep:
    mp: tgn.MemoryPhase
    q_node: np.ndarray
    q_t: np.ndarray
    n_tar: int
    delta: np.ndarray
    z: np.ndarray
    link: tgn.LinkLoss
    d_mem: np.ndarray
    grads: dict


def memory_phase(prec, dims, batch, mem, lu, x_all, params):
    """Eq. 1-2 with the recurrent update: select, build messages (as ``tgn``), RNN, write back."""
    uniq, winner = tgn.select_last(batch["src"], batch["dst"], batch["t"], batch["eid"], batch.get("flags"))
    msg, dt = tgn.build_messages(prec, dims, batch["src"], batch["dst"], batch["t"], batch["eid"], uniq, winner,
                                 mem, lu, x_all, params["time_w"], params["time_b"])
    h_old = np.asarray(mem[uniq], F64)
    h_new = rnn_cell(msg, h_old, prec.weight(params["W_ih"]), prec.weight(params["W_hh"]),
                     np.asarray(params["b_ih"], F64), np.asarray(params["b_hh"], F64))
    mem2 = np.array(mem, copy=True)
    lu2 = np.array(lu, copy=True)
    if len(uniq):
        mem2[uniq] = prec.store(h_new)
        lu2[uniq] = np.asarray(batch["t"], F32)[winner // 2]
    return tgn.MemoryPhase(uniq, winner, msg, dt, h_old, (), h_new, mem2, lu2)


def step(prec, dims, mem, lu, params, x_all, mem_batch, emb_batch, scale, flips=None) -> JodieStep:
    """One JODIE training step: memory phase on mem_batch, projection of emb_batch's queries with the
    updated table, the masked link loss, and the backward pass (memory is detached across steps).
    ``flips`` inverts chosen decoder ReLU decisions, as ``tgn.step``'s."""
    flips = flips or {}
    if mem_batch is None:
        mem_batch = {"src": np.zeros(0, np.int64), "dst": np.zeros(0, np.int64), "t": np.zeros(0, F32),
                     "eid": np.zeros(0, np.int64)}
    mp = memory_phase(prec, dims, mem_batch, mem, lu, x_all, params)
    q_node, q_t, n_tar = tgn.queries(emb_batch)
    delta = projection_delta(prec, q_t, mp.lu[q_node], scale)
    Mq = np.asarray(mp.mem[q_node], F64)
    z = project(Mq, delta, params["W_p"], params["b_p"])
    link = tgn.link_loss(params, z, n_tar, flips.get("pos"), flips.get("neg"))
    dz = link.dz
    g = dict(link.grads)
    # z = M (1 + W_p Delta + b_p)
    dl = np.asarray(delta, F64)[:, None]
    g["W_p"] = (dz * Mq * dl).sum(0)[:, None]
    g["b_p"] = (dz * Mq).sum(0)
    dMq = dz * (1.0 + dl * np.asarray(params["W_p"], F64)[:, 0] + np.asarray(params["b_p"], F64))
    # d M' for the rows updated in this step's memory phase (query occurrences only)
    d_mem = np.zeros((len(mp.uniq), dims.d_mem))
    pos = {int(n): i for i, n in enumerate(mp.uniq)}
    for qi, n in enumerate(q_node):
        i = pos.get(int(n))
        if i is not None:
            d_mem[i] += dMq[qi]
    # h' = tanh(pre): dpre = d_mem (1 - h'^2)
    dpre = d_mem * (1.0 - mp.h_new ** 2)
    g["W_ih"] = dpre.T @ mp.msg
    g["W_hh"] = dpre.T @ mp.h_old
    g["b_ih"] = dpre.sum(0)
    g["b_hh"] = dpre.sum(0)
    dx = dpre @ prec.weight(params["W_ih"])
    dtw, dtb = tgn.message_bwd(prec, dims, dx, mp.dt, params["time_w"], params["time_b"])
    g["time_w"], g["time_b"] = dtw, dtb
    return JodieStep(mp, q_node, q_t, n_tar, delta, z, link, d_mem, g)
