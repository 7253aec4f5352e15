"""The JODIE batch step on one GPU, driven through the C ABI (Section VII-A's second model).

A step on batch b (lag-1 order, as TGNStep):
  memory phase on batch b-1:  aggregate_last -> build_messages -> rnn_update
  embedding of batch b:       build_queries -> time_projection
  loss:                       link_loss (the masked loss of Eq. 13, giving dZ)
  backward:                   time_projection_bwd -> rnn_update_bwd -> build_messages_bwd
all on one stream, with no host synchronisation.  Every computation runs in the library's kernels.
"""

import numpy as np
import torch

from . import mtgnn as M

LINK = ("W_d1", "b_d1", "W_d2", "b_d2")
FLOAT_PARAMS = LINK + ("b_ih", "b_hh", "W_p", "b_p", "time_w", "time_b")


class JodieStep:
    def __init__(self, w, stream, params: dict, memory, last_update, time_scale=None, device="cuda", lag=1):
        if w.d_attn != w.d_mem:
            raise ValueError("the JODIE embedding is d_mem wide: the decoder needs d_attn == d_mem")
        self.w, self.lag, self.dev = w, lag, torch.device(device)
        self.dtype_code = M.BF16 if w.dtype == "bf16" else M.F32
        self.sdt = torch.bfloat16 if self.dtype_code == M.BF16 else torch.float32
        self.d = M.dims(w.n_nodes, w.d_mem, w.d_time, w.d_edge, w.d_mem, 1, 1, self.dtype_code)
        dev = self.dev
        E = stream.n_events
        self.n_events = E
        self.src = torch.from_numpy(stream.src).to(dev)
        self.dst = torch.from_numpy(stream.dst).to(dev)
        self.t = torch.from_numpy(stream.t).to(dev)
        self.neg = torch.from_numpy(stream.neg).to(dev)
        self.eid = torch.arange(E, dtype=torch.int32, device=dev)
        self.x = torch.from_numpy(stream.x).to(dev) if w.d_edge > 0 else None
        self.flags = torch.from_numpy(stream.flags).to(dev) if stream.flags is not None else None
        # Delta = (tau - last_update) s: by default s maps the stream's time span to 10
        span = float(stream.t[-1] - stream.t[0]) if E > 1 else 1.0
        self.time_scale = float(time_scale) if time_scale is not None else 10.0 / max(span, 1e-30)
        self.params = {}
        for k, v in params.items():
            tv = torch.from_numpy(np.ascontiguousarray(v)).to(dev)
            self.params[k] = tv.float() if k in FLOAT_PARAMS else tv.to(self.sdt)
        self.memory = torch.from_numpy(np.ascontiguousarray(memory)).to(dev).to(self.sdt).contiguous()
        self.last_update = torch.from_numpy(np.ascontiguousarray(last_update, np.float32)).to(dev)
        B = w.batch
        self.B, self.max_rows, self.max_q = B, 2 * B, 3 * B
        R, Q, d = self.max_rows, self.max_q, self.d
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.uniq, self.winner, self.n_uniq = torch.empty(R, **i32), torch.empty(R, **i32), torch.zeros(1, **i32)
        self.msg = torch.empty(R, w.d_msg, dtype=self.sdt, device=dev)
        self.dt = torch.empty(R, **f32)
        self.save = M.alloc_bytes(M.save_bytes(M.OP_RNN_UPDATE, d, R, 0), dev)
        self.q_node, self.q_t, self.n_q = torch.empty(Q, **i32), torch.empty(Q, **f32), torch.zeros(1, **i32)
        self.z = torch.empty(Q, w.d_mem, **f32)
        self.dz = torch.empty(Q, w.d_mem, **f32)
        self.loss = torch.zeros(1, **f32)
        self.scores = torch.empty(2, B, **f32)
        self.d_mem = torch.empty(R, w.d_mem, **f32)
        self.dmsg_time = torch.empty(R, max(w.d_time, 1), **f32)
        self.grads = {k: torch.empty(tuple(v.shape), **f32) for k, v in self.params.items()}
        ops = [(M.OP_BUILD_QUERIES, B, 0), (M.OP_AGGREGATE_LAST, B, 0), (M.OP_RNN_UPDATE, R, 0),
               (M.OP_RNN_UPDATE_BWD, R, 0), (M.OP_TIME_PROJECTION_BWD, 0, Q), (M.OP_BUILD_MESSAGES_BWD, R, 0),
               (M.OP_LINK_LOSS, 0, Q)]
        self.ws = M.alloc_bytes(max(M.workspace_bytes(op, d, r, q) for op, r, q in ops), dev)
        self.lp = M.link_params(self.params)
        self.lg = M.link_grads(self.grads)

    def batch_range(self, b):
        lo = b * self.B
        return lo, min(self.n_events, lo + self.B)

    def _batch(self, lo, hi):
        if hi <= lo:
            return M.Batch(0, None, None, None, None, None)
        f = self.flags[lo:hi] if self.flags is not None else None
        return M.batch(self.src[lo:hi], self.dst[lo:hi], self.t[lo:hi], self.eid[lo:hi], f)

    def step(self, b):
        p, d, g, R, Q = self.params, self.d, self.grads, self.max_rows, self.max_q
        elo, ehi = self.batch_range(b)
        mlo, mhi = (self.batch_range(b - 1) if b > 0 else (0, 0)) if self.lag == 1 else (elo, ehi)
        mb = self._batch(mlo, mhi)
        M.mtgnn_aggregate_last(mb, self.w.n_nodes, self.uniq, self.winner, self.n_uniq, self.ws)
        M.mtgnn_build_messages(mb, self.uniq, self.winner, self.n_uniq, R, self.memory, self.last_update, self.x,
                               p["time_w"], p["time_b"], d, self.msg, self.dt)
        M.mtgnn_rnn_update(mb, self.uniq, self.winner, self.n_uniq, R, self.msg, p["W_ih"], p["W_hh"], p["b_ih"],
                           p["b_hh"], d, self.memory, self.last_update, self.save, self.ws)
        M.mtgnn_build_queries(self._batch(elo, ehi), self.neg[elo:ehi], self.q_node, self.q_t, self.n_q, self.ws)
        M.mtgnn_time_projection(self.q_node, self.q_t, self.n_q, Q, self.memory, self.last_update, p["W_p"], p["b_p"],
                                self.time_scale, d, self.z)
        M.mtgnn_link_loss(self.z, self.n_q, Q, self.lp, d, self.loss, self.scores, self.dz, self.lg, self.ws)
        M.mtgnn_time_projection_bwd(self.q_node, self.q_t, self.n_q, Q, self.memory, self.last_update, p["W_p"],
                                    p["b_p"], self.time_scale, self.dz, self.uniq, self.n_uniq, R, d, g["W_p"],
                                    g["b_p"], self.d_mem, self.ws)
        M.mtgnn_rnn_update_bwd(self.d_mem, self.save, self.msg, self.n_uniq, R, p["W_ih"], p["W_hh"], d, g["W_ih"],
                               g["W_hh"], g["b_ih"], g["b_hh"], self.dmsg_time, self.ws)
        g["time_w"].zero_()   # the messages are the time encoder's only consumer here: their share accumulates
        g["time_b"].zero_()
        M.mtgnn_build_messages_bwd(self.dmsg_time, self.dt, self.n_uniq, R, p["time_w"], p["time_b"], d, g["time_w"],
                                   g["time_b"], self.ws)
