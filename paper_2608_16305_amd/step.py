"""Device-resident state and buffers for the batch step, driven through the C ABI.

A step on batch b (default lag-1 order) runs
  memory phase on batch b-1:  aggregate_last -> build_messages -> gru_update
  embedding on batch b:       build_queries  -> sample_recent  -> temporal_attn (prepare, prepared)
  loss:                       link_loss (decoder and the masked loss of Eq. 13, giving dZ)
  backward:                   temporal_attn_bwd -> gru_update_bwd -> build_messages_bwd
all enqueued on one HIP stream with no host synchronisation (the only
data-dependent sizes, updated rows and queries, stay in device memory), except
that with overlap=True (the default) several pieces run on a second stream, forked
and joined with events: the queries, their sampling and the attention's
preparation, during the memory phase; the next step's aggregation and
messages (lag-1 order: its memory batch is this step's batch, read from the
memory this step's update leaves), and the attention backward's d_mem
grouping (a key sort), during the embedding; the decoder's first-layer weight
gradient, during the backward's data gradients; the output and merge layers'
weight gradients at batches of 65,536 queries or more, beside the score
backward; and the backward's d_mem sums followed by the GRU backward, during
the attention parameter gradients.  Results are bitwise those of overlap=False.
"""

import numpy as np
import torch

from . import mtgnn as M

ATTN_W = ("W_q", "W_k", "W_v", "W_o", "W_1", "W_2")
ATTN_B = ("b_q", "b_k", "b_v", "b_o", "b_1", "b_2")
LINK = ("W_d1", "b_d1", "W_d2", "b_d2")   # the decoder: float32 in every storage mode


class TGNStep:
    def __init__(self, w, stream, params: dict, memory: np.ndarray, last_update: np.ndarray, device="cuda",
                 lag: int = 1, torch_stream=None, overlap: bool = True, batch_off=None):
        """batch_off: optional batch boundaries ([n_batches + 1] event offsets, e.g. a worker's mixed
        batches); by default the stream is cut into batches of w.batch events."""
        self.w = w
        self.batch_off = None if batch_off is None else np.asarray(batch_off, np.int64)
        self.lag = lag
        self.overlap = overlap
        self.dev = torch.device(device)
        self.ts = torch_stream
        self.dtype_code = M.BF16 if w.dtype == "bf16" else M.F32
        self.sdt = torch.bfloat16 if self.dtype_code == M.BF16 else torch.float32
        self.d = M.dims(w.n_nodes, w.d_mem, w.d_time, w.d_edge, w.d_attn, w.n_heads, w.k, self.dtype_code)
        dev = self.dev
        E = stream.n_events
        self.n_events = E
        # stream (resident in HBM)
        self.src = torch.from_numpy(stream.src).to(dev)
        self.dst = torch.from_numpy(stream.dst).to(dev)
        self.t = torch.from_numpy(stream.t).to(dev)
        self.neg = torch.from_numpy(stream.neg).to(dev)
        self.eid = torch.arange(E, dtype=torch.int32, device=dev)
        self.x = torch.from_numpy(stream.x).to(dev) if w.d_edge > 0 else None
        self.flags = torch.from_numpy(stream.flags).to(dev) if stream.flags is not None else None
        # parameters: weights in the storage dtype, biases and time encoder in float32
        self.params = {}
        for k, v in params.items():
            tv = torch.from_numpy(np.ascontiguousarray(v)).to(dev)
            self.params[k] = tv.to(self.sdt) if k.startswith("W") and k not in LINK else tv.float()
        self.memory = torch.from_numpy(np.ascontiguousarray(memory)).to(dev).to(self.sdt).contiguous()
        self.last_update = torch.from_numpy(np.ascontiguousarray(last_update, np.float32)).to(dev)
        # temporal adjacency, built once on the device
        N = w.n_nodes
        self.csr_off = torch.empty(N + 1, dtype=torch.int64, device=dev)
        self.csr_nbr = torch.empty(max(2 * E, 1), dtype=torch.int32, device=dev)
        self.csr_t = torch.empty(max(2 * E, 1), dtype=torch.float32, device=dev)
        self.csr_eid = torch.empty(max(2 * E, 1), dtype=torch.int32, device=dev)
        ws = M.alloc_bytes(M.workspace_bytes(M.OP_BUILD_CSR, self.d, E, 0), dev)
        M.mtgnn_build_temporal_csr(self.src, self.dst, self.t, N, self.csr_off, self.csr_nbr, self.csr_t,
                                   self.csr_eid, ws, stream=self.ts)
        del ws
        self._alloc(w.batch if self.batch_off is None else max(1, int(np.diff(self.batch_off).max(initial=1))))

    # ------------------------------------------------------------------ buffers
    def _alloc(self, B):
        dev, w, d = self.dev, self.w, self.d
        self.B = B
        self.max_rows = 2 * B
        self.max_q = 3 * B
        R, Q, k = self.max_rows, self.max_q, w.k
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        # two sets of the memory phase's aggregation and message buffers: with overlap, the next
        # step's set is filled on the second stream while this step's is still read by its backward
        self._sets = [dict(uniq=torch.empty(R, **i32), winner=torch.empty(R, **i32), n_uniq=torch.zeros(1, **i32),
                           msg=torch.empty(R, w.d_msg, dtype=self.sdt, device=dev), dt=torch.empty(R, **f32))
                      for _ in range(2)]
        self._bind(0)
        self._pre = None   # (lo, hi) of the batch whose aggregation and messages fill the other set
        self.gru_save = M.alloc_bytes(M.save_bytes(M.OP_GRU_UPDATE, d, R, 0), dev)
        # two sets of the query-side buffers (queries, their samples, the attention's save): with overlap,
        # a step's queries fill the set the step before last used (see step())
        self._qsets = [dict(q_node=torch.empty(Q, **i32), q_t=torch.empty(Q, **f32), n_q=torch.zeros(1, **i32),
                            nbr=torch.empty(Q, k, **i32), nt=torch.empty(Q, k, **f32), neid=torch.empty(Q, k, **i32),
                            attn_save=M.alloc_bytes(M.save_bytes(M.OP_TEMPORAL_ATTN, d, 0, Q), dev))
                       for _ in range(2)]
        self._qbind(0)
        self._q_chain = 0   # overlapped step() calls in a row (nothing else in between)
        self._in_step = False
        self.z = torch.empty(Q, w.d_attn, **f32)
        self.d_mem = torch.empty(R, w.d_mem, **f32)
        self.dmsg_time = torch.empty(R, max(w.d_time, 1), **f32)
        self.grads = {n: torch.empty(tuple(self.params[n].shape), **f32)
                      for n in list(ATTN_W) + list(ATTN_B) + ["W_ih", "W_hh", "b_ih", "b_hh", "time_w", "time_b"]
                      + [n for n in LINK if n in self.params]}
        self.has_link = all(n in self.params for n in LINK)
        if self.has_link:
            # the masked loss: its value, the edge scores and dZ; its own workspace, because the second
            # stream's d_mem grouping fills the main workspace during the embedding
            self.loss = torch.zeros(1, **f32)
            self.scores = torch.empty(2, B, **f32)
            self.dz = torch.empty(Q, w.d_attn, **f32)
            self.ws_link = M.alloc_bytes(M.workspace_bytes(M.OP_LINK_LOSS, d, 0, Q), dev)
            self.lp = M.link_params(self.params)
            self.lg = M.link_grads(self.grads)
        ops = [(M.OP_BUILD_QUERIES, B, 0), (M.OP_AGGREGATE_LAST, B, 0), (M.OP_GRU_UPDATE, R, 0),
               (M.OP_TEMPORAL_ATTN, 0, Q), (M.OP_TEMPORAL_ATTN_BWD, R, Q), (M.OP_GRU_UPDATE_BWD, R, 0),
               (M.OP_BUILD_MESSAGES_BWD, R, 0)]
        need = max(M.workspace_bytes(op, d, r, q) for op, r, q in ops)
        self.ws = M.alloc_bytes(need, dev)   # the calls of one step run in stream order and share it
        # work on the second stream (queries, sampling and the attention's preparation during the memory
        # phase, the GRU backward during the attention backward's parameter gradients) has its own workspace
        self.ws_q = M.alloc_bytes(max(M.workspace_bytes(M.OP_BUILD_QUERIES, d, B, 0),
                                      M.workspace_bytes(M.OP_AGGREGATE_LAST, d, B, 0),
                                      M.workspace_bytes(M.OP_TEMPORAL_ATTN, d, 0, Q),
                                      M.workspace_bytes(M.OP_GRU_UPDATE_BWD, d, R, 0), 256), dev)
        self.ap = M.attn_params(self.params, d)
        self.ag = M.attn_grads(self.grads)
        # second stream (default priority) and fork/join events for the work that overlaps the main stream
        # (device-scope events: no system-scope fence per record)
        self.side_stream = torch.cuda.Stream(device=dev)
        self.fork, self.join = M.DeviceEvent(), M.DeviceEvent()
        self.q_fork, self.q_join = M.DeviceEvent(), M.DeviceEvent()
        self.g_join = M.DeviceEvent()
        self.l_fork = M.DeviceEvent()   # the link loss's fork (decoder weight gradient on the second stream)
        self.m_done, self.pre_join = M.DeviceEvent(), M.DeviceEvent()
        self.group_ahead = True   # step(): the backward's d_mem grouping during the embedding (second stream)
        self._grouped = False     # ... and it has been enqueued
        self._link_ready = False  # step(): the decoder's weight copies made for its loss

    def _batch(self, lo, hi):
        if hi <= lo:
            return M.Batch(0, None, None, None, None, None)
        f = self.flags[lo:hi] if self.flags is not None else None
        return M.batch(self.src[lo:hi], self.dst[lo:hi], self.t[lo:hi], self.eid[lo:hi], f)

    def _qbind(self, i):
        """Make query set i the current one (self.q_node, q_t, n_q, nbr, nt, neid, attn_save)."""
        self._qcur = i
        for k, v in self._qsets[i].items():
            setattr(self, k, v)

    def _bind(self, i):
        """Make buffer set i the current one (self.uniq, winner, n_uniq, msg, dt)."""
        self._cur = i
        for k, v in self._sets[i].items():
            setattr(self, k, v)

    # ------------------------------------------------------------------ phases
    def _messages(self, lo, hi, bufs, ws, stream):
        """Most-recent aggregation and message construction of events lo..hi into the buffer set bufs."""
        b = self._batch(lo, hi)
        p = self.params
        M.mtgnn_aggregate_last(b, self.w.n_nodes, bufs["uniq"], bufs["winner"], bufs["n_uniq"], ws, stream=stream)
        M.mtgnn_build_messages(b, bufs["uniq"], bufs["winner"], bufs["n_uniq"], self.max_rows, self.memory,
                               self.last_update, self.x, p["time_w"], p["time_b"], self.d, bufs["msg"], bufs["dt"],
                               stream=stream)

    def _gru(self, lo, hi, save=True):
        p = self.params
        M.mtgnn_gru_update(self._batch(lo, hi), self.uniq, self.winner, self.n_uniq, self.max_rows, self.msg,
                           p["W_ih"], p["W_hh"], p["b_ih"], p["b_hh"], self.d, self.memory, self.last_update,
                           self.gru_save if save else None, self.ws, stream=self.ts)

    def memory_phase(self, lo, hi, save=True):
        self._q_chain = self._q_chain if self._in_step else 0
        self._pre = None   # the memory changes: nothing prepared from the old state stays valid
        self._messages(lo, hi, self._sets[self._cur], self.ws, self.ts)
        self._gru(lo, hi, save)

    def queries(self, lo, hi, stream):
        """Queries of the batch's target events, their most-recent-k neighbours and the attention's
        per-query valid-slot counts and offsets: no memory read."""
        self._q_chain = self._q_chain if self._in_step else 0
        b = self._batch(lo, hi)
        M.mtgnn_build_queries(b, self.neg[lo:hi], self.q_node, self.q_t, self.n_q, self.ws_q, stream=stream)
        M.mtgnn_sample_recent(self.csr_off, self.csr_nbr, self.csr_t, self.csr_eid, self.w.n_nodes, self.q_node,
                              self.q_t, self.n_q, self.max_q, self.w.k, self.nbr, self.nt, self.neid, stream=stream)
        M.mtgnn_temporal_attn_prepare_slots(self.nbr, self.n_q, self.max_q, self.d, self.attn_save, self.ws_q,
                                            stream=stream)

    def prepare_weights(self, stream, link=False):
        """The attention's weight copies (stacked K|V, padded merge layers): they read only the weights.
        link: with the decoder's (same launch), for this step's link loss."""
        self._q_chain = self._q_chain if self._in_step else 0
        p = self.params
        if link:
            M.mtgnn_temporal_attn_prepare_weights_link(self.ap, p["time_w"], p["time_b"], self.d, self.attn_save,
                                                       self.lp, self.max_q, self.ws_link, stream=stream)
            self._link_ready = True
        else:
            M.mtgnn_temporal_attn_prepare_weights(self.ap, p["time_w"], p["time_b"], self.d, self.attn_save,
                                                  stream=stream)

    def embed(self, lo, hi, queries_done=False):
        self._q_chain = self._q_chain if self._in_step else 0
        p, s = self.params, self.ts
        if not queries_done:
            self.prepare_weights(s)
            self.queries(lo, hi, s)
        M.mtgnn_temporal_attn_prepared(self.q_node, self.q_t, self.n_q, self.max_q, self.nbr, self.nt, self.neid,
                                       self.memory, self.x, p["time_w"], p["time_b"], self.ap, self.d, self.z,
                                       self.attn_save, stream=s)

    def link_loss(self):
        """The masked loss of the embedded batch (Eq. 13) and dZ, on the main stream; with overlap, the
        loss value, the second layer's gradient sums and the first layer's weight gradient run on the second
        stream (idle between the embedding and the backward's d_mem sums), ahead of the d_mem work there,
        so the backward's join covers them."""
        if self.overlap:
            # prepared: the step made the decoder's weight copies with the attention's, on this stream
            M.mtgnn_link_loss(self.z, self.n_q, self.max_q, self.lp, self.d, self.loss, self.scores, self.dz,
                              self.lg, self.ws_link, stream=self.ts, dw_stream=self.side_stream, fork=self.l_fork,
                              prepared=self._link_ready)
            self._link_ready = False
        else:
            M.mtgnn_link_loss(self.z, self.n_q, self.max_q, self.lp, self.d, self.loss, self.scores, self.dz,
                              self.lg, self.ws_link, stream=self.ts)
        return self.dz

    def backward(self, dz):
        self._q_chain = self._q_chain if self._in_step else 0
        p, g, s = self.params, self.grads, self.ts
        if self.overlap:
            # d_mem, then the GRU backward, on the second stream while the attention parameter gradients
            # run here; the time-encoder gradient of the messages accumulates here after the join, in the
            # same order as without overlap
            M.mtgnn_temporal_attn_bwd_overlap(self.q_node, self.q_t, self.n_q, self.max_q, self.nbr, self.nt, dz,
                                              self.attn_save, self.uniq, self.n_uniq, self.max_rows, p["time_w"],
                                              p["time_b"], self.ap, self.d, self.ag, self.d_mem, g["time_w"],
                                              g["time_b"], self.ws, self.side_stream, self.fork,
                                              None if self._grouped else self.join, stream=s,
                                              grouped=self._grouped)
            self._grouped = False
            M.mtgnn_gru_update_bwd(self.d_mem, self.gru_save, self.msg, self.n_uniq, self.max_rows, p["W_ih"],
                                   p["W_hh"], self.d, g["W_ih"], g["W_hh"], g["b_ih"], g["b_hh"], self.dmsg_time,
                                   self.ws_q, stream=self.side_stream)
            self.g_join.record(self.side_stream)
            main = s if s is not None else torch.cuda.current_stream(self.dev)
            self.g_join.wait(main)
        else:
            M.mtgnn_temporal_attn_bwd(self.q_node, self.q_t, self.n_q, self.max_q, self.nbr, self.nt, dz,
                                      self.attn_save, self.uniq, self.n_uniq, self.max_rows, p["time_w"], p["time_b"],
                                      self.ap, self.d, self.ag, self.d_mem, g["time_w"], g["time_b"], self.ws,
                                      stream=s)
            M.mtgnn_gru_update_bwd(self.d_mem, self.gru_save, self.msg, self.n_uniq, self.max_rows, p["W_ih"],
                                   p["W_hh"], self.d, g["W_ih"], g["W_hh"], g["b_ih"], g["b_hh"], self.dmsg_time,
                                   self.ws, stream=s)
        M.mtgnn_build_messages_bwd(self.dmsg_time, self.dt, self.n_uniq, self.max_rows, p["time_w"], p["time_b"],
                                   self.d, g["time_w"], g["time_b"], self.ws, stream=s)

    def params_changed(self):
        """The caller updated the parameters in place: messages built ahead from the old time encoder
        (during the previous step's embedding) are discarded, and the next step builds its own."""
        self._pre = None

    def batch_range(self, b):
        if self.batch_off is not None:
            return int(self.batch_off[b]), int(self.batch_off[b + 1])
        lo = b * self.B
        return lo, min(self.n_events, lo + self.B)

    def step(self, b, dz=None):
        """One training step on batch b: memory phase (lag order), embedding, the masked link-prediction
        loss, backward.  A given dz [max_q, d_attn] replaces the loss's gradient (the loss is not run)."""
        elo, ehi = self.batch_range(b)
        self._in_step = True
        if self.lag == 1:
            mlo, mhi = self.batch_range(b - 1) if b > 0 else (0, 0)
        else:
            mlo, mhi = elo, ehi
        if self.overlap:
            # queries, sampling and preparation on the second stream while the memory phase runs here (they
            # read only the batch, the adjacency and the weights); joined before the attention reads memory
            main = self.ts if self.ts is not None else torch.cuda.current_stream(self.dev)
            side = self.side_stream
            # the queries fill the other query set, last used by the step before the previous one: after
            # an overlapped step, all its uses here precede that step's m_done, which the second stream
            # waited for, so no fork is needed (the first step, or after other calls, forks)
            self._qbind(1 - self._qcur)
            if self._q_chain == 0:
                self.q_fork.record(main)
                self.q_fork.wait(side)
            self.queries(elo, ehi, side)
            self.q_join.record(side)
            # one launch here, so the second stream's chain is shorter; after any parameter update the
            # caller made on this stream, and with the decoder's weight copies when the loss runs
            self.prepare_weights(main, link=dz is None and self.has_link)
            if self.lag == 1 and self._pre == (mlo, mhi):
                # this memory batch's aggregation and messages were built during the previous step's
                # embedding, from the memory as it is now: only the GRU update is left
                self._bind(1 - self._cur)
                if self._q_chain == 0:   # else implied: the previous step's backward waited for g_join,
                    self.pre_join.wait(main)   # recorded on the second stream after these messages
                self._pre = None
                self._gru(mlo, mhi)
            else:
                self.memory_phase(mlo, mhi)
            self.m_done.record(main)
            self.m_done.wait(side)
            if self.lag == 1:
                # the next step's memory batch is this step's batch: its aggregation and messages read the
                # memory as this update leaves it, which nothing changes before the next step's GRU update;
                # built on the second stream into the other buffer set while the embedding runs here
                self._messages(elo, ehi, self._sets[1 - self._cur], self.ws_q, side)
                self.pre_join.record(side)
                self._pre = (elo, ehi)
            # the backward's d_mem grouping (a key sort) needs only this step's updated rows and sampled
            # slots: on the second stream during the embedding, into the backward's workspace, which
            # nothing here touches until the backward
            if self.group_ahead:
                M.mtgnn_temporal_attn_bwd_group(self.q_node, self.n_q, self.max_q, self.nbr, self.attn_save,
                                                self.uniq, self.n_uniq, self.max_rows, self.d, self.ws, stream=side)
                self._grouped = True
            self.q_join.wait(main)
            self.embed(elo, ehi, queries_done=True)
        else:
            self.memory_phase(mlo, mhi)
            self.embed(elo, ehi)
        if dz is None:
            dz = self.link_loss()
        self.backward(dz)
        self._in_step = False
        self._q_chain = self._q_chain + 1 if self.overlap else 0
