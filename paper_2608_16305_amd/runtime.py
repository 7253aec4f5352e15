"""One worker's adaptive training loop on one GPU (Algorithm 2), driven through the C ABI.

The worker p owns the nodes the ownership map assigns it.  Offline, the
dependency scan (Algorithm 1) marks every event of the stream as a target of
p (its source is owned by p), an auxiliary replay event of p, or absent, per
synchronization window of `window` batches, and leaves each window's
candidate refresh set; the worker's local stream is its mixed batches (Eq. 5)
in stream order, replay events flagged.  Then, per batch r:

1. at a candidate boundary (r % window == 0) the controller decides S_r
   (Eq. 7); with S_r = 1 the cached states of the window's refresh set take
   the authoritative states (Eq. 25);
2. the controller decides the heavy-load mode H_r (Eq. 9) and PruneAux marks
   the batch's replay events pruned under it (Eq. 10-11);
3. the batch step runs (memory phase, embedding, masked link-prediction loss
   of Eq. 12-13, backward);
4. the gradient norm g_r, the Adam update, and the batch time c_r (HIP events
   around the step on the main stream, or a caller's clock) feed the
   controller's averages (Eq. 6, 8).

Every computation runs in the library's kernels; this module allocates buffers,
orders the calls and moves the two scalars the controller needs to the host.
"""

from dataclasses import dataclass

import numpy as np
import torch

from . import mtgnn as M
from .step import LINK, TGNStep


@dataclass
class BatchRecord:
    r: int
    boundary: int
    sync: int
    heavy: int
    grad_norm: float
    batch_ms: float
    loss: float
    n_events: int


class WorkerStreamData:
    """A stream in host memory (the fields the step reads): the worker's local copy."""

    def __init__(self, w, src, dst, t, x, neg, flags):
        self.w, self.src, self.dst, self.t, self.x, self.neg, self.flags = w, src, dst, t, x, neg, flags

    @property
    def n_events(self):
        return int(self.src.shape[0])


def worker_stream(stream, owner, p, n_workers, batch, window, device="cuda"):
    """Algorithm 1 on the device for every worker and window, then worker p's mixed batches.

    Returns (local stream, batch offsets [n_batches + 1] (host), refresh-set bitmaps
    [n_windows, ceil(n_nodes / 32)] (device), roles [P, E] (device))."""
    dev = torch.device(device)
    E, N = stream.n_events, int(owner.shape[0])
    src = torch.from_numpy(np.ascontiguousarray(stream.src, np.int32)).to(dev)
    dst = torch.from_numpy(np.ascontiguousarray(stream.dst, np.int32)).to(dev)
    own = torch.from_numpy(np.ascontiguousarray(owner, np.int32)).to(dev)
    n_batches = -(-E // batch)
    n_windows = -(-n_batches // window)
    role = torch.empty(n_workers, E, dtype=torch.uint8, device=dev)
    sync = torch.empty(n_workers, n_windows, -(-N // 32), dtype=torch.int32, device=dev)
    M.mtgnn_dependency_scan(src, dst, own, n_workers, batch, window, role, sync)
    eid = torch.empty(E, dtype=torch.int32, device=dev)
    flags = torch.empty(E, dtype=torch.uint8, device=dev)
    off = torch.empty(n_batches + 1, dtype=torch.int32, device=dev)
    ws = M.alloc_bytes(M.workspace_bytes(M.OP_MIXED_BATCHES, None, E, 0), dev)
    M.mtgnn_mixed_batches(role[p].contiguous(), batch, eid, flags, off, ws)
    off_h = off.cpu().numpy().astype(np.int64)
    n = int(off_h[-1])
    ids = eid[:n].cpu().numpy().astype(np.int64)
    fl = flags[:n].cpu().numpy()
    local = WorkerStreamData(stream.w, stream.src[ids], stream.dst[ids], stream.t[ids],
                             stream.x[ids] if stream.x is not None else None, stream.neg[ids], fl)
    return local, off_h, sync[p], role


class AdaptiveTrainer:
    def __init__(self, w, stream, params, memory, last_update, owner, p, n_workers, window, device="cuda",
                 alpha=0.1, beta=0.1, tau_g=0.9, tau_c=1.5, lr=1e-4, betas=(0.9, 0.999), eps=1e-8):
        self.w, self.p, self.window = w, p, window
        self.local, self.batch_off, self.sync_bits, self.role = worker_stream(stream, owner, p, n_workers, w.batch,
                                                                              window, device)
        self.n_batches = self.batch_off.size - 1
        self.step = TGNStep(w, self.local, params, memory, last_update, device=device, batch_off=self.batch_off)
        self.ctrl = M.Controller(alpha, beta, tau_g, tau_c, window)
        self.lr, self.betas, self.eps = lr, betas, eps
        st = self.step
        names = list(st.grads.keys())
        self.names = names
        # float32 master parameters (the step's own tensors where they are float32), Adam moments
        self.master = {k: st.params[k] if st.params[k].dtype == torch.float32 else st.params[k].float().clone()
                       for k in names}
        self.shadow = {k: (st.params[k] if st.params[k].dtype == torch.bfloat16 else None) for k in names}
        self.m = {k: torch.zeros_like(self.master[k]) for k in names}
        self.v = {k: torch.zeros_like(self.master[k]) for k in names}
        self.t = 0
        self.norm = torch.zeros(1, dtype=torch.float64, device=st.dev)
        self.norm_ws = M.alloc_bytes(M.grad_norm_ws_bytes([st.grads[k] for k in names]), st.dev)
        self.ev0 = torch.cuda.Event(enable_timing=True)
        self.ev1 = torch.cuda.Event(enable_timing=True)
        self.records = []

    def refresh(self, r, authority):
        """Eq. 25 for window r // window's refresh set from authority = (memory, last_update) tables."""
        st = self.step
        M.mtgnn_cache_refresh(self.sync_bits[r // self.window], self.w.n_nodes, authority[0], authority[1], st.d,
                              st.memory, st.last_update, stream=st.ts)
        st._pre = None   # the memory changed: messages built ahead from the old state are stale

    def batch(self, r, authority=None, clock=None):
        """Algorithm 2's body for batch r; returns its record."""
        st = self.step
        boundary, sync, heavy = self.ctrl.decide(r)
        if boundary and sync and authority is not None:
            self.refresh(r, authority)
        lo, hi = st.batch_range(r)
        if hi > lo:
            M.mtgnn_prune_aux(st.flags[lo:hi], heavy, stream=st.ts)
        main = st.ts if st.ts is not None else torch.cuda.current_stream(st.dev)
        self.ev0.record(main)
        st.step(r)
        self.ev1.record(main)
        grads = [st.grads[k] for k in self.names]
        M.mtgnn_grad_norm(grads, self.norm, self.norm_ws, stream=st.ts)
        self.t += 1
        M.mtgnn_adam_step([self.master[k] for k in self.names], grads, [self.m[k] for k in self.names],
                          [self.v[k] for k in self.names], [self.shadow[k] for k in self.names], self.lr,
                          self.betas[0], self.betas[1], self.eps, self.t, stream=st.ts)
        st.params_changed()
        torch.cuda.synchronize(st.dev)
        c_r = float(clock(r)) if clock is not None else float(self.ev0.elapsed_time(self.ev1))
        g_r = float(self.norm.item())
        self.ctrl.observe(g_r, c_r)
        rec = BatchRecord(r, boundary, sync, heavy, g_r, c_r, float(st.loss.item()), hi - lo)
        self.records.append(rec)
        return rec

    def run(self, n_batches=None, authority=None, clock=None):
        for r in range(self.n_batches if n_batches is None else n_batches):
            self.batch(r, authority, clock)
        return self.records


__all__ = ["AdaptiveTrainer", "BatchRecord", "worker_stream", "LINK"]
