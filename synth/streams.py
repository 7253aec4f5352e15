"""Seeded event streams, masks, negatives, parameters and start states.

Every draw comes from ``np.random.default_rng(SeedSequence([base, stream_cid,
part, chunk]))`` so that any piece can be regenerated on its own and large
streams can be drawn chunk by chunk.  Event ids are stream positions: the
stream is sorted by (t, eid), which is the chronological order of the paper's
event tuples (Section III-A).
"""

from dataclasses import dataclass
from typing import Optional

import numpy as np

from .configs import Workload

CHUNK = 10_000_000  # events per generation chunk

# seed "parts"
_SRC, _DST, _T, _X, _NEG, _FLAGS, _PERM, _PARAMS, _M0, _G, _BIAS, _OWNER = range(12)

FLAG_REPLAY = 1   # bit 0: event replayed from the temporal-event cache (auxiliary)
FLAG_PRUNED = 2   # bit 1: replay event removed by load-aware pruning


def _rng(base: int, cid: int, part: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([base, cid, part, chunk]))


@dataclass
class Stream:
    """A chronologically sorted event stream (structure of arrays)."""
    w: Workload
    src: np.ndarray              # int32 [E]
    dst: np.ndarray              # int32 [E]
    t: np.ndarray                # float32 [E], non-decreasing
    x: Optional[np.ndarray]      # float32 [E, d_edge] or None when d_edge == 0
    neg: np.ndarray              # int32 [E], one negative destination per event
    flags: Optional[np.ndarray]  # uint8 [E] (bit0 replay, bit1 pruned) or None

    @property
    def n_events(self) -> int:
        return int(self.src.shape[0])


def _zipf_cdf(n_ranks: int, s: float) -> np.ndarray:
    w = np.arange(1, n_ranks + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    return cdf


def _zipf_guide(cdf: np.ndarray) -> np.ndarray:
    """Guide table of the inverse-CDF search: g[j] = first rank whose CDF exceeds j / M."""
    M = cdf.shape[0]
    return np.searchsorted(cdf, np.arange(M, dtype=np.float64) / M, side="right")


def _zipf_draw(rng: np.random.Generator, cdf: np.ndarray, n: int, guide=None) -> np.ndarray:
    """Ranks r = first index with cdf[r] > u for u ~ U[0, 1): the inverse CDF.

    The guide table gives, for u in [j/M, (j+1)/M), a start that is never past
    the answer; a short forward scan finishes it, so the result equals a
    binary search (``searchsorted(cdf, u, side="right")``) exactly.
    """
    u = rng.random(n)
    if guide is None:
        r = np.searchsorted(cdf, u, side="right")
    else:
        M = cdf.shape[0]
        r = guide[np.minimum((u * M).astype(np.int64), M - 1)]
        np.minimum(r, M - 1, out=r)
        act = np.nonzero(cdf[r] <= u)[0]
        while act.size:
            r[act] += 1
            np.minimum(r, M - 1, out=r)
            act = act[(cdf[r[act]] <= u[act]) & (r[act] < M - 1)]
    np.minimum(r, cdf.shape[0] - 1, out=r)
    return r


def _chunks(n: int):
    for c, lo in enumerate(range(0, n, CHUNK)):
        yield c, lo, min(n, lo + CHUNK)


def _each_chunk(n: int, fn) -> None:
    """fn(c, lo, hi) for every chunk; chunks have their own generators, so they run on threads."""
    chunks = list(_chunks(n))
    if len(chunks) == 1:
        fn(*chunks[0])
        return
    import os
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=min(len(chunks), os.cpu_count() or 1, 16)) as ex:
        for f in [ex.submit(fn, *c) for c in chunks]:
            f.result()


def make_stream(w: Workload, base_seed: int = 0) -> Stream:
    """Draw the event stream of workload ``w`` (deterministic per seed)."""
    E, N = w.n_events, w.n_nodes
    cid = w.stream_cid
    src = np.empty(E, np.int32)
    dst = np.empty(E, np.int32)
    neg = np.empty(E, np.int32)
    perm = None
    if w.src_rule.startswith("zipf") or w.dst_rule.startswith("zipf"):
        n_ranks = (N - w.n_src) if w.dst_rule == "zipf_dst" else N
        cdf = _zipf_cdf(n_ranks, w.zipf_s)
        guide = _zipf_guide(cdf) if n_ranks > 2_000_000 else None   # same draws; faster for large rank counts
        perm = _rng(base_seed, cid, _PERM).permutation(n_ranks).astype(np.int64)
    def endpoints(c, lo, hi):
        n = hi - lo
        rs = _rng(base_seed, cid, _SRC, c)
        rd = _rng(base_seed, cid, _DST, c)
        if w.src_rule == "uniform":
            src[lo:hi] = rs.integers(0, N, n)
        elif w.src_rule == "uniform_src":
            src[lo:hi] = rs.integers(0, w.n_src, n)
        else:  # zipf over all nodes through a seeded permutation
            src[lo:hi] = perm[_zipf_draw(rs, cdf, n, guide)]
        if w.dst_rule == "uniform":
            dst[lo:hi] = rd.integers(0, N, n)
        elif w.dst_rule == "zipf_dst":
            dst[lo:hi] = w.n_src + perm[_zipf_draw(rd, cdf, n, guide)]
        else:
            dst[lo:hi] = perm[_zipf_draw(rd, cdf, n, guide)]
        rn = _rng(base_seed, cid, _NEG, c)
        if w.neg_rule == "dst":
            neg[lo:hi] = rn.integers(w.n_src, N, n)
        else:
            neg[lo:hi] = rn.integers(0, N, n)

    _each_chunk(E, endpoints)

    if w.t_rule == "uniform_sorted":
        t64 = np.empty(E, np.float64)

        def times(c, lo, hi):
            t64[lo:hi] = _rng(base_seed, cid, _T, c).random(hi - lo) * 1e5
        _each_chunk(E, times)
        t64.sort()
    elif w.t_rule == "exp_gaps":
        gaps = np.empty(E, np.float64)
        for c, lo, hi in _chunks(E):
            gaps[lo:hi] = _rng(base_seed, cid, _T, c).exponential(15.0, hi - lo)
        t64 = np.cumsum(gaps)
    else:
        raise ValueError(w.t_rule)
    t = t64.astype(np.float32)  # monotone rounding keeps the order
    del t64

    x = None
    if w.d_edge > 0:
        x = np.empty((E, w.d_edge), np.float32)

        def feats(c, lo, hi):
            _rng(base_seed, cid, _X, c).standard_normal((hi - lo, w.d_edge), dtype=np.float32, out=x[lo:hi])
        _each_chunk(E, feats)

    flags = None
    if w.replay_p > 0:
        flags = np.empty(E, np.uint8)
        for c, lo, hi in _chunks(E):
            r = _rng(base_seed, w.cid, _FLAGS, c)
            replay = r.random(hi - lo) < w.replay_p
            pruned = replay & (r.random(hi - lo) < w.prune_p)
            flags[lo:hi] = replay.astype(np.uint8) * FLAG_REPLAY + pruned.astype(np.uint8) * FLAG_PRUNED
    return Stream(w, src, dst, t, x, neg, flags)


def batch_slice(w: Workload, b: int):
    """Event index range [lo, hi) of batch ``b``."""
    lo = b * w.batch
    return lo, min(w.n_events, lo + w.batch)


def init_params(w: Workload, base_seed: int = 0, random_bias: bool = False,
                bias_scale: float = 0.1) -> dict:
    """Xavier-uniform weights drawn in a fixed order from one generator.

    Weights use the nn.Linear [out, in] layout.  Biases are zero unless
    ``random_bias`` (tests use it so that every bias term is exercised).
    The time encoder starts from w_j = 10^(-9 j/(d_t-1)), b = 0.
    All arrays are float32.
    """
    dm, dt, de, da = w.d_mem, w.d_time, w.d_edge, w.d_attn
    shapes = [
        ("W_ih", (3 * dm, w.d_msg)), ("W_hh", (3 * dm, dm)),
        ("W_q", (da, w.d_q)), ("W_k", (da, w.d_kv)), ("W_v", (da, w.d_kv)),
        ("W_o", (da, da)), ("W_1", (da, da + dm)), ("W_2", (da, da)),
    ]
    rng = np.random.default_rng(base_seed)
    p = {}
    for name, (fo, fi) in shapes:
        a = np.sqrt(6.0 / (fi + fo))
        p[name] = rng.uniform(-a, a, size=(fo, fi)).astype(np.float32)
    bias_shapes = [("b_ih", 3 * dm), ("b_hh", 3 * dm), ("b_q", da), ("b_k", da), ("b_v", da),
                   ("b_o", da), ("b_1", da), ("b_2", da)]
    rb = _rng(base_seed, w.cid, _BIAS)
    for name, n in bias_shapes:
        if random_bias:
            p[name] = rb.uniform(-bias_scale, bias_scale, n).astype(np.float32)
        else:
            p[name] = np.zeros(n, np.float32)
    j = np.arange(dt, dtype=np.float64)
    p["time_w"] = (10.0 ** (-9.0 * j / max(dt - 1, 1))).astype(np.float32)
    p["time_b"] = (rb.uniform(-1.0, 1.0, dt).astype(np.float32) if random_bias
                   else np.zeros(dt, np.float32))
    # link-prediction decoder [z_src || z_other] -> d_attn -> 1, drawn after everything above
    for name, (fo, fi) in (("W_d1", (da, 2 * da)), ("W_d2", (1, da))):
        a = np.sqrt(6.0 / (fi + fo))
        p[name] = rng.uniform(-a, a, size=(fo, fi)).astype(np.float32)
    for name, n in (("b_d1", da), ("b_d2", 1)):
        p[name] = (rb.uniform(-bias_scale, bias_scale, n).astype(np.float32) if random_bias
                   else np.zeros(n, np.float32))
    return p


def window_state(w: Workload, s: Stream, b0: int, base_seed: int = 0):
    """Shared start state for a mid-stream window beginning at batch ``b0``.

    memory ~ U(-1, 1) (float32), and last_update[n] = the time of n's last
    event strictly before batch ``b0`` (0 for nodes without one).
    """
    N, dm = w.n_nodes, w.d_mem
    mem = np.empty((N, dm), np.float32)
    step = max(1, CHUNK // max(dm, 1))
    for c, lo in enumerate(range(0, N, step)):
        hi = min(N, lo + step)
        mem[lo:hi] = _rng(base_seed, w.cid, _M0, c).uniform(-1.0, 1.0, (hi - lo, dm)).astype(np.float32)
    e0 = min(s.n_events, b0 * w.batch)
    lu = np.zeros(N, np.float32)
    if e0 > 0:
        lu[:] = last_event_time(s.src[:e0], s.dst[:e0], s.t[:e0], N)
    return mem, lu


def last_event_time(src, dst, t, n_nodes: int) -> np.ndarray:
    """t of each node's last event (as either endpoint) in a time-sorted stream, else 0 (times are >= 0)."""
    lu = np.zeros(n_nodes, np.float32)
    tt = np.asarray(t, np.float32)
    np.maximum.at(lu, np.asarray(src, np.int64), tt)
    np.maximum.at(lu, np.asarray(dst, np.int64), tt)
    return lu


def loss_noise(w: Workload, step: int, n_rows: int, base_seed: int = 0) -> np.ndarray:
    """Seeded N(0,1) noise G [n_rows, d_attn] (float32) for one step's loss gradient."""
    return _rng(base_seed, w.cid, _G, step).standard_normal((n_rows, w.d_attn), dtype=np.float32)


def node_owner(n_nodes: int, n_workers: int, base_seed: int = 0, cid: int = 0) -> np.ndarray:
    """A node ownership map pi for n_workers workers: each node's owner drawn uniformly (int32 [n_nodes])."""
    return _rng(base_seed, cid, _OWNER).integers(0, n_workers, n_nodes).astype(np.int32)


def init_params_jodie(w: Workload, base_seed: int = 0, random_bias: bool = False, bias_scale: float = 0.1) -> dict:
    """JODIE's parameters: the recurrent cell W_ih [d_m, d_msg], W_hh [d_m, d_m] (Xavier-uniform), the time
    projection W_p [d_m, 1], b_p [d_m], the time encoder and the link decoder (as init_params)."""
    dm = w.d_mem
    rng = np.random.default_rng(np.random.SeedSequence([base_seed, w.cid, _PARAMS, 1]))
    p = {}
    for name, (fo, fi) in (("W_ih", (dm, w.d_msg)), ("W_hh", (dm, dm)), ("W_p", (dm, 1))):
        a = np.sqrt(6.0 / (fi + fo))
        p[name] = rng.uniform(-a, a, size=(fo, fi)).astype(np.float32)
    for name in ("b_ih", "b_hh", "b_p"):
        p[name] = (rng.uniform(-bias_scale, bias_scale, dm).astype(np.float32) if random_bias
                   else np.zeros(dm, np.float32))
    base = init_params(w, base_seed, random_bias, bias_scale)
    for k in ("time_w", "time_b", "W_d1", "b_d1", "W_d2", "b_d2"):
        p[k] = base[k]
    return p
