"""Small hand-sized inputs for the CPU pins and the GPU edge cases."""

from dataclasses import replace

import numpy as np

from synth import Stream, workload


def tiny_workload(**kw):
    base = dict(n_nodes=6, n_events=40, d_edge=2, d_mem=4, d_time=3, d_attn=4, n_heads=2,
                batch=8, k=3)
    base.update(kw)
    return replace(workload(1), **base)


def tiny_stream(w, seed=0, t_scale=10.0, tie_every=0, self_loops=True, flags_p=None):
    """A small stream with optional timestamp ties, self-loops and masks."""
    rng = np.random.default_rng(seed)
    E, N = w.n_events, w.n_nodes
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    if not self_loops:
        same = src == dst
        dst[same] = (dst[same] + 1) % N
    t = np.sort(rng.random(E) * t_scale).astype(np.float32)
    if tie_every:
        for i in range(tie_every, E, tie_every):
            t[i] = t[i - 1]
    x = rng.standard_normal((E, w.d_edge)).astype(np.float32) if w.d_edge else None
    neg = rng.integers(0, N, E).astype(np.int32)
    flags = None
    if flags_p is not None:
        rep = rng.random(E) < flags_p[0]
        pr = rep & (rng.random(E) < flags_p[1])
        flags = (rep.astype(np.uint8) + 2 * pr.astype(np.uint8)).astype(np.uint8)
    return Stream(w, src, dst, t, x, neg, flags)


def random_state(w, seed=1, t_max=0.0):
    rng = np.random.default_rng(seed)
    mem = rng.uniform(-1, 1, (w.n_nodes, w.d_mem)).astype(np.float32)
    lu = (rng.random(w.n_nodes) * t_max).astype(np.float32)
    return mem, lu
