"""Literal per-event reading of Eq. 1-2 (test infrastructure only).

Events are applied one at a time in stream order: both messages of event k
are formed from the memories just before t_k (the state after event k-1),
then both endpoint memories are replaced.  This is the semantics a batch of
size 1 must reproduce.  The code is deliberately separate from ``tgn`` (its
own GRU arithmetic, its own message assembly) so that it can pin it.
"""

import math

import numpy as np


def _sig(v):
    return 1.0 / (1.0 + math.exp(-v)) if v >= -700 else 0.0


def gru_scalar(x, h, W_ih, W_hh, b_ih, b_hh):
    """GRU cell expanded element by element in plain Python floats."""
    dm = len(h)
    D = len(x)

    def lin(W, b, v, row):
        acc = float(b[row])
        for c in range(len(v)):
            acc += float(W[row][c]) * float(v[c])
        return acc

    out = []
    for j in range(dm):
        r = _sig(lin(W_ih, b_ih, x, j) + lin(W_hh, b_hh, h, j))
        z = _sig(lin(W_ih, b_ih, x, dm + j) + lin(W_hh, b_hh, h, dm + j))
        n = math.tanh(lin(W_ih, b_ih, x, 2 * dm + j) + r * lin(W_hh, b_hh, h, 2 * dm + j))
        out.append((1.0 - z) * n + z * float(h[j]))
    assert D == len(x)
    return out


def _gru_vec(x, h, W_ih, W_hh, b_ih, b_hh):
    dm = h.shape[0]
    a = W_ih @ x + b_ih
    c = W_hh @ h + b_hh
    r = 1.0 / (1.0 + np.exp(-(a[:dm] + c[:dm])))
    z = 1.0 / (1.0 + np.exp(-(a[dm:2 * dm] + c[dm:2 * dm])))
    n = np.tanh(a[2 * dm:] + r * c[2 * dm:])
    return (1.0 - z) * n + z * h


def replay_events(src, dst, t, x, flags, mem, lu, params, scalar=False):
    """Apply events one by one; returns the final (memory, last_update) in float64.

    Pruned events (flag bit 1) are skipped; every other event updates both
    endpoints.  Time encoding: cos(w * (t - lu) + b) in float64 without any
    intermediate rounding.
    """
    mem = np.array(mem, dtype=np.float64, copy=True)
    lu = np.array(lu, dtype=np.float64, copy=True)
    W_ih = np.asarray(params["W_ih"], np.float64)
    W_hh = np.asarray(params["W_hh"], np.float64)
    b_ih = np.asarray(params["b_ih"], np.float64)
    b_hh = np.asarray(params["b_hh"], np.float64)
    tw = np.asarray(params["time_w"], np.float64)
    tb = np.asarray(params["time_b"], np.float64)
    for e in range(len(src)):
        if flags is not None and (int(flags[e]) & 2):
            continue
        u, v, te = int(src[e]), int(dst[e]), float(t[e])
        feats = [] if x is None else [np.asarray(x[e], np.float64)]
        m_u, m_v = mem[u].copy(), mem[v].copy()
        s_u = np.concatenate([m_u, m_v, np.cos(tw * (te - lu[u]) + tb)] + feats)
        s_v = np.concatenate([m_v, m_u, np.cos(tw * (te - lu[v]) + tb)] + feats)
        if scalar:
            new_u = np.array(gru_scalar(s_u, m_u, W_ih, W_hh, b_ih, b_hh))
            new_v = np.array(gru_scalar(s_v, m_v, W_ih, W_hh, b_ih, b_hh))
        else:
            new_u = _gru_vec(s_u, m_u, W_ih, W_hh, b_ih, b_hh)
            new_v = _gru_vec(s_v, m_v, W_ih, W_hh, b_ih, b_hh)
        mem[u] = new_u
        mem[v] = new_v          # a self-loop computes the same value twice
        lu[u] = te
        lu[v] = te
    return mem, lu
