"""Adaptive runtime controller (Section V, Algorithm 2) -- TEST INFRASTRUCTURE ONLY.

Plain Python/NumPy, in the paper's notation:

* ``ema``            -- Eq. 6 and Eq. 8: the first observation initialises the
                        average (previous average 0), later ones blend with the
                        factor (alpha for gradient norms, beta for batch times);
* ``sync_decision``  -- Eq. 7: S_r = 0 (skip the boundary refresh) iff r > 0,
                        the gradient EMA is positive and g_{r-1} < tau_g EMA;
* ``heavy_load``     -- Eq. 9: H_r = 1 iff r > 0, the time EMA is positive and
                        c_{r-1} > tau_c EMA;
* ``prune_aux``      -- Eq. 10-11: under heavy load the auxiliary replay events
                        (source not owned by the worker: event-type mask bit 0)
                        are removed (marked pruned, bit 1); target events stay;
* ``cache_refresh``  -- Eq. 25: the cached state of every node of the refresh
                        set takes the authoritative state (memory row and
                        last update time);
* ``grad_norm``      -- g_r, the Euclidean norm of every parameter gradient;
* ``adam``           -- the parameter update of Algorithm 2 (Adam with bias
                        correction; the paper names no optimizer, TGN trains
                        with Adam);
* ``Controller``     -- the state of Algorithm 2 (g_bar, g_last, c_bar, c_prev)
                        and its per-batch decisions.
"""

import math

import numpy as np


def ema(prev: float, x: float, factor: float) -> float:
    return float(x) if prev == 0 else factor * float(x) + (1.0 - factor) * prev


def sync_decision(r: int, g_last: float, g_bar: float, tau_g: float) -> int:
    return 0 if (r > 0 and g_bar > 0 and g_last < tau_g * g_bar) else 1


def heavy_load(r: int, c_prev: float, c_bar: float, tau_c: float) -> int:
    return 1 if (r > 0 and c_bar > 0 and c_prev > tau_c * c_bar) else 0


def prune_aux(flags, heavy: int) -> np.ndarray:
    """The event-type masks of a mixed batch after PruneAux: bit 1 (pruned) on every auxiliary event
    (bit 0) when heavy, on none otherwise."""
    f = np.asarray(flags, np.uint8)
    aux = (f & 1) != 0
    return np.where(aux & bool(heavy), f | 2, f & ~np.uint8(2)).astype(np.uint8)


def cache_refresh(cache_mem, cache_lu, auth_mem, auth_lu, nodes):
    m = np.array(cache_mem, copy=True)
    l = np.array(cache_lu, copy=True)
    idx = np.asarray(sorted(nodes), np.int64)
    if idx.size:
        m[idx] = np.asarray(auth_mem)[idx]
        l[idx] = np.asarray(auth_lu)[idx]
    return m, l


def grad_norm(grads) -> float:
    return math.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in grads))


def adam(theta, grad, m, v, t: int, lr: float, beta1: float, beta2: float, eps: float):
    """One Adam step (t >= 1); float64 arithmetic."""
    g = np.asarray(grad, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1 - beta2) * g * g
    mh = m / (1 - beta1 ** t)
    vh = v / (1 - beta2 ** t)
    return np.asarray(theta, np.float64) - lr * mh / (np.sqrt(vh) + eps), m, v


class Controller:
    """Algorithm 2's controller state for one worker."""

    def __init__(self, alpha, beta, tau_g, tau_c, interval):
        self.alpha, self.beta, self.tau_g, self.tau_c, self.K = alpha, beta, tau_g, tau_c, interval
        self.g_bar = self.g_last = self.c_bar = self.c_prev = 0.0

    def boundary(self, r: int) -> bool:
        return r % self.K == 0

    def sync(self, r: int) -> int:
        return sync_decision(r, self.g_last, self.g_bar, self.tau_g)

    def heavy(self, r: int) -> int:
        return heavy_load(r, self.c_prev, self.c_bar, self.tau_c)

    def observe(self, g_r: float, c_r: float):
        self.g_bar = ema(self.g_bar, g_r, self.alpha)
        self.g_last = float(g_r)
        self.c_bar = ema(self.c_bar, c_r, self.beta)
        self.c_prev = float(c_r)
