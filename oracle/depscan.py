"""Offline backward dependency scan and mixed-batch construction (Algorithm 1, Section IV-B).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain Python sets and
lists, in the algorithm's order and notation.  For one worker p and one
synchronization window W_q (Definition 1: K consecutive batches):

* the batches are visited in reverse chronological order;
* B_tar^s = the events of batch s whose source u is owned by p;
* the frontier F gains the remote destinations of those target events;
* every event of batch s that is not a target of p (its source is remote)
  and touches F becomes an auxiliary replay event of batch s (once: the set
  I_aux of inserted event ids), and its remote endpoints join F;
* after the scan, F is the candidate boundary refresh set N_sync;
* each mixed batch is sort_t(B_tar^s u B_aux^s) (Eq. 5).

Within a batch the algorithm does not fix the order in which events are
visited; this reading visits them in reverse chronological order (latest
first, by (t, eid)), the direction of the scan, so that a node an event adds
to F can pull in the earlier events of the same batch that touch it.
"""

import numpy as np


def backward_scan(src, dst, owner, p, batches):
    """Algorithm 1 for worker p over one window.

    batches: list of lists of event ids of the window's batches, chronological
    (each batch's ids in chronological order).  Returns (tar, aux, n_sync):
    per batch the target and auxiliary event ids, and the refresh set.
    """
    tar = [[] for _ in batches]
    aux = [[] for _ in batches]
    F = set()
    I_aux = set()
    for s in reversed(range(len(batches))):
        B = batches[s]
        tar[s] = [e for e in B if owner[src[e]] == p]
        F |= {int(dst[e]) for e in tar[s] if owner[dst[e]] != p}
        for e in reversed(B):
            u, v = int(src[e]), int(dst[e])
            if (u in F or v in F) and owner[u] != p:
                if e not in I_aux:
                    aux[s].append(e)
                    I_aux.add(e)
                F |= {i for i in (u, v) if owner[i] != p}
    return tar, aux, F


def mixed_batch(t, tar_s, aux_s):
    """sort_t(B_tar u B_aux) with the event-type mask: (event ids, is_aux) in (t, eid) order."""
    ids = sorted(set(tar_s) | set(aux_s), key=lambda e: (float(t[e]), e))
    aux_set = set(aux_s)
    return ids, [e in aux_set for e in ids]


def scan_stream(src, dst, t, owner, n_workers, batch, window):
    """Algorithm 1 for every worker and every window of a stream split into batches of `batch`
    events and windows of `window` batches.  Returns role [P, E] (0 = not in the worker's mixed
    batches, 1 = target, 2 = auxiliary replay) and n_sync[p][q] (sets)."""
    E = len(src)
    n_batches = (E + batch - 1) // batch
    n_windows = (n_batches + window - 1) // window
    role = np.zeros((n_workers, E), np.uint8)
    n_sync = [[None] * n_windows for _ in range(n_workers)]
    for q in range(n_windows):
        bl = [list(range(b * batch, min(E, (b + 1) * batch)))
              for b in range(q * window, min(n_batches, (q + 1) * window))]
        for p in range(n_workers):
            tar, aux, F = backward_scan(src, dst, owner, p, bl)
            for s in range(len(bl)):
                role[p, tar[s]] = 1
                role[p, aux[s]] = 2
            n_sync[p][q] = F
    return role, n_sync
