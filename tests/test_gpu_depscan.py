"""GPU parity of the offline dependency scan and mixed-batch construction (Algorithm 1) through the C ABI.

Integer work: the roles (target / auxiliary replay / absent) of every event for every worker, the
frontier bitmaps (refresh sets) and the compacted mixed batches must equal the oracle's bit for bit.
"""

import time

import numpy as np
import pytest
import torch

from oracle import depscan
from paper_2608_16305_amd import mtgnn as M
from synth import make_stream, node_owner, workload
from tests._gpu import log, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


def _gpu_scan(src, dst, owner, P, batch, window):
    E, N = len(src), len(owner)
    n_windows = -(-(-(-E // batch)) // window)
    words = -(-N // 32)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()   # noqa: E731
    role = torch.full((P, E), 255, dtype=torch.uint8, device="cuda")
    sync = torch.full((P, n_windows, words), -1, dtype=torch.int32, device="cuda")
    M.mtgnn_dependency_scan(d(src), d(dst), d(owner), P, batch, window, role, sync)
    torch.cuda.synchronize()
    return role, sync, n_windows, words


def _bits(nodes, words):
    b = np.zeros(words * 32, bool)
    b[list(nodes)] = True
    return (b.reshape(words, 32).astype(np.uint64) << np.arange(32, dtype=np.uint64)).sum(1).astype(np.uint32)


def _check_mixed(role_p, batch, t):
    E = role_p.numel()
    nb = -(-E // batch)
    eid = torch.full((E,), -7, dtype=torch.int32, device="cuda")
    fl = torch.full((E,), 9, dtype=torch.uint8, device="cuda")
    off = torch.full((nb + 1,), -7, dtype=torch.int32, device="cuda")
    ws = M.alloc_bytes(M.workspace_bytes(M.OP_MIXED_BATCHES, None, E, 0))
    M.mtgnn_mixed_batches(role_p, batch, eid, fl, off, ws)
    torch.cuda.synchronize()
    r = role_p.cpu().numpy()
    ids = np.nonzero(r)[0]
    n = ids.size
    mixed, is_aux = depscan.mixed_batch(t, list(ids[r[ids] == 1]), list(ids[r[ids] == 2]))
    assert np.array_equal(eid[:n].cpu().numpy(), np.array(mixed, np.int32))
    assert np.array_equal(fl[:n].cpu().numpy(), np.array(is_aux, np.uint8))
    starts = np.searchsorted(ids, np.arange(nb + 1) * batch)
    assert np.array_equal(off.cpu().numpy(), starts.astype(np.int32))


@pytest.mark.parametrize("seed,N,E,P,batch,window", [(0, 50, 3000, 4, 100, 5), (1, 9, 777, 3, 50, 4),
                                                     (2, 400, 5000, 8, 333, 7), (3, 30, 64, 2, 1, 16)])
def test_dependency_scan_small_streams(seed, N, E, P, batch, window):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    dst[::11] = src[::11]            # self-loops
    t = np.sort(rng.random(E) * 100).astype(np.float32)
    owner = rng.integers(0, P, N).astype(np.int32)
    role, sync, nw, words = _gpu_scan(src, dst, owner, P, batch, window)
    ref_role, ref_sync = depscan.scan_stream(src, dst, t, owner, P, batch, window)
    assert np.array_equal(role.cpu().numpy(), ref_role)
    got = sync.cpu().numpy().view(np.uint32)
    for p in range(P):
        for q in range(nw):
            assert np.array_equal(got[p, q], _bits(ref_sync[p][q], words)), (p, q)
    for p in range(P):
        _check_mixed(role[p], batch, t)
    log(f"  {P} workers x {nw} windows: roles, refresh sets and mixed batches bit-exact "
        f"({int((ref_role == 2).sum())} auxiliary events)")


def test_dependency_scan_skewed_stream():
    """The skewed stream (1M nodes, 10M events, Zipf(1.2)), 8 workers, batches of 4,000, windows of 10
    batches: every event's target role for every worker, and the whole scan (roles and refresh set) of the
    first, a middle and the last window for every worker, against the oracle."""
    w = workload(3)
    log("[depscan] generating the skewed stream")
    s = make_stream(w)
    P, batch, window = 8, w.batch, 10
    owner = node_owner(w.n_nodes, P)
    t0 = time.time()
    role, sync, nw, words = _gpu_scan(s.src, s.dst, owner, P, batch, window)
    log(f"[depscan] {P} x {nw} scans on the GPU in {time.time() - t0:.2f} s (with uploads)")
    r = role.cpu().numpy()
    tgt = owner[s.src]
    for p in range(P):
        assert np.array_equal(r[p] == 1, tgt == p)
    log(f"  replay fraction per worker: {((r == 2).sum(1) / (r != 0).sum(1)).round(3).tolist()}")
    got = sync.cpu().numpy().view(np.uint32)
    for q in (0, nw // 2, nw - 1):
        lo_b, hi_b = q * window, min(w.n_batches, (q + 1) * window)
        bl = [list(range(b * batch, min(w.n_events, (b + 1) * batch))) for b in range(lo_b, hi_b)]
        e_lo, e_hi = bl[0][0], bl[-1][-1] + 1
        for p in range(P):
            tar, aux, F = depscan.backward_scan(s.src, s.dst, owner, p, bl)
            exp = np.zeros(e_hi - e_lo, np.uint8)
            exp[np.concatenate([np.array(x, np.int64) for x in tar]) - e_lo] = 1
            a = [np.array(x, np.int64) for x in aux if x]
            if a:
                exp[np.concatenate(a) - e_lo] = 2
            assert np.array_equal(r[p, e_lo:e_hi], exp), (p, q)
            assert np.array_equal(got[p, q], _bits(F, words)), (p, q)
    _check_mixed(role[0], batch, s.t)
    log(f"  windows 0, {nw // 2}, {nw - 1}: every worker's scan bit-exact; worker 0's mixed batches bit-exact")
