"""Helpers for the GPU parity tests: run the HIP path, run the oracle on the same inputs, compare."""

import sys

import numpy as np
import pytest
import torch

from oracle import tgn
from oracle.bf16 import round_bf16
from synth import loss_noise

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(x, y):
    """max|x - y| / max|y| (the per-tensor tolerance of the floating-point parity gate)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    if y.size == 0:
        return 0.0
    return float(np.abs(x - y).max() / max(np.abs(y).max(), 1e-30))


def to_np(t):
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy()
    return t.cpu().numpy()


def noise_for(w, step, n_rows):
    return loss_noise(w, step, max(n_rows, 1))


def dz_tensor(runner, w, step, n_tar):
    G = noise_for(w, step, runner.max_q)
    dz = (G / n_tar) if n_tar > 0 else np.zeros_like(G)
    return torch.from_numpy(dz.astype(np.float32)).to(runner.dev), G


def n_targets(stream, lo, hi):
    if stream.flags is None:
        return hi - lo
    return int(((stream.flags[lo:hi] & 3) == 0).sum())


def oracle_prec(w):
    return tgn.Prec("bf16" if w.dtype == "bf16" else "f32")


def mem_snapshot(runner):
    return to_np(runner.memory).copy(), runner.last_update.cpu().numpy().copy()


def compare_step(runner, w, stream, adj, b, tol, lag=1, check=None):
    """Run GPU step b and the oracle step from the same state; assert parity; return both results."""
    mem0, lu0 = mem_snapshot(runner)
    elo, ehi = runner.batch_range(b)
    if lag == 1:
        mlo, mhi = runner.batch_range(b - 1) if b > 0 else (0, 0)
    else:
        mlo, mhi = elo, ehi
    n_tar = n_targets(stream, elo, ehi)
    dz, G = dz_tensor(runner, w, b, n_tar)
    runner.lag = lag
    runner.step(b, dz)
    torch.cuda.synchronize()
    prec = oracle_prec(w)
    params = {k: v.float().cpu().numpy() for k, v in runner.params.items()}
    mem_b = tgn.batch_dict(stream, mlo, mhi) if mhi > mlo else None
    ref = tgn.step(prec, w, mem0, lu0, params, adj, stream.x, mem_b, tgn.batch_dict(stream, elo, ehi), G)
    gpu = {
        "n_uniq": int(runner.n_uniq.item()), "uniq": runner.uniq.cpu().numpy(), "winner": runner.winner.cpu().numpy(),
        "n_q": int(runner.n_q.item()), "q_node": runner.q_node.cpu().numpy(), "q_t": runner.q_t.cpu().numpy(),
        "nbr": runner.nbr.cpu().numpy(), "nt": runner.nt.cpu().numpy(), "neid": runner.neid.cpu().numpy(),
        "z": runner.z.cpu().numpy(), "mem": to_np(runner.memory), "lu": runner.last_update.cpu().numpy(),
        "msg": to_np(runner.msg), "dt": runner.dt.cpu().numpy(), "d_mem": runner.d_mem.cpu().numpy(),
        "grads": {k: v.cpu().numpy() for k, v in runner.grads.items()},
    }
    U, Q = gpu["n_uniq"], gpu["n_q"]
    # integer / copied outputs: bit-exact.  The library lists updated rows in
    # increasing order of their winning message; the oracle by node id.  Check
    # the library's order, then compare row by row in the oracle's order.
    assert U == len(ref.mp.uniq), (U, len(ref.mp.uniq))
    assert np.all(np.diff(gpu["winner"][:U]) > 0)
    perm = np.argsort(gpu["uniq"][:U], kind="stable")
    assert np.array_equal(gpu["uniq"][:U][perm], ref.mp.uniq)
    assert np.array_equal(gpu["winner"][:U][perm], ref.mp.winner)
    gpu["perm"] = perm
    assert Q == ref.q_node.size
    assert np.array_equal(gpu["q_node"][:Q], ref.q_node)
    assert np.array_equal(gpu["q_t"][:Q].view(np.uint32), ref.q_t.view(np.uint32))
    assert np.array_equal(gpu["nbr"][:Q], ref.nbr)
    assert np.array_equal(gpu["neid"][:Q], ref.neid)
    assert np.array_equal(gpu["nt"][:Q].view(np.uint32), ref.nt.view(np.uint32))
    assert np.array_equal(gpu["lu"].view(np.uint32), ref.mp.lu.view(np.uint32))
    touched = np.zeros(w.n_nodes, bool)
    touched[ref.mp.uniq] = True
    assert np.array_equal(gpu["mem"][~touched].view(np.uint32), np.asarray(mem0)[~touched].view(np.uint32))
    if U:
        assert np.array_equal(gpu["dt"][:U][perm].view(np.uint32), np.asarray(ref.mp.dt, np.float32).view(np.uint32))
    # floating point: normalised max error
    errs = {}
    if U:
        errs["msg"] = rel_err(gpu["msg"][:U][perm], ref.mp.msg)
        errs["mem"] = rel_err(gpu["mem"][ref.mp.uniq], ref.mp.h_new)
        errs["d_mem"] = rel_err(gpu["d_mem"][:U][perm], ref.d_mem)
    if Q:
        errs["z"] = rel_err(gpu["z"][:Q], ref.attn.z)
    for name, g in ref.grads.items():
        if name == "b_k":   # identically zero in exact arithmetic: compare against the W_k scale
            errs[name] = float(np.abs(gpu["grads"][name]).max() / max(np.abs(ref.grads["W_k"]).max(), 1e-30))
        elif np.abs(g).max() > 0:
            errs[name] = rel_err(gpu["grads"][name], g)
        else:
            errs[name] = float(np.abs(gpu["grads"][name]).max())
    worst = max(errs.items(), key=lambda kv: kv[1]) if errs else ("-", 0.0)
    log(f"  step {b}: U={U} Q={Q} worst {worst[0]}={worst[1]:.3e}")
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad
    if check:
        check(gpu, ref)
    return gpu, ref
