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


_rel_err = rel_err


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


def compare_step(runner, w, stream, adj, b, tol, lag=1, check=None, loss="link"):
    """Run GPU step b and the oracle step from the same state; assert parity; return both results.

    loss="link": the step's dZ comes from the masked link-prediction loss (Eq. 13), as in training;
    loss="noise": dZ = G / n_tar with seeded G (the loss's masking with a linear stand-in)."""
    mem0, lu0 = mem_snapshot(runner)
    elo, ehi = runner.batch_range(b)
    if lag == 1:
        mlo, mhi = runner.batch_range(b - 1) if b > 0 else (0, 0)
    else:
        mlo, mhi = elo, ehi
    n_tar = n_targets(stream, elo, ehi)
    runner.lag = lag
    if loss == "link":
        G = None
        runner.step(b)
    else:
        dz, G = dz_tensor(runner, w, b, n_tar)
        runner.step(b, dz)
    torch.cuda.synchronize()
    prec = oracle_prec(w)
    params = {k: v.float().cpu().numpy() for k, v in runner.params.items()}
    mem_b = tgn.batch_dict(stream, mlo, mhi) if mhi > mlo else None
    ref = tgn.step(prec, w, mem0, lu0, params, adj, stream.x, mem_b, tgn.batch_dict(stream, elo, ehi), G, loss=loss)
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
    # floating point: normalised max error.  A ReLU decision whose pre-activation lies within rounding
    # distance of zero (|x| <= RELU_AMBIGUOUS * max|x| of its tensor) may go either way in a correct
    # float32 evaluation: both results are valid.  Each such decision in turn is inverted in the oracle
    # and kept inverted if that brings the oracle closer to the GPU (summed squared relative errors,
    # to which separate decisions contribute separately); the gate then applies to the closest result.
    amb = ambiguous_relu(ref, Q, n_tar if loss == "link" else 0)
    if len(amb) > RELU_MAX_AMBIGUOUS:
        raise AssertionError(f"{len(amb)} ReLU pre-activations within {RELU_AMBIGUOUS:g} of zero")
    chosen, best = [], step_errors(gpu, ref, runner, U, Q, n_tar, perm, loss)
    for cand in amb:
        trial = chosen + [cand]
        r = tgn.step(prec, w, mem0, lu0, params, adj, stream.x, mem_b, tgn.batch_dict(stream, elo, ehi), G,
                     loss=loss, flips=relu_flips(ref, trial))
        e = step_errors(gpu, r, runner, U, Q, n_tar, perm, loss)
        if e[1] < best[1]:
            chosen, best, ref = trial, e, r
    errs = best[0]
    worst = max(errs.items(), key=lambda kv: kv[1]) if errs else ("-", 0.0)
    note = f" ({len(amb)} ReLU decisions within rounding of zero; {len(chosen)} taken the other way)" if amb else ""
    log(f"  step {b}: U={U} Q={Q} worst {worst[0]}={worst[1]:.3e}{note}")
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad
    if check:
        check(gpu, ref)
    return gpu, ref


RELU_AMBIGUOUS = 1e-6      # relative to the tensor's max: above the float32 evaluation error of these inputs
RELU_MAX_AMBIGUOUS = 32


def ambiguous_relu(ref, Q, n_tar):
    """(site, flat index) of the ReLU decisions of the merge layer and the decoder that lie within
    RELU_AMBIGUOUS of zero."""
    out = []
    sites = [("m1", ref.attn.m1[:Q])]
    if n_tar and ref.link is not None:
        sites += [("pos", ref.link.pre_pos), ("neg", ref.link.pre_neg)]
    for name, x in sites:
        if x.size == 0:
            continue
        idx = np.nonzero(np.abs(x).ravel() <= RELU_AMBIGUOUS * np.abs(x).max())[0]
        out += [(name, int(i)) for i in idx]
    return out


def relu_flips(ref, chosen):
    shapes = {"m1": ref.attn.m1.shape}
    if ref.link is not None:
        shapes.update(pos=ref.link.pre_pos.shape, neg=ref.link.pre_neg.shape)
    flips = {k: np.zeros(v, bool) for k, v in shapes.items()}
    for site, i in chosen:
        flips[site].ravel()[i] = True
    return flips


def step_errors(gpu, ref, runner, U, Q, n_tar, perm, loss):
    """Per-tensor max-norm relative errors (the gate), and the sum over tensors of the squared
    Frobenius-norm relative errors (to rank alternative oracle results)."""
    errs, sq = {}, [0.0]

    def rel_err(x, y):
        x = np.asarray(x, np.float64)
        y = np.asarray(y, np.float64)
        if y.size:
            sq[0] += float(((x - y) ** 2).sum() / max((y ** 2).sum(), 1e-300))
        return _rel_err(x, y)

    if U:
        errs["msg"] = rel_err(gpu["msg"][:U][perm], ref.mp.msg)
        errs["mem"] = rel_err(gpu["mem"][ref.mp.uniq], ref.mp.h_new)
        errs["d_mem"] = rel_err(gpu["d_mem"][:U][perm], ref.d_mem)
    if Q:
        errs["z"] = rel_err(gpu["z"][:Q], ref.attn.z)
    if loss == "link":
        gpu["loss"] = float(runner.loss.item())
        errs["loss"] = abs(gpu["loss"] - ref.link.loss) / max(abs(ref.link.loss), 1e-30) if n_tar else abs(gpu["loss"])
        if n_tar:
            sc = runner.scores.cpu().numpy()
            errs["scores"] = rel_err(np.concatenate([sc[0, :n_tar], sc[1, :n_tar]]),
                                     np.concatenate([ref.link.s_pos, ref.link.s_neg]))
            errs["dz"] = rel_err(runner.dz[:Q].cpu().numpy(), ref.link.dz)
    for name, g in ref.grads.items():
        if name == "b_k":   # identically zero in exact arithmetic: compare against the W_k scale
            errs[name] = float(np.abs(gpu["grads"][name]).max() / max(np.abs(ref.grads["W_k"]).max(), 1e-30))
        elif np.abs(g).max() > 0:
            errs[name] = rel_err(gpu["grads"][name], g)
        else:
            errs[name] = float(np.abs(gpu["grads"][name]).max())
    return errs, sq[0]


def query_nodes_of(stream, w, batches):
    """Every node queried by the target events of the given batches (src, dst and negative)."""
    out = []
    for b in batches:
        lo, hi = b * w.batch, min(stream.n_events, (b + 1) * w.batch)
        tar = tgn.target_mask(stream.flags[lo:hi] if stream.flags is not None else None, hi - lo)
        out += [stream.src[lo:hi][tar], stream.dst[lo:hi][tar], stream.neg[lo:hi][tar]]
    return np.unique(np.concatenate(out).astype(np.int64))


def check_csr_full_size(runner, stream, w, adj, nodes):
    """The GPU-built adjacency at full size: every offset against the node degrees of the stream, and
    the whole lists of ``nodes`` element by element against the oracle's adjacency restricted to them."""
    deg = np.bincount(stream.src, minlength=w.n_nodes) + np.bincount(stream.dst, minlength=w.n_nodes)
    off = runner.csr_off.cpu().numpy()
    assert off[0] == 0 and np.array_equal(np.diff(off), deg)
    lo, hi = off[nodes], off[nodes + 1]
    n = hi - lo
    idx = np.repeat(lo - np.concatenate([[0], np.cumsum(n)[:-1]]), n) + np.arange(n.sum())
    ti = torch.from_numpy(idx).to(runner.dev)
    olo, ohi = adj.off[nodes], adj.off[nodes + 1]
    assert np.array_equal(ohi - olo, n)
    oidx = np.repeat(olo - np.concatenate([[0], np.cumsum(n)[:-1]]), n) + np.arange(n.sum())
    assert np.array_equal(runner.csr_nbr[ti].cpu().numpy(), adj.nbr[oidx])
    assert np.array_equal(runner.csr_eid[ti].cpu().numpy(), adj.eid[oidx])
    assert np.array_equal(runner.csr_t[ti].cpu().numpy().view(np.uint32), adj.t[oidx].view(np.uint32))
    log(f"  adjacency: {off.size - 1} offsets, the lists of {nodes.size} queried nodes ({int(n.sum())} entries) "
        "bit-exact")


def compare_step_sampled(runner, w, stream, b, tol, n_sample, adj, seed=0):
    """Full-size step b (lag-1) with the loss gradient restricted to the queries of a sample of target events.

    The GPU runs the whole step at its real size, exactly as the benchmark
    does.  Compared bit for bit: the whole memory phase's integer and copied
    outputs, and the queries and most-recent-k neighbours of EVERY query row
    of the step (``adj`` is the oracle's adjacency restricted to the queried
    nodes).  dZ is nonzero only on the src / dst / negative rows of
    ``n_sample`` target events; because the backward is linear in dZ, every
    gradient and d_mem then equals the oracle's step over those events alone,
    which the oracle computes with the full memory phase of batch b-1.
    Floating-point tensors (messages, memory rows, the sampled queries'
    embeddings, d_mem, every gradient) are gated at ``tol``.
    """
    mem0, lu0 = mem_snapshot(runner)
    elo, ehi = runner.batch_range(b)
    mlo, mhi = runner.batch_range(b - 1)
    flags = stream.flags[elo:ehi] if stream.flags is not None else None
    tar = np.nonzero(tgn.target_mask(flags, ehi - elo))[0]
    n_tar = tar.size
    pick = np.sort(np.random.default_rng(seed).choice(n_tar, size=min(n_sample, n_tar), replace=False))
    rows = np.concatenate([pick, n_tar + pick, 2 * n_tar + pick])
    G = noise_for(w, b, runner.max_q)
    dz = np.zeros_like(G)
    dz[rows] = G[rows] / np.float32(n_tar)
    runner.lag = 1
    runner.step(b, torch.from_numpy(dz).to(runner.dev))
    torch.cuda.synchronize()

    # every query row of the step: queries and sampled neighbours, bit for bit
    Q = int(runner.n_q.item())
    assert Q == 3 * n_tar
    q_all, qt_all, _ = tgn.queries(tgn.batch_dict(stream, elo, ehi))
    assert np.array_equal(runner.q_node[:Q].cpu().numpy(), q_all)
    assert np.array_equal(runner.q_t[:Q].cpu().numpy().view(np.uint32), qt_all.view(np.uint32))
    nbr_all, nt_all, neid_all = tgn.sample_recent(adj, q_all, qt_all, w.k)
    assert np.array_equal(runner.nbr[:Q].cpu().numpy(), nbr_all)
    assert np.array_equal(runner.neid[:Q].cpu().numpy(), neid_all)
    assert np.array_equal(runner.nt[:Q].cpu().numpy().view(np.uint32), nt_all.view(np.uint32))
    log(f"  step {b}: all {Q} query rows' neighbours bit-exact ({int((nbr_all >= 0).sum())} valid slots)")
    del nbr_all, nt_all, neid_all

    ev = (elo + tar[pick]).astype(np.int64)
    emb = {"src": stream.src[ev], "dst": stream.dst[ev], "t": stream.t[ev], "eid": ev, "neg": stream.neg[ev]}
    noise_sub = G[rows].astype(np.float64) * (pick.size / n_tar)
    params = {k: v.float().cpu().numpy() for k, v in runner.params.items()}
    mb = tgn.batch_dict(stream, mlo, mhi)
    ref = tgn.step(oracle_prec(w), w, mem0, lu0, params, adj, stream.x, mb, emb, noise_sub)
    spread = {}
    if w.dtype == "bf16":
        # diagnostic only (not a gate): how far the oracle's own bf16 gradients move when the values
        # before each bf16 rounding carry a 1e-7 relative perturbation, the size of an fp32 evaluation's
        alt = tgn.step(_PerturbedPrec("bf16", 1), w, mem0, lu0, params, adj, stream.x, mb, emb, noise_sub)
        for name, g in ref.grads.items():
            if name != "b_k":
                spread[name] = rel_err(alt.grads[name], g)
        spread["d_mem"] = rel_err(alt.d_mem, ref.d_mem)

    U = int(runner.n_uniq.item())
    uniq = runner.uniq[:U].cpu().numpy()
    winner = runner.winner[:U].cpu().numpy()
    assert U == len(ref.mp.uniq)
    assert np.all(np.diff(winner) > 0)
    perm = np.argsort(uniq, kind="stable")
    assert np.array_equal(uniq[perm], ref.mp.uniq)
    assert np.array_equal(winner[perm], ref.mp.winner)
    dt = runner.dt[:U].cpu().numpy()
    assert np.array_equal(dt[perm].view(np.uint32), np.asarray(ref.mp.dt, np.float32).view(np.uint32))
    mem1 = to_np(runner.memory)
    lu1 = runner.last_update.cpu().numpy()
    assert np.array_equal(lu1.view(np.uint32), ref.mp.lu.view(np.uint32))
    h_new = mem1[ref.mp.uniq].copy()
    mem1[ref.mp.uniq] = mem0[ref.mp.uniq]      # rows outside the update set must be untouched, bit for bit
    assert np.array_equal(mem1.view(np.uint32), np.asarray(mem0).view(np.uint32))
    del mem1
    # the sampled queries' embeddings
    ti = torch.from_numpy(rows).to(runner.dev)
    assert np.array_equal(runner.q_node[ti].cpu().numpy(), ref.q_node)
    errs = {
        "msg": rel_err(to_np(runner.msg[:U])[perm], ref.mp.msg),
        "mem": rel_err(h_new, ref.mp.h_new),
        "d_mem": rel_err(runner.d_mem[:U].cpu().numpy()[perm], ref.d_mem),
        "z": rel_err(runner.z[ti].cpu().numpy(), ref.attn.z),
    }
    for name, g in ref.grads.items():
        gg = runner.grads[name].cpu().numpy()
        if name == "b_k":
            errs[name] = float(np.abs(gg).max() / max(np.abs(ref.grads["W_k"]).max(), 1e-30))
        else:
            errs[name] = rel_err(gg, g)
    worst = max(errs.items(), key=lambda kv: kv[1])
    log(f"  step {b}: U={U} Q={Q} sampled events={pick.size} worst {worst[0]}={worst[1]:.3e} (gate {tol:.0e})")
    log("  errors: " + ", ".join(f"{k}={v:.1e}" for k, v in sorted(errs.items())))
    if spread:
        log("  oracle's own bf16 spread (diagnostic): " + ", ".join(f"{k}={v:.1e}" for k, v in sorted(spread.items())))
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad


class _PerturbedPrec(tgn.Prec):
    """The oracle's bf16 mode with a relative 1e-7 perturbation of every computed value just before it
    is rounded to bf16 (weights, which are rounded once from fixed parameters, are left alone)."""

    def __init__(self, mode, seed):
        super().__init__(mode)
        self._rng = np.random.default_rng(seed)

    def pack(self, x):
        x = np.asarray(x, np.float64)
        return super().pack(x * (1.0 + 1e-7 * self._rng.standard_normal(x.shape)))

    def weight(self, x):
        return tgn.Prec.pack(self, x)
