"""GPU parity of the JODIE variant's step (recurrent update, time projection, masked link loss and the
backward) through the C ABI, against the oracle, each step from the GPU's state before it."""

from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import jodie, tgn
from oracle.bf16 import round_bf16
from synth import init_params_jodie, make_stream, window_state, workload
from tests._gpu import RELU_AMBIGUOUS, log, needs_gpu, rel_err, to_np
from tests._tiny import random_state, tiny_stream, tiny_workload

pytestmark = [pytest.mark.gpu, needs_gpu]


def _compare(r, w, s, b, tol):
    from oracle.tgn import Prec
    mem0, lu0 = to_np(r.memory).copy(), r.last_update.cpu().numpy().copy()
    r.step(b)
    torch.cuda.synchronize()
    elo, ehi = r.batch_range(b)
    mb = tgn.batch_dict(s, *r.batch_range(b - 1)) if b > 0 else None
    eb = tgn.batch_dict(s, elo, ehi)
    params = {k: v.float().cpu().numpy() for k, v in r.params.items()}
    prec = Prec("bf16" if w.dtype == "bf16" else "f32")
    ref = jodie.step(prec, w, mem0, lu0, params, s.x, mb, eb, r.time_scale)
    U, Q = int(r.n_uniq.item()), int(r.n_q.item())
    assert U == len(ref.mp.uniq) and Q == ref.q_node.size
    perm = np.argsort(r.uniq[:U].cpu().numpy(), kind="stable")
    assert np.array_equal(r.uniq[:U].cpu().numpy()[perm], ref.mp.uniq)
    assert np.array_equal(r.winner[:U].cpu().numpy()[perm], ref.mp.winner)
    mem1 = to_np(r.memory)
    assert np.array_equal(r.last_update.cpu().numpy().view(np.uint32), ref.mp.lu.view(np.uint32))
    touched = np.zeros(w.n_nodes, bool)
    touched[ref.mp.uniq] = True
    assert np.array_equal(mem1[~touched].view(np.uint32), np.asarray(mem0)[~touched].view(np.uint32))

    def errors(ref):
        e = {"mem": rel_err(mem1[ref.mp.uniq], ref.mp.h_new) if U else 0.0}
        if Q:
            e["z"] = rel_err(r.z[:Q].cpu().numpy(), ref.z)
            e["loss"] = abs(r.loss.item() - ref.link.loss) / abs(ref.link.loss)
            e["dz"] = rel_err(r.dz[:Q].cpu().numpy(), ref.link.dz)
        if U:
            e["d_mem"] = rel_err(r.d_mem[:U].cpu().numpy()[perm], ref.d_mem)
        for k, gref in ref.grads.items():
            gg = r.grads[k].cpu().numpy()
            e[k] = rel_err(gg, gref) if np.abs(gref).max() > 0 else float(np.abs(gg).max())
        return e

    errs = errors(ref)
    # decoder ReLU decisions within rounding distance of zero may go either way (as in the TGN step)
    if Q and ref.n_tar:
        for site, x in (("pos", ref.link.pre_pos), ("neg", ref.link.pre_neg)):
            for i in np.nonzero(np.abs(x).ravel() <= RELU_AMBIGUOUS * np.abs(x).max())[0]:
                fl = {"pos": np.zeros_like(ref.link.pre_pos, bool), "neg": np.zeros_like(ref.link.pre_neg, bool)}
                fl[site].ravel()[i] = True
                alt = jodie.step(prec, w, mem0, lu0, params, s.x, mb, eb, r.time_scale, flips=fl)
                ea = errors(alt)
                if max(ea.values()) < max(errs.values()):
                    errs = ea
    worst = max(errs.items(), key=lambda kv: kv[1])
    log(f"  step {b}: U={U} Q={Q} worst {worst[0]}={worst[1]:.2e}")
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad


def _runner(w, s, mem, lu, seed_bias=True):
    from paper_2608_16305_amd.jodie_step import JodieStep
    return JodieStep(w, s, init_params_jodie(w, random_bias=seed_bias), mem, lu)


def test_jodie_tiny_stream_from_empty_memory():
    w = workload(1)
    s = make_stream(w)
    r = _runner(w, s, np.zeros((w.n_nodes, w.d_mem), np.float32), np.zeros(w.n_nodes, np.float32))
    for b in range(5):
        _compare(r, w, s, b, 1e-4)


def test_jodie_skewed_window():
    w = workload(3)
    log("[jodie] skewed stream window")
    s = make_stream(w)
    mem, lu = window_state(w, s, w.window_b0)
    r = _runner(w, s, mem, lu)
    for b in range(w.window_b0, w.window_b0 + 3):
        _compare(r, w, s, b, 1e-4)


def test_jodie_masks_ragged_and_bf16():
    w = tiny_workload(n_nodes=61, n_events=600, batch=37, k=1, d_mem=37, d_time=11, d_edge=5, d_attn=37, n_heads=1)
    s = tiny_stream(w, seed=8, t_scale=300.0, tie_every=5, flags_p=(0.3, 0.3))
    s.flags[74:111] = 3     # an all-pruned batch
    mem, lu = random_state(w, seed=4)
    r = _runner(w, s, mem, lu)
    for b in range(0, 6):
        _compare(r, w, s, b, 1e-4)
    wb = replace(tiny_workload(n_nodes=50, n_events=800, batch=80, k=1, d_mem=16, d_time=8, d_edge=0, d_attn=16,
                               n_heads=1), dtype="bf16")
    sb = tiny_stream(wb, seed=9, t_scale=100.0, flags_p=(0.25, 0.1))
    mem, lu = random_state(wb, seed=5)
    rb = _runner(wb, sb, round_bf16(mem), lu)
    for b in range(1, 5):
        _compare(rb, wb, sb, b, 2e-2)
