"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, exact rational arithmetic, brute force, an independent per-event
reading of Eq. 1-2, a library routine (torch on the CPU, float64), finite
differences, or an invariant the paper states.
"""

import json
import math
import os
import struct
from dataclasses import replace
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import sequential, tgn
from oracle.bf16 import round_bf16
from synth import init_params, workload
from tests._tiny import random_state, tiny_stream, tiny_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


def _to_f32(fr: Fraction) -> float:
    """Round an exact rational to the nearest binary32 (ties to even) by bisection on the bit pattern."""
    x = float(fr)                       # nearest double (ties-to-even)
    f = struct.unpack("<f", struct.pack("<f", x))[0]   # double -> single, nearest-even
    # correct a possible double-rounding error by checking the neighbours exactly
    best, best_err = f, abs(Fraction(f) - fr)
    for cand in (np.nextafter(F32(f), F32(np.inf)), np.nextafter(F32(f), F32(-np.inf))):
        err = abs(Fraction(float(cand)) - fr)
        if err < best_err or (err == best_err and (struct.unpack("<I", struct.pack("<f", float(cand)))[0] & 1) == 0):
            best, best_err = float(cand), err
    return best


# --------------------------------------------------------------------------- time encoding

def test_time_encoding_special_cases():
    p64 = tgn.Prec("f64")
    w = np.array([1.0, 0.5, 0.0, 1e-3], F32)
    b = np.array([0.0, 0.25, 0.0, -1.0], F32)
    # dt = 0 -> cos(b); w = b = 0 -> 1
    phi0 = tgn.time_encode(p64, np.zeros(1), w, b)[0]
    assert np.allclose(phi0, np.cos(b.astype(np.float64)), rtol=0, atol=0)
    assert phi0[2] == 1.0
    # evenness for b = 0 and 2*pi/w periodicity
    dt = np.array([0.3, 2.0, 7.5])
    wz = np.array([1.0, 2.0], F32)
    bz = np.zeros(2, F32)
    assert np.allclose(tgn.time_encode(p64, dt, wz, bz), tgn.time_encode(p64, -dt, wz, bz), atol=1e-15)
    per = 2 * math.pi / wz.astype(np.float64)
    shifted = np.stack([tgn.time_encode(p64, dt + per[j], wz[j:j + 1], bz[j:j + 1])[:, 0] for j in range(2)], 1)
    assert np.allclose(shifted, tgn.time_encode(p64, dt, wz, bz), atol=1e-12)
    # a known value: w dt + b = pi -> -1
    assert abs(tgn.time_encode(p64, np.array([math.pi]), np.array([1.0]), np.array([0.0]))[0, 0] + 1) < 1e-15


def test_time_argument_rounding_is_two_fp32_roundings():
    """The float32 cosine argument is round(round(w*dt) + b): two separate roundings, no fused multiply-add."""
    rng = np.random.default_rng(3)
    p32 = tgn.Prec("f32")
    dts = np.concatenate([rng.random(200) * 1e5, rng.random(50) * 2.4e6, [0.0, 1e-3, 99999.99]]).astype(F32)
    w = np.array([1.0, 0.7, 3.3e-5, 1e-9], F32)
    b = np.array([0.0, 0.3, -1.7, 2.5], F32)
    got = p32.time_arg(dts, w, b)
    for i, d in enumerate(dts):
        for j in range(w.size):
            prod = _to_f32(Fraction(float(w[j])) * Fraction(float(d)))
            ref = _to_f32(Fraction(prod) + Fraction(float(b[j])))
            assert got[i, j] == F32(ref), (d, w[j], b[j])
    # the fused form differs for some inputs: the rounding rule is observable
    fused = np.array([[_to_f32(Fraction(float(w[1])) * Fraction(float(d)) + Fraction(float(b[1])))
                       for d in dts]]).T
    two = p32.time_arg(dts, w[1:2], b[1:2])
    assert (fused.astype(F32) != two).any()
    # cosine of the rounded argument, in float64
    phi = tgn.time_encode(p32, dts[:5], w, b)
    for i in range(5):
        for j in range(w.size):
            assert phi[i, j] == math.cos(float(got[i, j]))


# --------------------------------------------------------------------------- selection (most recent message)

def _select_bruteforce(src, dst, t, eid, flags):
    best = {}
    for i in range(len(src)):
        if flags is not None and flags[i] & 2:
            continue
        for role, node in ((0, int(src[i])), (1, int(dst[i]))):
            key = (F32(t[i]), int(eid[i]), role)
            if node not in best or key > best[node][0]:
                best[node] = (key, 2 * i + role)
    nodes = sorted(best)
    return np.array(nodes, np.int64), np.array([best[n][1] for n in nodes], np.int64)


@pytest.mark.parametrize("seed", range(6))
def test_select_last_matches_bruteforce(seed):
    w = tiny_workload(n_nodes=7, n_events=60)
    s = tiny_stream(w, seed=seed, tie_every=3, flags_p=(0.3, 0.4) if seed % 2 else None)
    eid = np.arange(len(s.src)) + 1000
    u, win = tgn.select_last(s.src, s.dst, s.t, eid, s.flags)
    u2, win2 = _select_bruteforce(s.src, s.dst, s.t, eid, s.flags)
    assert np.array_equal(u, u2) and np.array_equal(win, win2)
    # invariants: each non-pruned endpoint once; the winner carries the node's latest time
    act = tgn.active_mask(s.flags, len(s.src))
    ends = set(s.src[act].tolist()) | set(s.dst[act].tolist())
    assert sorted(ends) == u.tolist()
    for n, wv in zip(u, win):
        i, role = wv // 2, wv % 2
        assert (s.src[i] if role == 0 else s.dst[i]) == n
        times = [s.t[j] for j in range(len(s.src)) if act[j] and n in (s.src[j], s.dst[j])]
        assert s.t[i] == max(times)


def test_select_last_self_loop_dst_role_wins():
    u, win = tgn.select_last([3], [3], np.array([1.0], F32), [0])
    assert u.tolist() == [3] and win.tolist() == [1]


# --------------------------------------------------------------------------- GRU

def test_gru_matches_hand_expansion_two_nodes():
    rng = np.random.default_rng(5)
    dm, D = 3, 7
    W_ih = rng.normal(size=(3 * dm, D))
    W_hh = rng.normal(size=(3 * dm, dm))
    b_ih, b_hh = rng.normal(size=3 * dm), rng.normal(size=3 * dm)
    x = rng.normal(size=(2, D))
    h = rng.normal(size=(2, dm))
    got, _ = tgn.gru_cell(x, h, W_ih, W_hh, b_ih, b_hh)
    for r in range(2):
        ref = sequential.gru_scalar(x[r], h[r], W_ih, W_hh, b_ih, b_hh)
        assert np.allclose(got[r], ref, rtol=0, atol=1e-14)


def test_gru_matches_torch_grucell_float64():
    rng = np.random.default_rng(6)
    dm, D, R = 5, 11, 9
    cell = torch.nn.GRUCell(D, dm).double()
    with torch.no_grad():
        for prm in cell.parameters():
            prm.copy_(torch.from_numpy(rng.normal(size=tuple(prm.shape))))
    x = rng.normal(size=(R, D))
    h = rng.normal(size=(R, dm))
    got, _ = tgn.gru_cell(x, h, cell.weight_ih.detach().numpy(), cell.weight_hh.detach().numpy(),
                          cell.bias_ih.detach().numpy(), cell.bias_hh.detach().numpy())
    ref = cell(torch.from_numpy(x), torch.from_numpy(h)).detach().numpy()
    assert np.allclose(got, ref, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------- memory phase semantics

def _run_batches(prec, w, s, mem, lu, params, B):
    for lo in range(0, len(s.src), B):
        hi = min(len(s.src), lo + B)
        mp = tgn.memory_phase(prec, w, tgn.batch_dict(s, lo, hi), mem, lu, s.x, params)
        mem, lu = mp.mem, mp.lu
    return mem, lu


def test_batch_of_one_equals_sequential_events():
    """Batch size 1 reproduces the per-event reading of Eq. 1-2 over 2,000 events of the tiny workload."""
    w = replace(workload(1), n_events=2000)
    s = tiny_stream(w, seed=11, t_scale=1e3, tie_every=7)
    params = init_params(w, random_bias=True)
    mem0, lu0 = random_state(w, seed=2)
    p64 = tgn.Prec("f64")
    mem_b, lu_b = _run_batches(p64, w, s, mem0.astype(np.float64), lu0.astype(np.float64), params, 1)
    mem_s, lu_s = sequential.replay_events(s.src, s.dst, s.t, s.x, None, mem0, lu0, params)
    assert np.array_equal(lu_b, lu_s)
    assert np.max(np.abs(mem_b - mem_s)) < 1e-12


def test_disjoint_batch_equals_sequential_events():
    """When no two events of a batch share a node, the batch step equals the event-by-event step."""
    w = tiny_workload(n_nodes=40, n_events=8, d_mem=6, d_time=5, d_edge=3)
    rng = np.random.default_rng(9)
    nodes = rng.permutation(40)[:16]
    s = tiny_stream(w, seed=1)
    s.src[:] = nodes[:8]
    s.dst[:] = nodes[8:]
    params = init_params(w, random_bias=True)
    mem0, lu0 = random_state(w, seed=4)
    p64 = tgn.Prec("f64")
    mem_b, lu_b = _run_batches(p64, w, s, mem0.astype(np.float64), lu0.astype(np.float64), params, 8)
    mem_s, lu_s = sequential.replay_events(s.src, s.dst, s.t, s.x, None, mem0, lu0, params)
    assert np.array_equal(lu_b, lu_s)
    assert np.max(np.abs(mem_b - mem_s)) < 1e-13


def test_batch_uses_pre_batch_snapshot_and_last_message():
    """Inside a batch every message reads the pre-batch state; a node keeps only its latest message."""
    w = tiny_workload(n_nodes=5, n_events=3, d_edge=0)
    s = tiny_stream(w, seed=2)
    s.src[:] = [0, 0, 2]
    s.dst[:] = [1, 2, 3]
    s.t[:] = np.array([1.0, 2.0, 3.0], F32)
    params = init_params(w, random_bias=True)
    mem0, lu0 = random_state(w, seed=6)
    p64 = tgn.Prec("f64")
    mp = tgn.memory_phase(p64, w, tgn.batch_dict(s, 0, 3), mem0.astype(np.float64), lu0.astype(np.float64),
                          None, params)
    # node 0: last message is event 1 (role 0) with partner 2, both read before the batch
    assert mp.uniq.tolist() == [0, 1, 2, 3]
    assert mp.winner.tolist() == [2, 1, 4, 5]
    one = sequential.replay_events(np.array([0]), np.array([2]), np.array([2.0]), None, None, mem0, lu0, params)
    assert np.max(np.abs(mp.mem[0] - one[0][0])) < 1e-13


def test_untouched_rows_bit_identical_and_last_update():
    w = workload(1)
    s = tiny_stream(replace(w, n_events=400), seed=3, t_scale=1e5)
    params = init_params(w)
    mem0, lu0 = random_state(w, seed=8)
    p32 = tgn.Prec("f32")
    mp = tgn.memory_phase(p32, w, tgn.batch_dict(s, 0, 200), mem0, lu0, s.x, params)
    touched = np.zeros(w.n_nodes, bool)
    touched[mp.uniq] = True
    assert mp.mem.dtype == np.float32
    assert np.array_equal(mp.mem[~touched].view(np.uint32), mem0[~touched].view(np.uint32))
    assert np.array_equal(mp.lu[~touched].view(np.uint32), lu0[~touched].view(np.uint32))
    # last_update of a touched node is its latest event time in the batch
    for n in mp.uniq[:50]:
        ev = [i for i in range(200) if n in (s.src[i], s.dst[i])]
        assert mp.lu[n] == s.t[max(ev)]


# --------------------------------------------------------------------------- sampling

@pytest.mark.parametrize("seed", range(5))
def test_sampling_matches_bruteforce(seed):
    w = tiny_workload(n_nodes=6, n_events=70)
    s = tiny_stream(w, seed=seed, tie_every=4)
    adj = tgn.build_adjacency(s.src, s.dst, s.t, w.n_nodes)
    rng = np.random.default_rng(seed)
    q_node = rng.integers(0, w.n_nodes, 40)
    q_t = np.concatenate([rng.random(30) * 11, s.t[rng.integers(0, 70, 10)]]).astype(F32)
    for k in (1, 3, 8, 40):
        got = tgn.sample_recent(adj, q_node, q_t, k)
        ref = tgn.sample_recent_bruteforce(s.src, s.dst, s.t, q_node, q_t, k)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b)
        nbr, nt, neid = got
        for qi in range(len(q_node)):
            valid = nbr[qi] >= 0
            m = int(valid.sum())
            assert valid[:m].all() and not valid[m:].any()          # padding only at the tail
            assert (nt[qi, :m] < q_t[qi]).all()                       # strictly earlier
            assert (np.diff(nt[qi, :m]) <= 0).all()                   # newest first
            n_elig = sum(int(s.t[e] < q_t[qi]) * (int(s.src[e] == q_node[qi]) + int(s.dst[e] == q_node[qi]))
                         for e in range(len(s.src)))
            assert m == min(k, n_elig)
            assert (neid[qi, m:] == -1).all() and (nt[qi, m:] == 0).all()


def test_adjacency_self_loop_twice_and_sorted():
    w = tiny_workload(n_nodes=3, n_events=4)
    s = tiny_stream(w, seed=0)
    s.src[:] = [0, 1, 2, 2]
    s.dst[:] = [1, 1, 0, 2]
    adj = tgn.build_adjacency(s.src, s.dst, s.t, 3)
    seg = slice(adj.off[1], adj.off[2])
    assert adj.nbr[seg].tolist() == [0, 1, 1] and adj.eid[seg].tolist() == [0, 1, 1]
    seg2 = slice(adj.off[2], adj.off[3])
    assert adj.eid[seg2].tolist() == [2, 3, 3]


# --------------------------------------------------------------------------- attention

def _attn_inputs(seed=0, H=2, k=4, Q=5, dm=6, dt=3, de=2, da=8, n_valid=None):
    w = tiny_workload(n_nodes=9, d_mem=dm, d_time=dt, d_edge=de, d_attn=da, n_heads=H, k=k, n_events=30)
    s = tiny_stream(w, seed=seed)
    params = init_params(w, random_bias=True)
    rng = np.random.default_rng(seed)
    mem = rng.uniform(-1, 1, (w.n_nodes, dm))
    q_node = rng.integers(0, w.n_nodes, Q)
    q_t = (rng.random(Q) * 10 + 10).astype(F32)
    nbr = rng.integers(0, w.n_nodes, (Q, k))
    nt = (rng.random((Q, k)) * 10).astype(F32)
    neid = rng.integers(0, 30, (Q, k))
    if n_valid is not None:
        for qi in range(Q):
            nbr[qi, n_valid[qi]:] = -1
            nt[qi, n_valid[qi]:] = 0
            neid[qi, n_valid[qi]:] = -1
    return w, s, params, mem, q_node, q_t, nbr, nt, neid


def test_attention_core_matches_torch_sdpa():
    w, s, params, mem, q_node, q_t, nbr, nt, neid = _attn_inputs(n_valid=[4, 1, 2, 3, 4])
    p64 = tgn.Prec("f64")
    sv = tgn.attention_fwd(p64, w, mem, s.x, params, q_node, q_t, nbr, nt, neid)
    Q, k, H, dh = 5, 4, w.n_heads, w.d_attn // w.n_heads
    q = torch.from_numpy(sv.q.reshape(Q, 1, H, dh).transpose(0, 2, 1, 3).copy())
    K = torch.from_numpy(sv.K.reshape(Q, k, H, dh).transpose(0, 2, 1, 3).copy())
    V = torch.from_numpy(sv.V.reshape(Q, k, H, dh).transpose(0, 2, 1, 3).copy())
    mask = torch.from_numpy(sv.valid[:, None, None, :])
    ref = torch.nn.functional.scaled_dot_product_attention(q, K, V, attn_mask=mask)
    ref = ref.transpose(1, 2).reshape(Q, -1).numpy()
    assert np.allclose(sv.attn, ref, rtol=0, atol=1e-13)


def test_attention_single_neighbour_and_empty():
    w, s, params, mem, q_node, q_t, nbr, nt, neid = _attn_inputs(n_valid=[1, 0, 1, 0, 1])
    sv = tgn.attention_fwd(tgn.Prec("f64"), w, mem, s.x, params, q_node, q_t, nbr, nt, neid)
    for qi in (0, 2, 4):   # one valid slot: softmax weight 1, output = V of that slot
        assert np.allclose(sv.attn[qi], sv.V[qi, 0], rtol=0, atol=1e-14)
    for qi in (1, 3):      # no valid slot: attention output 0, o = b_o
        assert np.all(sv.attn[qi] == 0)
        assert np.allclose(sv.o[qi], params["b_o"], rtol=0, atol=0)


def test_attention_permutation_invariant_over_slots():
    w, s, params, mem, q_node, q_t, nbr, nt, neid = _attn_inputs(n_valid=[4, 2, 3, 4, 1])
    p64 = tgn.Prec("f64")
    a = tgn.attention_fwd(p64, w, mem, s.x, params, q_node, q_t, nbr, nt, neid)
    perm = np.array([2, 0, 3, 1])
    b = tgn.attention_fwd(p64, w, mem, s.x, params, q_node, q_t, nbr[:, perm], nt[:, perm], neid[:, perm])
    assert np.allclose(a.z, b.z, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------- backward (finite differences)

def _fd_setup(seed=0):
    w = tiny_workload(n_nodes=6, n_events=24, batch=8, k=3, d_mem=4, d_time=3, d_edge=2, d_attn=4, n_heads=2)
    s = tiny_stream(w, seed=seed, t_scale=6.0, tie_every=5)
    params = {k: v.astype(np.float64) for k, v in init_params(w, random_bias=True).items()}
    rng = np.random.default_rng(seed + 10)
    params["time_w"] = rng.uniform(0.2, 1.5, w.d_time)
    mem0 = rng.uniform(-1, 1, (w.n_nodes, w.d_mem))
    lu0 = np.zeros(w.n_nodes)
    adj = tgn.build_adjacency(s.src, s.dst, s.t, w.n_nodes)
    prev = tgn.batch_dict(s, 8, 16)
    cur = tgn.batch_dict(s, 16, 24)
    noise = rng.standard_normal((24, w.d_attn))
    return w, s, params, mem0, lu0, adj, prev, cur, noise


def test_backward_matches_central_differences():
    w, s, params, mem0, lu0, adj, prev, cur, noise = _fd_setup()
    p64 = tgn.Prec("f64")
    res = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur, noise)
    assert len(res.mp.uniq) > 0 and np.abs(res.d_mem).max() > 0   # the GRU path is exercised

    def loss(pp):
        r = tgn.step(p64, w, mem0, lu0, pp, adj, s.x, prev, cur, noise)
        return float(np.sum(r.dz * r.attn.z))

    h = 1e-6
    for name, g in res.grads.items():
        base = params[name]
        fd = np.zeros(base.size)
        for i in range(base.size):
            pp = dict(params)
            for sgn in (1, -1):
                arr = base.copy().reshape(-1)
                arr[i] += sgn * h
                pp[name] = arr.reshape(base.shape)
                fd[i] += sgn * loss(pp)
        fd /= 2 * h
        scale = max(np.abs(fd).max(), 1e-3)      # FD noise is ~1e-10 here
        err = np.abs(fd - np.asarray(g).reshape(-1)).max() / scale
        assert err < 1e-6, (name, err)
    # adding the same vector to every key shifts all scores of a head equally: d b_k = 0
    assert np.abs(res.grads["b_k"]).max() < 1e-12


def test_memory_grad_counts_query_and_neighbour_occurrences():
    uniq = np.array([2, 5])
    q_node = np.array([5, 1, 2, 5])
    nbr = np.array([[2, -1], [5, 2], [0, 0], [-1, -1]])
    dhq = np.arange(8, dtype=float).reshape(4, 2)
    dhn = np.arange(16, dtype=float).reshape(4, 2, 2) * 10
    out = tgn.memory_grad(uniq, q_node, nbr, dhq, dhn)
    exp2 = dhq[2] + dhn[0, 0] + dhn[1, 1]
    exp5 = dhq[0] + dhq[3] + dhn[1, 0]
    assert np.array_equal(out, np.stack([exp2, exp5]))


# --------------------------------------------------------------------------- masks (Def. 2, Eq. 10-13)

def test_masks_replay_only_all_pruned_and_no_target():
    w, s, params, mem0, lu0, adj, prev, cur, noise = _fd_setup(seed=3)
    p64 = tgn.Prec("f64")
    # replay-only embedding batch: no query, no loss, memory phase unchanged
    cur_r = dict(cur, flags=np.ones(8, np.uint8))
    r = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur_r, noise)
    assert r.q_node.size == 0 and r.n_tar == 0
    assert all(np.all(np.asarray(g) == 0) for g in r.grads.values())
    # replay events still advance memory
    prev_r = dict(prev, flags=np.ones(8, np.uint8))
    r2 = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev_r, cur, noise)
    assert len(r2.mp.uniq) > 0 and not np.array_equal(r2.mp.mem, mem0)
    # all-pruned memory batch: state unchanged bit for bit
    prev_p = dict(prev, flags=np.full(8, 3, np.uint8))
    r3 = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev_p, cur, noise)
    assert len(r3.mp.uniq) == 0
    assert np.array_equal(r3.mp.mem, mem0) and np.array_equal(r3.mp.lu, lu0)
    # the masked loss normalises by the number of target events
    cur_m = dict(cur, flags=np.array([0, 1, 0, 1, 1, 0, 3, 0], np.uint8))
    r4 = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur_m, noise)
    assert r4.n_tar == 4 and r4.q_node.size == 12
    assert np.allclose(r4.dz, noise[:12] / 4)


# --------------------------------------------------------------------------- bf16

def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(10000).astype(F32) * 10.0 ** rng.integers(-30, 30, 10000),
        np.array([0.0, -0.0, np.inf, -np.inf, 1e-40, -3e-39, 3.4e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8], F32),
    ]).astype(F32)
    # exact ties: mantissa pattern ...8000 with even/odd kept bit
    ties = (np.arange(1000, dtype=np.uint32) << 16 | 0x8000).view(F32) + 0
    vals = np.concatenate([vals, ties.astype(F32), -ties.astype(F32)])
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float32).numpy()
    got = round_bf16(vals)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    assert np.isnan(round_bf16(np.array([np.nan], F32))[0])


def test_bf16_mode_close_to_f32_mode():
    w = replace(workload(5), n_nodes=300, n_events=3000, batch=500, k=5)
    s = tiny_stream(w, seed=4, t_scale=1e3, flags_p=(0.25, 0.1))
    params = init_params(w, random_bias=True)
    mem0, lu0 = random_state(w, seed=3)
    adj = tgn.build_adjacency(s.src, s.dst, s.t, w.n_nodes)
    prev, cur = tgn.batch_dict(s, 1000, 1500), tgn.batch_dict(s, 1500, 2000)
    noise = np.random.default_rng(1).standard_normal((1500, w.d_attn))
    r32 = tgn.step(tgn.Prec("f32"), w, mem0, lu0, params, adj, s.x, prev, cur, noise)
    r16 = tgn.step(tgn.Prec("bf16"), w, round_bf16(mem0), lu0, params, adj, s.x, prev, cur, noise)

    def rel(a, b):
        return np.abs(np.asarray(a, float) - b).max() / max(np.abs(b).max(), 1e-30)

    assert rel(r16.attn.z, r32.attn.z) < 2e-2
    assert rel(r16.mp.h_new, r32.mp.h_new) < 2e-2
    # gradients move more (ReLU masks flip near zero); d b_k is identically zero in both
    for name in r32.grads:
        if name != "b_k":
            assert rel(r16.grads[name], r32.grads[name]) < 0.1, name
    assert np.abs(r16.grads["b_k"]).max() < 1e-9 * np.abs(r16.grads["W_k"]).max()


# --------------------------------------------------------------------------- the paper's worked example

def test_example_dependency_chain():
    """Example 2 (Section III-C): the state of node 3 before e8 = (4, 3, t8) depends on e7, e6, e3 and e1."""
    with open(os.path.join(GOLDEN, "example2_dependency.json")) as f:
        ex = json.load(f)
    ev = ex["events"]
    src = np.array([e[0] for e in ev])
    dst = np.array([e[1] for e in ev])
    t = np.arange(1, len(ev) + 1, dtype=F32)
    w = tiny_workload(n_nodes=16, n_events=len(ev), d_edge=2)
    params = init_params(w, random_bias=True)
    rng = np.random.default_rng(0)
    x = rng.standard_normal((len(ev), 2)).astype(F32)
    mem0 = np.zeros((16, w.d_mem), F32)
    lu0 = np.zeros(16, F32)
    target = ex["target_event"] - 1
    node = ex["node"]

    def state_before_target(xx):
        m, _ = sequential.replay_events(src[:target], dst[:target], t[:target], xx[:target], None, mem0, lu0, params)
        return m[node]

    base = state_before_target(x)
    deps = []
    for e in range(target):
        xx = x.copy()
        xx[e] += 1.0
        if np.abs(state_before_target(xx) - base).max() > 0:
            deps.append(e + 1)
    assert set(ex["must_depend_on"]) <= set(deps)
    assert not set(ex["must_not_depend_on"]) & set(deps)


def test_restricted_adjacency_equals_full_lists():
    """The per-node lists built from the events touching a node subset equal the full build's lists."""
    rng = np.random.default_rng(21)
    E, N = 3000, 80
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    t = np.sort(rng.random(E) * 50).astype(np.float32)
    t[5::7] = t[4::7][: t[5::7].size]          # timestamp ties
    full = tgn.build_adjacency(src, dst, t, N)
    nodes = rng.choice(N, 17, replace=False)
    part = tgn.build_adjacency_for(src, dst, t, N, nodes)
    for n in range(N):
        lo, hi = part.off[n], part.off[n + 1]
        if n in nodes:
            flo, fhi = full.off[n], full.off[n + 1]
            assert np.array_equal(part.nbr[lo:hi], full.nbr[flo:fhi])
            assert np.array_equal(part.t[lo:hi], full.t[flo:fhi])
            assert np.array_equal(part.eid[lo:hi], full.eid[flo:fhi])
        else:
            assert hi == lo
    q = rng.choice(nodes, 40)
    qt = rng.random(40).astype(np.float32) * 50
    for a, b in zip(tgn.sample_recent(part, q, qt, 6), tgn.sample_recent(full, q, qt, 6)):
        assert np.array_equal(a, b)


# --------------------------------------------------------------------------- independent torch rendering

def _torch_step_forward(mode, w, mem, x_all, params, mem_batch, q_node, q_t, nbr, nt, neid):
    """The forward of one step written again in torch (float64 on the CPU), from the raw parameters:
    torch.nn.GRUCell for the memory update, torch.nn.functional.linear for every layer, masked
    scaled-dot-product attention per head, ReLU, and the concatenations of the embedding (query input
    [M || phi(0)], key/value input [M || x || phi(tau - t)], merge input [o || M]).  In "bf16" mode the
    values that enter a matrix product are cast to bfloat16 with torch (float64 -> float32 -> bfloat16)
    at exactly the points of the bf16 reading: messages, the query and key/value inputs, the attention
    output before W_o, o before the merge, relu(m1) before W_2, and the weights; the memory update is
    stored rounded; the time argument is formed as two float32 operations."""
    f64 = torch.float64
    T = lambda a: torch.as_tensor(np.asarray(a, np.float64))   # noqa: E731
    if mode == "bf16":
        rnd = lambda v: v.to(torch.float32).to(torch.bfloat16).to(f64)   # noqa: E731
    else:
        rnd = lambda v: v                                                 # noqa: E731
    tw, tb = params["time_w"], params["time_b"]

    def phi(dt):
        if mode == "bf16":
            arg = torch.as_tensor(np.asarray(dt, F32))[..., None] * torch.as_tensor(tw) + torch.as_tensor(tb)
            return torch.cos(arg.to(f64))
        return torch.cos(T(dt)[..., None] * T(tw) + T(tb))

    Wt = {n: rnd(T(params[n])) for n in ("W_ih", "W_hh", "W_q", "W_k", "W_v", "W_o", "W_1", "W_2")}
    bt = {n: T(params[n]) for n in ("b_ih", "b_hh", "b_q", "b_k", "b_v", "b_o", "b_1", "b_2")}
    out = {}
    # ---- memory phase: the last message of each node (selection taken from the pinned select_last)
    uniq, winner = tgn.select_last(mem_batch["src"], mem_batch["dst"], mem_batch["t"], mem_batch["eid"])
    ev, role = winner // 2, winner % 2
    node = np.where(role == 0, mem_batch["src"][ev], mem_batch["dst"][ev]).astype(np.int64)
    partner = np.where(role == 0, mem_batch["dst"][ev], mem_batch["src"][ev]).astype(np.int64)
    tt = np.asarray(mem_batch["t"], F32)[ev]
    lu0 = np.zeros(w.n_nodes, F32)
    dtm = (tt - lu0[node]).astype(F32) if mode == "bf16" else tt.astype(np.float64)
    M0 = T(mem)
    parts = [M0[node], M0[partner], rnd(phi(dtm))]
    if w.d_edge:
        parts.append(rnd(T(x_all[np.asarray(mem_batch["eid"])[ev]])))
    msg = torch.cat(parts, 1)
    cell = torch.nn.GRUCell(w.d_msg, w.d_mem, dtype=f64)
    with torch.no_grad():
        cell.weight_ih.copy_(Wt["W_ih"])
        cell.weight_hh.copy_(Wt["W_hh"])
        cell.bias_ih.copy_(bt["b_ih"])
        cell.bias_hh.copy_(bt["b_hh"])
        h_new = cell(msg, M0[uniq])
    M1 = M0.clone()
    M1[uniq] = rnd(h_new) if mode == "bf16" else h_new
    out.update(msg=msg, h_new=h_new, uniq=uniq)
    # ---- embedding from the updated table
    Q, k = nbr.shape
    H, da = w.n_heads, w.d_attn
    dh = da // H
    valid = torch.as_tensor(nbr >= 0)
    hq = M1[q_node]
    q_in = torch.cat([hq, rnd(phi(np.zeros(Q, F32)))], 1)
    q = torch.nn.functional.linear(q_in, Wt["W_q"], bt["b_q"])
    nb = np.where(nbr >= 0, nbr, 0)
    if mode == "bf16":
        dts = (np.asarray(q_t, F32)[:, None] - np.asarray(nt, F32)).astype(F32)
    else:
        dts = np.asarray(q_t, np.float64)[:, None] - np.asarray(nt, np.float64)
    kparts = [M1[nb]]
    if w.d_edge:
        kparts.append(rnd(T(x_all[np.where(nbr >= 0, neid, 0)])))
    kparts.append(rnd(phi(dts)))
    kv_in = torch.cat(kparts, 2)
    K = torch.nn.functional.linear(kv_in, Wt["W_k"], bt["b_k"])
    V = torch.nn.functional.linear(kv_in, Wt["W_v"], bt["b_v"])
    qh = q.reshape(Q, H, 1, dh)
    Kh = K.reshape(Q, k, H, dh).transpose(1, 2)
    Vh = V.reshape(Q, k, H, dh).transpose(1, 2)
    mask = valid[:, None, None, :].expand(Q, H, 1, k)
    a = torch.nn.functional.scaled_dot_product_attention(qh, Kh, Vh, attn_mask=mask)
    a = torch.where(valid.any(1)[:, None, None, None], a, torch.zeros_like(a))   # no neighbour: 0
    attn = rnd(a.reshape(Q, da))
    o = torch.nn.functional.linear(attn, Wt["W_o"], bt["b_o"])
    m_in = torch.cat([rnd(o), hq], 1)
    m1 = torch.nn.functional.linear(m_in, Wt["W_1"], bt["b_1"])
    a1 = rnd(torch.relu(m1))
    z = torch.nn.functional.linear(a1, Wt["W_2"], bt["b_2"])
    out.update(q_in=q_in, q=q, kv_in=kv_in, K=K, V=V, attn=attn, o=o, m_in=m_in, m1=m1, a1=a1, z=z,
               valid=valid.numpy())
    return {kk: (v.numpy() if torch.is_tensor(v) else v) for kk, v in out.items()}


def _composition_case(seed, H, de, n_valid, mode="f64"):
    w = tiny_workload(n_nodes=11, n_events=40, d_mem=7, d_time=5, d_edge=de, d_attn=12, n_heads=H, k=4,
                      batch=10)
    if mode == "bf16":
        w = replace(w, dtype="bf16")
    s = tiny_stream(w, seed=seed, t_scale=20.0, tie_every=4)
    params = init_params(w, random_bias=True)
    rng = np.random.default_rng(seed + 100)
    params["time_w"] = rng.uniform(0.05, 1.2, w.d_time).astype(F32)
    mem = rng.uniform(-1, 1, (w.n_nodes, w.d_mem))
    if mode == "bf16":
        mem = round_bf16(mem.astype(F32)).astype(np.float64)
    mb = tgn.batch_dict(s, 0, 10)
    Q = len(n_valid)
    q_node = rng.integers(0, w.n_nodes, Q)
    q_t = (rng.random(Q) * 10 + 20).astype(F32)
    nbr = rng.integers(0, w.n_nodes, (Q, w.k))
    nt = (rng.random((Q, w.k)) * 20).astype(F32)
    neid = rng.integers(0, s.n_events, (Q, w.k))
    for qi, nv in enumerate(n_valid):
        nbr[qi, nv:], nt[qi, nv:], neid[qi, nv:] = -1, 0, -1
    return w, s, params, mem, mb, q_node, q_t, nbr, nt, neid


@pytest.mark.parametrize("H", [1, 2, 3])
@pytest.mark.parametrize("de", [0, 3])
def test_attention_forward_composition_matches_torch_module(H, de):
    """The whole embedding (projection inputs, W_q/W_k/W_v, per-head softmax, W_o, the merge
    W_2 relu(W_1 [o || M] + b_1) + b_2) against an independent float64 torch rendering, with queries
    that have no, one, some and all valid neighbour slots."""
    n_valid = [0, 1, 2, 4, 4, 3]
    w, s, params, mem, mb, q_node, q_t, nbr, nt, neid = _composition_case(7 + H + de, H, de, n_valid)
    p64 = tgn.Prec("f64")
    mp = tgn.memory_phase(p64, w, mb, mem, np.zeros(w.n_nodes), s.x, params)
    sv = tgn.attention_fwd(p64, w, mp.mem, s.x, params, q_node, q_t, nbr, nt, neid)
    ref = _torch_step_forward("f64", w, mem, s.x, params, mb, q_node, q_t, nbr, nt, neid)
    v = ref["valid"]
    pairs = [("msg", mp.msg, ref["msg"]), ("h_new", mp.h_new, ref["h_new"]), ("q_in", sv.q_in, ref["q_in"]),
             ("q", sv.q, ref["q"]), ("kv_in", sv.kv_in[v], ref["kv_in"][v]), ("K", sv.K[v], ref["K"][v]),
             ("V", sv.V[v], ref["V"][v]), ("attn", sv.attn, ref["attn"]), ("o", sv.o, ref["o"]),
             ("m_in", sv.m_in, ref["m_in"]), ("m1", sv.m1, ref["m1"]), ("a1", sv.a1, ref["a1"]),
             ("z", sv.z, ref["z"])]
    for name, a, b in pairs:
        assert a.shape == b.shape, name
        assert np.allclose(a, b, rtol=0, atol=1e-12), (name, np.abs(a - b).max())
    assert np.all(sv.attn[0] == 0) and np.allclose(sv.o[0], params["b_o"], rtol=0, atol=0)


def _bf16_exact(a):
    a = np.asarray(a, np.float64)
    return np.array_equal(round_bf16(a.astype(F32)).astype(np.float64), a)


def test_bf16_rounding_placement():
    """bf16 mode rounds exactly the values the bf16 reading names, and nothing else.

    An independent torch rendering applies torch's bfloat16 cast at those points only; every
    intermediate of the oracle must then agree with it to float64 rounding (a missed or extra rounding
    moves values by ~4e-3).  The rounded tensors are bf16-representable; the unrounded ones are not."""
    n_valid = [0, 1, 3, 4, 4, 2, 4, 1]
    w, s, params, mem, mb, q_node, q_t, nbr, nt, neid = _composition_case(31, 2, 3, n_valid, mode="bf16")
    p16 = tgn.Prec("bf16")
    lu0 = np.zeros(w.n_nodes, F32)
    mp = tgn.memory_phase(p16, w, mb, mem.astype(F32), lu0, s.x, params)
    sv = tgn.attention_fwd(p16, w, mp.mem, s.x, params, q_node, q_t, nbr, nt, neid)
    ref = _torch_step_forward("bf16", w, mem, s.x, params, mb, q_node, q_t, nbr, nt, neid)
    v = ref["valid"]
    rounded = [("msg", mp.msg, ref["msg"]), ("q_in", sv.q_in, ref["q_in"]), ("kv_in", sv.kv_in[v], ref["kv_in"][v]),
               ("attn", sv.attn, ref["attn"]), ("m_in", sv.m_in, ref["m_in"]), ("a1", sv.a1, ref["a1"]),
               ("stored memory rows", mp.mem[mp.uniq], round_bf16(ref["h_new"].astype(F32)))]
    unrounded = [("h_new", mp.h_new, ref["h_new"]), ("q", sv.q, ref["q"]), ("K", sv.K[v], ref["K"][v]),
                 ("V", sv.V[v], ref["V"][v]), ("o", sv.o, ref["o"]), ("m1", sv.m1, ref["m1"]), ("z", sv.z, ref["z"])]
    for name, a, b in rounded:
        assert _bf16_exact(a), name
        # equal bit for bit, except where the value before the cast sits within float64 noise of a tie
        diff = np.asarray(a, np.float64) != np.asarray(b, np.float64)
        assert diff.mean() < 1e-3, (name, int(diff.sum()))
    for name, a, b in unrounded:
        assert not _bf16_exact(a), name
        scale = max(np.abs(b).max(), 1.0)
        assert np.allclose(a, b, rtol=0, atol=1e-12 * scale), (name, np.abs(a - b).max())
    # weights enter the products rounded: a product with unrounded W_2 differs from z by ~1e-3
    z_unrounded_w = sv.a1 @ np.asarray(params["W_2"], np.float64).T + params["b_2"]
    assert np.abs(z_unrounded_w - sv.z).max() > 1e-5


# --------------------------------------------------------------------------- link prediction loss (Eq. 12-13)

def _link_case(seed=0, n=7, da=6):
    w = tiny_workload(d_attn=da, n_heads=2)
    p = init_params(w, random_bias=True)
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((3 * n, da))
    return p, z


def test_link_loss_matches_torch_bce_with_logits():
    """The masked loss and every gradient against torch's binary cross-entropy with logits and autograd
    (float64 on the CPU), with the predictor written from its parameters: W_d2 relu(W_d1 [z_a || z_b] + b_d1) + b_d2."""
    p, z = _link_case()
    n = z.shape[0] // 3
    ref = tgn.link_loss(p, z, n)
    tz = torch.tensor(z, requires_grad=True)
    tp = {k: torch.tensor(np.asarray(p[k], np.float64), requires_grad=True) for k in ("W_d1", "b_d1", "W_d2", "b_d2")}

    def score(a, b):
        h = torch.relu(torch.nn.functional.linear(torch.cat([a, b], 1), tp["W_d1"], tp["b_d1"]))
        return torch.nn.functional.linear(h, tp["W_d2"], tp["b_d2"])[:, 0]

    pos, neg = score(tz[:n], tz[n:2 * n]), score(tz[:n], tz[2 * n:])
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    L = bce(pos, torch.ones(n, dtype=torch.float64)) + bce(neg, torch.zeros(n, dtype=torch.float64))
    L.backward()
    assert abs(ref.loss - L.item()) < 1e-13
    assert np.allclose(ref.s_pos, pos.detach().numpy(), rtol=0, atol=1e-13)
    assert np.allclose(ref.s_neg, neg.detach().numpy(), rtol=0, atol=1e-13)
    assert np.allclose(ref.dz, tz.grad.numpy(), rtol=0, atol=1e-14)
    for k in tp:
        assert np.allclose(ref.grads[k], tp[k].grad.numpy(), rtol=0, atol=1e-14), k


def test_link_loss_per_event_sum_and_special_cases():
    """Eq. 13 written event by event in plain Python: the mean over target events of
    -log sigmoid(s_pos) - log(1 - sigmoid(s_neg)); a zero output layer gives 2 log 2; no target, 0."""
    p, z = _link_case(seed=3, n=5)
    n = 5
    ref = tgn.link_loss(p, z, n)
    W1, b1, W2, b2 = (np.asarray(p[k], np.float64) for k in ("W_d1", "b_d1", "W_d2", "b_d2"))

    def s(a, b):
        x = list(a) + list(b)
        h = [max(0.0, sum(W1[j][c] * x[c] for c in range(len(x))) + b1[j]) for j in range(len(b1))]
        return sum(W2[0][j] * h[j] for j in range(len(h))) + b2[0]

    tot = 0.0
    for i in range(n):
        sp, sn = s(z[i], z[n + i]), s(z[i], z[2 * n + i])
        tot += -math.log(1.0 / (1.0 + math.exp(-sp))) - math.log(1.0 - 1.0 / (1.0 + math.exp(-sn)))
    assert abs(ref.loss - tot / n) < 1e-12
    p0 = dict(p, W_d2=np.zeros_like(p["W_d2"]), b_d2=np.zeros_like(p["b_d2"]))
    assert abs(tgn.link_loss(p0, z, n).loss - 2 * math.log(2.0)) < 1e-15
    empty = tgn.link_loss(p, z[:0], 0)
    assert empty.loss == 0.0 and empty.dz.shape == (0, z.shape[1])
    assert all(np.all(g == 0) for g in empty.grads.values())


def test_link_loss_masks_replay_and_pruned_events():
    """Only target events enter the loss (Eq. 12-13): replayed and pruned events get no query, so the
    step's loss equals the mean of the per-event losses of the target events alone."""
    w, s, params, mem0, lu0, adj, prev, cur, noise = _fd_setup(seed=5)
    params.update({k: np.asarray(v, np.float64) for k, v in init_params(w, random_bias=True).items()
                   if k.endswith(("d1", "d2"))})
    p64 = tgn.Prec("f64")
    flags = np.array([0, 1, 0, 3, 1, 0, 0, 1], np.uint8)
    r = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, dict(cur, flags=flags), None, loss="link")
    tar = np.nonzero(flags == 0)[0]
    assert r.n_tar == tar.size and r.q_node.size == 3 * tar.size
    full = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur, None, loss="link")
    # the same events' embeddings (each query sees the same neighbours whatever the mask)
    nf = full.n_tar
    zt = np.concatenate([full.attn.z[tar], full.attn.z[nf + tar], full.attn.z[2 * nf + tar]])
    assert np.allclose(zt, r.attn.z, rtol=0, atol=1e-14)
    per = tgn._softplus(-full.link.s_pos) + tgn._softplus(full.link.s_neg)
    assert abs(r.link.loss - per[tar].mean()) < 1e-14
    none = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, dict(cur, flags=np.ones(8, np.uint8)), None,
                    loss="link")
    assert none.link.loss == 0.0 and all(np.all(np.asarray(g) == 0) for g in none.grads.values())


def test_link_step_backward_matches_central_differences():
    """The whole step under the link loss (decoder, attention, GRU, time encoder): every parameter's
    gradient against central differences of the loss in float64."""
    w, s, params, mem0, lu0, adj, prev, cur, noise = _fd_setup(seed=2)
    params.update({k: np.asarray(v, np.float64) for k, v in init_params(w, random_bias=True).items()
                   if k.endswith(("d1", "d2"))})
    p64 = tgn.Prec("f64")
    res = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur, None, loss="link")
    assert {"W_d1", "b_d1", "W_d2", "b_d2", "W_ih", "W_k", "time_w"} <= set(res.grads)

    def loss(pp):
        return tgn.step(p64, w, mem0, lu0, pp, adj, s.x, prev, cur, None, loss="link").link.loss

    h = 1e-6
    for name, g in res.grads.items():
        base = params[name]
        fd = np.zeros(base.size)
        for i in range(base.size):
            pp = dict(params)
            for sgn in (1, -1):
                arr = base.copy().reshape(-1)
                arr[i] += sgn * h
                pp[name] = arr.reshape(base.shape)
                fd[i] += sgn * loss(pp)
        fd /= 2 * h
        scale = max(np.abs(fd).max(), 1e-4)
        err = np.abs(fd - np.asarray(g).reshape(-1)).max() / scale
        assert err < 1e-6, (name, err)


def test_relu_flips_only_change_the_chosen_decisions():
    """Inverting no ReLU decision changes nothing; inverting one whose pre-activation is zero changes
    no forward value and makes the backward take the other one-sided derivative."""
    w, s, params, mem0, lu0, adj, prev, cur, noise = _fd_setup(seed=4)
    p64 = tgn.Prec("f64")
    r0 = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur, None, loss="link")
    none = {"m1": np.zeros_like(r0.attn.m1, bool), "pos": np.zeros_like(r0.link.pre_pos, bool),
            "neg": np.zeros_like(r0.link.pre_neg, bool)}
    r1 = tgn.step(p64, w, mem0, lu0, params, adj, s.x, prev, cur, None, loss="link", flips=none)
    for k in r0.grads:
        assert np.array_equal(r0.grads[k], r1.grads[k]), k
    # shift b_d1 so that one decoder unit of event 0's true edge sits exactly at zero
    j = int(np.argmax(np.abs(r0.link.pre_pos[0])))
    pz = dict(params, b_d1=params["b_d1"].copy())
    pz["b_d1"][j] -= r0.link.pre_pos[0, j]
    a = tgn.step(p64, w, mem0, lu0, pz, adj, s.x, prev, cur, None, loss="link")
    assert a.link.pre_pos[0, j] == 0.0
    fl = dict(none, pos=none["pos"].copy())
    fl["pos"][0, j] = True
    bb = tgn.step(p64, w, mem0, lu0, pz, adj, s.x, prev, cur, None, loss="link", flips=fl)
    assert a.link.loss == bb.link.loss
    assert not np.array_equal(a.grads["W_d1"], bb.grads["W_d1"])


# --------------------------------------------------------------------------- Algorithm 1 (dependency scan)

def test_dependency_scan_example_chain():
    """The paper's worked dependency (Example 2, Section III-C) through Algorithm 1: worker p owns
    node 4, the source of e8 = (4, 3); node 3 and every other node are remote.  With the events in two
    batches (e1..e4, e5..e8) the auxiliary replay events are exactly the events node 3's state depends
    on (e7, e6, e3, e1), and the refresh set holds node 3 and their remote endpoints."""
    from oracle import depscan
    with open(os.path.join(GOLDEN, "example2_dependency.json")) as f:
        ex = json.load(f)
    ev = ex["events"]
    src = np.array([e[0] for e in ev])
    dst = np.array([e[1] for e in ev])
    owner = np.ones(16, np.int64)
    owner[4] = 0
    tar, aux, F = depscan.backward_scan(src, dst, owner, 0, [[0, 1, 2, 3], [4, 5, 6, 7]])
    assert sorted(e + 1 for s in tar for e in s) == [ex["target_event"]]
    assert sorted(e + 1 for s in aux for e in s) == sorted(ex["must_depend_on"])
    assert F == {3, 11, 10, 2, 1}


def _scan_fixed_point(src, dst, owner, p, batches):
    """Algorithm 1's result as the least fixed point of its membership rule, by repeated sweeps over
    all events: an event whose source is remote is auxiliary iff an endpoint is in the frontier before
    it, i.e. among the remote destinations of the targets of its batch or of later batches, or the
    remote endpoints of the auxiliary events visited before it (later batches, or later in its batch)."""
    order = [(s, e) for s in reversed(range(len(batches))) for e in reversed(batches[s])]
    pos = {e: i for i, (_, e) in enumerate(order)}
    batch_of = {e: s for s, b in enumerate(batches) for e in b}
    aux = set()
    changed = True
    while changed:
        changed = False
        for s, e in order:
            if owner[src[e]] == p or e in aux:
                continue
            front = {int(dst[x]) for b in batches[s:] for x in b if owner[src[x]] == p and owner[dst[x]] != p}
            for a in aux:
                if pos[a] < pos[e]:
                    front |= {int(i) for i in (src[a], dst[a]) if owner[i] != p}
            if int(src[e]) in front or int(dst[e]) in front:
                aux.add(e)
                changed = True
    return aux, batch_of


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dependency_scan_equals_fixed_point_of_its_rule(seed):
    from oracle import depscan
    rng = np.random.default_rng(seed)
    N, E, P = 14, 60, 3
    src = rng.integers(0, N, E)
    dst = rng.integers(0, N, E)
    owner = rng.integers(0, P, N)
    batches = [list(range(b, min(E, b + 12))) for b in range(0, E, 12)]
    for p in range(P):
        tar, aux, F = depscan.backward_scan(src, dst, owner, p, batches)
        fp, _ = _scan_fixed_point(src, dst, owner, p, batches)
        assert {e for s in aux for e in s} == fp
        assert all(owner[src[e]] == p for s in tar for e in s)
        # the refresh set: remote nodes only, and every remote endpoint of an auxiliary event
        assert all(owner[x] != p for x in F)
        assert all(x in F for s in aux for e in s for x in (src[e], dst[e]) if owner[x] != p)


def test_mixed_batches_sorted_and_masked():
    from oracle import depscan
    rng = np.random.default_rng(7)
    N, E = 20, 200
    src, dst = rng.integers(0, N, E), rng.integers(0, N, E)
    t = np.sort(rng.random(E) * 10).astype(np.float32)
    owner = rng.integers(0, 4, N)
    role, sync = depscan.scan_stream(src, dst, t, owner, 4, 25, 3)
    # every event is a target of exactly the worker owning its source
    assert np.array_equal((role == 1).argmax(0), owner[src]) and np.all((role == 1).sum(0) == 1)
    for p in range(4):
        ids = np.nonzero(role[p])[0]
        mixed, is_aux = depscan.mixed_batch(t, list(ids[role[p, ids] == 1]), list(ids[role[p, ids] == 2]))
        assert mixed == sorted(ids.tolist())          # the stream order is already sort_t
        assert is_aux == (role[p, mixed] == 2).tolist()


# --------------------------------------------------------------------------- runtime controller (Section V, Alg. 2)

def test_controller_equations_by_hand():
    from oracle import controller as C
    # Eq. 6 / 8: the first value initialises the average
    assert C.ema(0.0, 3.0, 0.2) == 3.0
    assert abs(C.ema(3.0, 1.0, 0.25) - (0.25 * 1.0 + 0.75 * 3.0)) < 1e-15
    # Eq. 7: skip only when r > 0, the EMA is positive and the last norm is below tau_g times it
    assert C.sync_decision(0, 0.1, 1.0, 0.9) == 1
    assert C.sync_decision(5, 0.1, 0.0, 0.9) == 1
    assert C.sync_decision(5, 0.8, 1.0, 0.9) == 0
    assert C.sync_decision(5, 0.9, 1.0, 0.9) == 1      # not strictly below
    # Eq. 9: heavy when the last time exceeds tau_c times the EMA
    assert C.heavy_load(0, 9.0, 1.0, 1.5) == 0
    assert C.heavy_load(3, 1.6, 1.0, 1.5) == 1
    assert C.heavy_load(3, 1.5, 1.0, 1.5) == 0
    assert C.heavy_load(3, 1.6, 0.0, 1.5) == 0
    # a worked sequence: norms 2, 1, 4; alpha 0.5 -> EMAs 2, 1.5, 2.75
    c = C.Controller(alpha=0.5, beta=0.5, tau_g=0.9, tau_c=1.2, interval=2)
    seq = []
    for r, (g, t) in enumerate([(2.0, 10.0), (1.0, 10.0), (4.0, 20.0), (1.0, 10.0)]):
        seq.append((c.boundary(r), c.sync(r), c.heavy(r)))
        c.observe(g, t)
    assert seq == [(True, 1, 0), (False, 1, 0), (True, 0, 0), (False, 1, 1)]
    assert c.g_bar == 0.5 * 1.0 + 0.5 * 2.75 and c.c_bar == 0.5 * 10 + 0.5 * 15


def test_prune_aux_keeps_targets_and_refresh_copies_rows():
    from oracle import controller as C
    f = np.array([0, 1, 0, 3, 1, 2], np.uint8)
    assert C.prune_aux(f, 1).tolist() == [0, 3, 0, 3, 3, 0]
    assert C.prune_aux(f, 0).tolist() == [0, 1, 0, 1, 1, 0]
    cm, cl = np.zeros((5, 2)), np.zeros(5)
    am, al = np.arange(10.0).reshape(5, 2), np.arange(5.0) + 0.5
    m, l = C.cache_refresh(cm, cl, am, al, {1, 4})
    assert m.tolist() == [[0, 0], [2, 3], [0, 0], [0, 0], [8, 9]] and l.tolist() == [0, 1.5, 0, 0, 4.5]


def test_adam_matches_torch_adam():
    from oracle import controller as C
    rng = np.random.default_rng(0)
    th = rng.standard_normal(7)
    p = torch.tensor(th.copy(), requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    m = v = np.zeros(7)
    for t in range(1, 5):
        g = rng.standard_normal(7)
        p.grad = torch.tensor(g)
        opt.step()
        th, m, v = C.adam(th, g, m, v, t, 1e-2, 0.9, 0.999, 1e-8)
        assert np.allclose(th, p.detach().numpy(), rtol=0, atol=1e-14)
    assert abs(C.grad_norm([np.array([3.0]), np.array([[4.0, 12.0]])]) - 13.0) < 1e-15


# --------------------------------------------------------------------------- JODIE variant (Section VII-A)

def _jodie_case(seed=0):
    from synth import init_params_jodie
    w = tiny_workload(n_nodes=7, n_events=24, batch=8, k=1, d_mem=5, d_time=3, d_edge=2, d_attn=5, n_heads=1)
    s = tiny_stream(w, seed=seed, t_scale=6.0, tie_every=5)
    params = {k: v.astype(np.float64) for k, v in init_params_jodie(w, random_bias=True).items()}
    rng = np.random.default_rng(seed + 20)
    params["time_w"] = rng.uniform(0.2, 1.5, w.d_time)
    mem0 = rng.uniform(-1, 1, (w.n_nodes, w.d_mem))
    lu0 = np.zeros(w.n_nodes)
    return w, s, params, mem0, lu0, tgn.batch_dict(s, 8, 16), tgn.batch_dict(s, 16, 24)


def test_jodie_rnn_matches_torch_rnncell():
    from oracle import jodie
    rng = np.random.default_rng(1)
    x, h = rng.standard_normal((4, 9)), rng.standard_normal((4, 5))
    cell = torch.nn.RNNCell(9, 5, nonlinearity="tanh", dtype=torch.float64)
    got = jodie.rnn_cell(x, h, cell.weight_ih.detach().numpy(), cell.weight_hh.detach().numpy(),
                         cell.bias_ih.detach().numpy(), cell.bias_hh.detach().numpy())
    ref = cell(torch.from_numpy(x), torch.from_numpy(h)).detach().numpy()
    assert np.allclose(got, ref, rtol=0, atol=1e-14)


def test_jodie_step_matches_torch_autograd():
    """The whole JODIE step (RNN memory update, time projection, link loss) written again with torch
    float64 modules from the raw parameters; the loss, z, the updated rows and every gradient agree."""
    from oracle import jodie
    w, s, params, mem0, lu0, prev, cur = _jodie_case(3)
    scale = 0.37
    r = jodie.step(tgn.Prec("f64"), w, mem0, lu0, params, s.x, prev, cur, scale)
    T = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in params.items()}
    uniq, winner = r.mp.uniq, r.mp.winner
    ev, role = winner // 2, winner % 2
    node = np.where(role == 0, prev["src"][ev], prev["dst"][ev])
    partner = np.where(role == 0, prev["dst"][ev], prev["src"][ev])
    M0 = torch.from_numpy(mem0)
    dt = torch.from_numpy(np.asarray(prev["t"], np.float64)[ev] - lu0[node])
    phi = torch.cos(dt[:, None] * T["time_w"] + T["time_b"])
    msg = torch.cat([M0[node], M0[partner], phi, torch.from_numpy(s.x[prev["eid"][ev]].astype(np.float64))], 1)
    cell = torch.nn.RNNCell(w.d_msg, w.d_mem, dtype=torch.float64)
    h = torch.tanh(torch.nn.functional.linear(msg, T["W_ih"], T["b_ih"])
                   + torch.nn.functional.linear(M0[uniq], T["W_hh"], T["b_hh"]))
    del cell
    M1 = M0.clone()
    M1[uniq] = h
    lu1 = lu0.copy()
    lu1[uniq] = np.asarray(prev["t"], np.float64)[ev]
    q_node, q_t, n = tgn.queries(cur)
    delta = torch.from_numpy((np.asarray(q_t, np.float64) - lu1[q_node]) * scale)
    z = M1[q_node] * (1 + delta[:, None] * T["W_p"][:, 0] + T["b_p"])

    def score(a, b):
        hh = torch.relu(torch.nn.functional.linear(torch.cat([a, b], 1), T["W_d1"], T["b_d1"]))
        return torch.nn.functional.linear(hh, T["W_d2"], T["b_d2"])[:, 0]

    bce = torch.nn.functional.binary_cross_entropy_with_logits
    L = bce(score(z[:n], z[n:2 * n]), torch.ones(n, dtype=torch.float64)) + \
        bce(score(z[:n], z[2 * n:]), torch.zeros(n, dtype=torch.float64))
    L.backward()
    assert abs(r.link.loss - L.item()) < 1e-13
    assert np.allclose(r.z, z.detach().numpy(), rtol=0, atol=1e-13)
    assert np.allclose(r.mp.h_new, h.detach().numpy(), rtol=0, atol=1e-14)
    for k, g in r.grads.items():
        ref = T[k].grad.numpy()
        assert np.allclose(g, ref, rtol=0, atol=1e-13), (k, np.abs(g - ref).max())


def test_jodie_projection_special_cases():
    from oracle import jodie
    rng = np.random.default_rng(2)
    M = rng.standard_normal((3, 4))
    Wp, bp = rng.standard_normal((4, 1)), np.zeros(4)
    assert np.array_equal(jodie.project(M, np.zeros(3, np.float32), Wp, bp), M)       # no elapsed time: z = M
    d = jodie.projection_delta(tgn.Prec("f32"), np.array([5.0, 7.5], np.float32), np.array([1.0, 7.5], np.float32), 0.5)
    assert d.tolist() == [2.0, 0.0]
