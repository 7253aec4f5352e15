"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer outputs (updated rows, winners, queries, sampled neighbours, event
ids, copied times, last_update, untouched memory rows) must be bit-exact.
Floating-point tensors must satisfy max|gpu - oracle| / max|oracle| <= 1e-4
for float32 storage and <= 2e-2 for bfloat16 storage.  Each oracle step
starts from the GPU's state before that step (teacher forcing).
"""

from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import tgn
from synth import init_params, make_stream, window_state, workload
from tests._gpu import compare_step, compare_step_sampled, log, needs_gpu, to_np
from tests._tiny import random_state, tiny_stream, tiny_workload

pytestmark = [pytest.mark.gpu, needs_gpu]

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _runner(w, s, params, mem, lu, lag=1):
    from paper_2608_16305_amd.step import TGNStep
    return TGNStep(w, s, params, mem, lu, lag=lag)


def _check_csr(runner, s, n_nodes):
    adj = tgn.build_adjacency(s.src, s.dst, s.t, n_nodes)
    assert np.array_equal(runner.csr_off.cpu().numpy(), adj.off)
    ne = 2 * s.n_events
    assert np.array_equal(runner.csr_nbr.cpu().numpy()[:ne], adj.nbr)
    assert np.array_equal(runner.csr_eid.cpu().numpy()[:ne], adj.eid)
    assert np.array_equal(runner.csr_t.cpu().numpy()[:ne].view(np.uint32), adj.t.view(np.uint32))
    return adj


@pytest.mark.parametrize("cid", [1, 2])
def test_full_stream_steps(cid):
    """Workloads 1-2 from an empty memory (M = 0, last_update = 0), steps 0..4, lag-1 order."""
    w = workload(cid)
    log(f"[parity] workload {cid} {w.name}")
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    r = _runner(w, s, params, np.zeros((w.n_nodes, w.d_mem), np.float32), np.zeros(w.n_nodes, np.float32))
    adj = _check_csr(r, s, w.n_nodes)
    for b in range(5):
        compare_step(r, w, s, adj, b, TOL[w.dtype])


def test_workload1_lag0_order():
    w = workload(1)
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    mem, lu = random_state(w, seed=5)
    r = _runner(w, s, params, mem, np.zeros(w.n_nodes, np.float32), lag=0)
    adj = tgn.build_adjacency(s.src, s.dst, s.t, w.n_nodes)
    for b in (0, 1, 7):
        compare_step(r, w, s, adj, b, TOL[w.dtype], lag=0)


def test_workload3_window():
    """Skewed Zipf(1.2) stream, 1M nodes / 10M events, mid-stream window at batch 100 (hub lists of 1e5+ entries)."""
    w = workload(3)
    log("[parity] workload 3 window")
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    mem, lu = window_state(w, s, w.window_b0)
    r = _runner(w, s, params, mem, lu)
    adj = _check_csr(r, s, w.n_nodes)
    for b in range(w.window_b0, w.window_b0 + 3):
        compare_step(r, w, s, adj, b, TOL[w.dtype])


@pytest.mark.parametrize("cid", [4, 5])
def test_full_size_sampled(cid):
    """Workloads 4 (10M nodes, 100M events, batch 60,000, k 20, fp32) and 5 (replay / pruned
    masks, bf16) at full size, mid-stream: the adjacency (every offset, and the whole lists of every
    queried node), the whole memory phase, every query row's neighbours, and every gradient with the
    loss gradient on the queries of 256 sampled target events per step."""
    from tests._gpu import check_csr_full_size, query_nodes_of
    w = workload(cid)
    log(f"[parity] workload {cid} {w.name}: generating the stream")
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    mem, lu = window_state(w, s, w.window_b0)
    log("[parity] stream ready; uploading and building the adjacency on the GPU")
    r = _runner(w, s, params, mem, lu)
    del mem, lu
    torch.cuda.synchronize()
    steps = range(w.window_b0, w.window_b0 + 2)
    nodes = query_nodes_of(s, w, steps)
    log(f"[parity] oracle adjacency of the {nodes.size} queried nodes")
    adj = tgn.build_adjacency_for(s.src, s.dst, s.t, w.n_nodes, nodes)
    check_csr_full_size(r, s, w, adj, nodes)
    for b in steps:
        compare_step_sampled(r, w, s, b, TOL[w.dtype], n_sample=256, adj=adj, seed=b)


# ----------------------------------------------------------------------------- edge cases

def _tiny_run(w, s, mem, lu, steps, lag=1):
    params = init_params(w, random_bias=True)
    r = _runner(w, s, params, mem, lu, lag=lag)
    adj = _check_csr(r, s, w.n_nodes)
    out = []
    for b in steps:
        out.append(compare_step(r, w, s, adj, b, TOL[w.dtype], lag=lag))
    return r, out


def test_edge_ties_self_loops_k_beyond_degree():
    """Timestamp ties, self-loops, and k larger than most neighbour lists (padding)."""
    w = tiny_workload(n_nodes=9, n_events=90, batch=10, k=8, d_mem=6, d_time=5, d_edge=3, d_attn=8, n_heads=2)
    s = tiny_stream(w, seed=3, tie_every=3)
    assert (s.src == s.dst).any()
    mem, lu = random_state(w, seed=1)
    _tiny_run(w, s, mem, lu, range(0, 9))


def test_edge_masks_replay_pruned():
    """Replay events update memory but get no query; pruned events do nothing; zero-target batches."""
    w = tiny_workload(n_nodes=12, n_events=120, batch=12, k=4, d_mem=8, d_time=4, d_edge=0, d_attn=8, n_heads=2)
    s = tiny_stream(w, seed=4, flags_p=(0.4, 0.3))
    s.flags[24:36] = 3          # batch 2: every event pruned -> memory phase of step 3 changes nothing
    s.flags[48:60] = 1          # batch 4: replay only -> no query at step 4
    mem, lu = random_state(w, seed=2)
    r, out = _tiny_run(w, s, mem, lu, range(1, 10))
    gpu3, ref3 = out[2]          # step 3 runs the memory phase on batch 2
    assert gpu3["n_uniq"] == 0
    gpu4, ref4 = out[3]          # step 4 embeds batch 4
    assert gpu4["n_q"] == 0
    assert all(np.abs(g).max() == 0 for k, g in gpu4["grads"].items())


def test_edge_batch_of_one():
    w = tiny_workload(n_nodes=5, n_events=30, batch=1, k=3, d_mem=4, d_time=3, d_edge=2, d_attn=4, n_heads=1)
    s = tiny_stream(w, seed=6)
    mem, lu = random_state(w, seed=3)
    _tiny_run(w, s, mem, lu, range(0, 12))


def test_edge_ragged_tiles():
    """Sizes that are not multiples of any tile: 37 events per batch, d_mem 37, d_attn 30 with 3 heads."""
    w = tiny_workload(n_nodes=61, n_events=600, batch=37, k=7, d_mem=37, d_time=11, d_edge=5, d_attn=30, n_heads=3)
    s = tiny_stream(w, seed=8, t_scale=300.0, tie_every=5)
    mem, lu = random_state(w, seed=4)
    _tiny_run(w, s, mem, lu, range(0, 6))


def test_bf16_small():
    w = tiny_workload(n_nodes=50, n_events=800, batch=80, k=6, d_mem=16, d_time=8, d_edge=0, d_attn=16, n_heads=2)
    w = replace(w, dtype="bf16")
    s = tiny_stream(w, seed=9, t_scale=100.0, flags_p=(0.25, 0.1))
    mem, lu = random_state(w, seed=5)
    from oracle.bf16 import round_bf16
    _tiny_run(w, s, round_bf16(mem), lu, range(1, 6))


def test_edge_large_batch_multiblock_paths():
    """A batch of 22,000 events: aggregation takes the multi-block sort path (44,000 messages),
    the query-count scan the multi-level path (66,000 queries); replay/pruned masks included."""
    w = tiny_workload(n_nodes=30000, n_events=66000, batch=22000, k=3, d_mem=8, d_time=4, d_edge=2, d_attn=8,
                      n_heads=2)
    s = tiny_stream(w, seed=11, t_scale=1000.0, tie_every=7, flags_p=(0.2, 0.3))
    mem, lu = random_state(w, seed=6)
    _tiny_run(w, s, mem, lu, range(1, 3))


@pytest.mark.parametrize("case", ["bipartite", "large_batch"])
def test_backward_overlap_bitwise(case):
    """The two-stream attention backward (d_mem part on a second stream) gives bitwise the
    results of the single-stream call, from the same state (bipartite stream, 3 steps), both with
    the d_mem grouping at the backward's entry (mtgnn_temporal_attn_bwd_overlap) and with it done
    during the embedding (mtgnn_temporal_attn_bwd_group, then _grouped).  large_batch: 22,000 events
    per batch (66,000 query rows), where the output and merge layers' weight gradients also run on
    the second stream."""
    from paper_2608_16305_amd.step import TGNStep
    if case == "bipartite":
        w = workload(2)
    else:
        w = tiny_workload(n_nodes=30000, n_events=88000, batch=22000, k=3, d_mem=8, d_time=4, d_edge=2, d_attn=8,
                          n_heads=2)
    log(f"[parity] overlap vs single stream, {case}")
    s = make_stream(w) if case == "bipartite" else tiny_stream(w, seed=3)
    params = init_params(w, random_bias=True)
    mem, lu = random_state(w, seed=11)
    outs = []
    for overlap, ahead in ((False, False), (True, False), (True, True)):
        r = TGNStep(w, s, params, mem, lu, overlap=overlap)
        r.group_ahead = ahead
        res = {}
        for b in range(1, 4):
            r.step(b)   # with the masked link-prediction loss, as in training
            torch.cuda.synchronize()
            n = int(r.n_uniq.item())
            res[f"d_mem{b}"] = to_np(r.d_mem)[:n].copy()
            res.update({f"{k}{b}": to_np(v).copy() for k, v in r.grads.items()})
            res[f"loss{b}"] = to_np(r.loss).copy()
        res["memory"] = to_np(r.memory).copy()
        outs.append(res)
        del r
        torch.cuda.empty_cache()
    for o in outs[1:]:
        assert outs[0].keys() == o.keys()
        for k in outs[0]:
            a, b = outs[0][k], o[k]
            assert a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32)), k


def test_param_update_between_steps_bitwise():
    """Parameters updated in place on the caller's stream between steps (as an optimizer does): the
    two-stream step gives bitwise the results of the single-stream step, so nothing the second stream
    runs reads a parameter before the update.  The caller's stream sleeps before each update, so that
    the second stream, which goes on to the next step's queries meanwhile, would read the old values
    if it read any (bipartite stream, 3 steps)."""
    from paper_2608_16305_amd.step import TGNStep
    w = workload(2)
    log("[parity] parameter update between steps, overlap vs single stream")
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    mem, lu = random_state(w, seed=5)
    outs = []
    for overlap in (False, True):
        r = TGNStep(w, s, params, mem, lu, overlap=overlap)
        snaps = {}
        for b in range(1, 4):
            r.step(b)
            # copies on the caller's stream (ordered after the step's join); no host wait until the end,
            # so the next step is enqueued while this stream still sleeps
            snaps[f"loss{b}"] = r.loss.clone()
            snaps[f"z{b}"] = r.z.clone()
            snaps.update({f"{k}{b}": v.clone() for k, v in r.grads.items()})
            torch.cuda._sleep(20_000_000)   # the update below waits behind it
            for v in r.params.values():
                if v.dtype == torch.float32:
                    v.mul_(1.0 + 1.0 / 64)
            r.params_changed()
        torch.cuda.synchronize()
        res = {k: to_np(v).copy() for k, v in snaps.items()}
        res["memory"] = to_np(r.memory).copy()
        outs.append(res)
        del r
        torch.cuda.empty_cache()
    assert outs[0].keys() == outs[1].keys()
    for k in outs[0]:
        a, b = outs[0][k], outs[1][k]
        assert a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32)), k


def test_forward_single_call_matches_prepare_prepared():
    """mtgnn_temporal_attn in one call gives bitwise the z and the save buffer of
    mtgnn_temporal_attn_prepare followed by mtgnn_temporal_attn_prepared, and of the preparation's
    two halves (slots, then weights) followed by _prepared (bipartite stream)."""
    from paper_2608_16305_amd import mtgnn as M
    from paper_2608_16305_amd.step import TGNStep
    w = workload(2)
    log("[parity] single-call forward vs prepare + prepared, workload 2")
    s = make_stream(w)
    params = init_params(w, random_bias=True)
    mem, lu = random_state(w, seed=5)
    r = TGNStep(w, s, params, mem, lu, overlap=False)
    b = 2
    r.memory_phase(*r.batch_range(b - 1))
    r.queries(*r.batch_range(b), None)
    p = r.params
    outs = []
    for split in (0, 1, 2):
        save = torch.zeros_like(r.attn_save)
        z = torch.zeros_like(r.z)
        args = (r.q_node, r.q_t, r.n_q, r.max_q, r.nbr, r.nt, r.neid, r.memory, r.x, p["time_w"], p["time_b"],
                r.ap, r.d, z, save)
        if split == 1:
            M.mtgnn_temporal_attn_prepare(r.nbr, r.n_q, r.max_q, r.ap, p["time_w"], p["time_b"], r.d, save, r.ws)
            M.mtgnn_temporal_attn_prepared(*args)
        elif split == 2:   # the two halves of the preparation, slots first
            M.mtgnn_temporal_attn_prepare_slots(r.nbr, r.n_q, r.max_q, r.d, save, r.ws)
            M.mtgnn_temporal_attn_prepare_weights(r.ap, p["time_w"], p["time_b"], r.d, save)
            M.mtgnn_temporal_attn_prepared(*args)
        else:
            M.mtgnn_temporal_attn(*args, r.ws)
        torch.cuda.synchronize()
        outs.append((to_np(z).copy(), to_np(save).copy()))
    for o in outs[1:]:
        assert np.array_equal(outs[0][0].view(np.uint32), o[0].view(np.uint32))
        assert np.array_equal(outs[0][1], o[1])
