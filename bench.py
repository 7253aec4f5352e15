"""Benchmark of the memory-based TGNN batch step on one MI355X.

One step = the whole hot path over one batch: memory phase on the previous
batch (most-recent aggregation, message construction, GRU update with
write-back), embedding of the current batch's target events (queries,
most-recent-k sampling, temporal attention), the masked link-prediction loss
(decoder, binary cross-entropy of the true and negative edges, mean over the
target events), and the backward pass (decoder, attention, GRU, time encoder).
Inputs (event stream, temporal adjacency, memory table, parameters) are
resident in HBM before the timed region.

Default workload: the skewed stream (1M nodes, 10M events, Zipf(1.2) endpoints,
batch 4,000, k = 10, memory/time/attention width 100, 2 heads, float32),
mid-stream window starting at batch 100.

Prints one JSON line.  `python bench.py --gpus N --steps K --warmup W`.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_PEAK_TFLOPS = 157.3       # MI355X dense fp32 matrix
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0, help="timed steps (0: 50, or 30 for batches of 60,000)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--model", choices=("tgn", "jodie", "adaptive"), default="tgn",
                    help="tgn: the TGN step (default); jodie: the JODIE variant's step; adaptive: Algorithm 2's loop "
                         "for one worker of --workers over its mixed batches (dependency scan, controller, PruneAux, "
                         "refresh, Adam)")
    ap.add_argument("--workers", type=int, default=8, help="workers of the partition (--model adaptive)")
    ap.add_argument("--window", type=int, default=10, help="synchronization window in batches (--model adaptive)")
    ap.add_argument("--cpu-steps", type=int, default=3, help="oracle steps timed for the CPU baseline (0: skip)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="before the warmup, copy a buffer of this many MiB twice (HBM counter calibration)")
    ap.add_argument("--kernel-report", nargs=3, metavar=("TRACE_CSV", "FETCH_CSV", "WRITE_CSV"),
                    help="turn a rocprofv3 --kernel-trace CSV and two --pmc CSVs (FETCH_SIZE, WRITE_SIZE; runs made "
                         "with --copy-probe) into per-kernel HBM traffic and achieved GB/s under profiles/, then exit")
    ap.add_argument("--mfma-report", nargs=2, metavar=("TRACE_CSV", "SQ_CSV"),
                    help="turn a rocprofv3 --kernel-trace CSV and a --pmc CSV of SQ_VALU_MFMA_BUSY_CYCLES into each "
                         "matrix kernel's MFMA-busy fraction under profiles/, then exit")
    ap.add_argument("--step-report", nargs=2, metavar=("TRACE_DIR", "BENCH_JSON"),
                    help="turn a rocprofv3 --kernel-trace --stats output directory of this bench and the bench's "
                         "JSON line into the per-step kernel table under profiles/, then exit")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE) of a run made with "
                         "--copy-probe into the traffic record under profiles/, then exit")
    return ap.parse_args()


def main():
    args = parse()
    if args.steps <= 0:   # 50 (30 for batches of 60,000), within the stream after the window start
        from synth import workload as _wl
        wl = _wl(args.workload)
        args.steps = min(30 if wl.batch >= 60_000 else 50, (wl.n_batches - wl.window_b0 - args.warmup) // 2)
    if args.traffic_from:
        write_traffic(args)
        return
    if args.kernel_report:
        kernel_report(args)
        return
    if args.mfma_report:
        mfma_report(args)
        return
    if args.step_report:
        step_report(args)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the multi-GPU sharding is described, not built.", file=sys.stderr)
        sys.exit(2)
    if args.model != "tgn":
        other_model(args)
        return
    import torch

    from paper_2608_16305_amd.step import TGNStep
    from synth import init_params, make_stream, window_state, workload

    w = workload(args.workload)
    s = make_stream(w)
    params = init_params(w)
    b0 = w.window_b0
    mem, lu = window_state(w, s, b0)
    n_steps = args.warmup + 2 * args.steps   # the headline's K steps, then K more for the kernel timer
    if b0 + n_steps > w.n_batches:
        raise SystemExit(f"window [{b0}, {b0 + n_steps}) exceeds the {w.n_batches} batches of the stream")
    runner = TGNStep(w, s, params, mem, lu)

    # target events per step (Eq. 12), for the target-only throughput
    n_tar = []
    for i in range(n_steps):
        lo, hi = (b0 + i) * w.batch, min(w.n_events, (b0 + i + 1) * w.batch)
        n_tar.append((hi - lo) if s.flags is None else int(((s.flags[lo:hi] & 3) == 0).sum()))
    torch.cuda.synchronize()

    from paper_2608_16305_amd import mtgnn as M

    if args.copy_probe > 0:   # plain device copies of known size, just before the first step
        n = args.copy_probe * (1 << 20) // 4
        xa = torch.randn(n, device="cuda")
        ya = torch.empty_like(xa)
        torch.cuda.synchronize()
        for _ in range(2):
            ya.copy_(xa)
        torch.cuda.synchronize()
        del xa, ya

    # warmup; the matrix-product sites over the neighbour slots are timed one
    # warmup step each to pick the dominant one
    site_ms = {}
    for i in range(args.warmup):
        site = HOT_SITES[i % len(HOT_SITES)] if i >= 1 else None
        if site:
            M.timer_start(site, 16)
        runner.step(b0 + i)
        if site:
            ms, n = M.timer_stop()
            site_ms[site] = max(site_ms.get(site, 0.0), ms)
    torch.cuda.synchronize()
    dominant = max(site_ms, key=site_ms.get) if site_ms else HOT_SITES[0]

    def timed(first, count, site=None):
        """GPU milliseconds of `count` steps from step index `first` (HIP events on the main stream), and the
        host's enqueue and wall time; with `site`, the library's launch timer brackets that kernel's launches
        with HIP events on their own stream."""
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if site:
            M.timer_start(site, 16 * count)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record()
        for i in range(first, first + count):
            runner.step(b0 + i)
        enq = time.perf_counter() - t0
        ev1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        site_t = M.timer_stop() if site else None
        return ev0.elapsed_time(ev1), enq, wall, site_t

    # the headline: K steps with nothing but the step in the timed region
    gpu_ms, enq, wall, _ = timed(args.warmup, args.steps)
    # the dominant kernel's launch durations: the next K steps, with its launches bracketed
    gpu_ms2, _, _, (dom_ms, dom_launches) = timed(args.warmup + args.steps, args.steps, dominant)
    ms_per_step = gpu_ms / args.steps
    events = w.batch * args.steps
    value = events / (gpu_ms / 1e3)
    target_events = sum(n_tar[args.warmup:args.warmup + args.steps])

    out = {
        "metric": "events/sec per batch step (fwd+bwd) on 1 MI355X; % HBM / MFMA roofline",
        "value": value,
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "wall_ms_per_step": wall * 1e3 / args.steps,
        "host_enqueue_ms_per_step": enq * 1e3 / args.steps,
        "target_events_per_s": target_events / (gpu_ms / 1e3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "n_nodes": w.n_nodes, "n_events": w.n_events, "batch": w.batch, "k": w.k,
                   "d_mem": w.d_mem, "d_time": w.d_time, "d_edge": w.d_edge, "d_attn": w.d_attn,
                   "n_heads": w.n_heads, "first_batch": b0, "order": "lag-1"},
    }

    # algorithmic work of the dominant kernel: valid neighbour slots of the steps it was timed on
    lo2, hi2 = args.warmup + args.steps, n_steps
    valid_pairs = sum(valid_slots(runner, s, w, b0 + i) for i in range(lo2, hi2))
    launches_per_step = dom_launches / args.steps
    # every launch of a hot site covers all valid slots of its step (K and V share one launch)
    per_launch_pairs = valid_pairs / args.steps / max(launches_per_step, 1.0)
    flops = 2.0 * per_launch_pairs * SITE_K(dominant, w) * SITE_N(dominant, w)
    avg_s = dom_ms / 1e3 / max(dom_launches, 1)
    peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    achieved = flops / avg_s / 1e12
    out["roofline"] = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                       "frac": achieved / peak, "traffic": read_traffic(dominant, w), "kernel": dominant,
                       "launches_per_step": launches_per_step, "avg_launch_us": avg_s * 1e6,
                       "flops_per_launch": flops, "timed_over": f"steps {lo2}..{hi2 - 1} after the headline's "
                       f"(their ms/step {gpu_ms2 / args.steps:.4f})",
                       "warmup_site_us": {k: v * 1e3 for k, v in site_ms.items()}}
    out["step_counts"] = step_counts(runner, s, w, b0, args.warmup, args.steps)

    if args.cpu_steps > 0:
        out["cpu_baseline"] = cpu_baseline(w, s, params, mem, lu, b0, args.cpu_steps)
    print(json.dumps(out), flush=True)


def other_model(args):
    """The JODIE step, or Algorithm 2's loop for one worker: one JSON line, events/s over K timed steps."""
    import torch

    from synth import init_params, init_params_jodie, make_stream, node_owner, window_state, workload
    w = workload(args.workload)
    s = make_stream(w)
    b0 = w.window_b0
    mem, lu = window_state(w, s, b0)
    out = {"metric": "events/sec per batch step (fwd+bwd) on 1 MI355X; % HBM / MFMA roofline", "unit": "events/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if w.dtype == "bf16" else "f32", "data": "synthetic",
           "roofline": None}
    if args.model == "jodie":
        from paper_2608_16305_amd.jodie_step import JodieStep
        r = JodieStep(w, s, init_params_jodie(w), mem, lu)
        for i in range(args.warmup):
            r.step(b0 + i)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record()
        for i in range(args.warmup, args.warmup + args.steps):
            r.step(b0 + i)
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1)
        out.update(value=w.batch * args.steps / (ms / 1e3), ms_per_step=ms / args.steps,
                   config={"workload": w.name, "model": "JODIE (recurrent update, time projection, masked link loss)",
                           "batch": w.batch, "d_mem": w.d_mem, "d_time": w.d_time, "first_batch": b0})
    else:
        from paper_2608_16305_amd.runtime import AdaptiveTrainer
        P = args.workers
        tr = AdaptiveTrainer(w, s, init_params(w), mem, lu, node_owner(w.n_nodes, P), 0, P, args.window)
        n = min(tr.n_batches, args.warmup + args.steps)
        for r in range(args.warmup):
            tr.batch(r)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for r in range(args.warmup, n):
            tr.batch(r)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        recs = tr.records[args.warmup:n]
        ev = sum(x.n_events for x in recs)
        tar = sum(int(((tr.local.flags[tr.batch_off[x.r]:tr.batch_off[x.r + 1]] & 1) == 0).sum()) for x in recs)
        out.update(value=ev / wall, ms_per_step=wall * 1e3 / len(recs), target_events_per_s=tar / wall,
                   decisions={"refresh": sum(x.sync for x in recs), "skipped": sum(x.boundary and not x.sync
                                                                                   for x in recs),
                              "heavy": sum(x.heavy for x in recs)},
                   config={"workload": w.name, "model": "TGN, Algorithm 2 loop of worker 0", "workers": P,
                           "window": args.window, "batches": len(recs), "replay_share": float(
                               (tr.local.flags & 1).mean()), "note": "from the stream's start; memory from the "
                           "window snapshot; wall-clock incl. the per-batch host reads Algorithm 2 needs"})
    print(json.dumps(out), flush=True)


# Matrix-product call sites over the neighbour slots (the largest products of the step).
HOT_SITES = ("gemm_kv_proj", "gemm_kv_dw", "gemm_kv_dx")


def SITE_K(site, w):
    """Reduction length per neighbour slot of each hot site's product."""
    return {"gemm_kv_proj": w.d_kv, "gemm_kv_dw": 2 * w.d_attn, "gemm_kv_dx": 2 * w.d_attn}[site]


def SITE_N(site, w):
    """Output width: K|V (2 d_attn), [dW_k; dW_v] (d_kv per row of 2 d_attn), dphi (d_time)."""
    return {"gemm_kv_proj": 2 * w.d_attn, "gemm_kv_dw": w.d_kv, "gemm_kv_dx": w.d_time}[site]


def valid_slots(runner, s, w, b):
    """Non-padded neighbour slots of step b's queries, counted on the host from the device-built
    adjacency (outside the timed regions): per query, min(k, entries of its node strictly before
    its time), by one binary search over the keys (node << 32 | float bits of t), which sort as the
    adjacency does since times are non-negative."""
    if not hasattr(runner, "_adj_keys"):
        off = runner.csr_off.cpu().numpy()
        ct = runner.csr_t.cpu().numpy()[:off[-1]]
        node = np.repeat(np.arange(off.size - 1, dtype=np.uint64), np.diff(off))
        runner._adj_keys = (node << np.uint64(32)) | ct.view(np.uint32).astype(np.uint64)
        runner._adj_off = off
    elo, ehi = runner.batch_range(b)
    tar = np.ones(ehi - elo, bool) if s.flags is None else (s.flags[elo:ehi] & 3) == 0
    q_node = np.concatenate([s.src[elo:ehi][tar], s.dst[elo:ehi][tar], s.neg[elo:ehi][tar]]).astype(np.uint64)
    q_t = np.tile(s.t[elo:ehi][tar], 3).astype(np.float32)
    qk = (q_node << np.uint64(32)) | q_t.view(np.uint32).astype(np.uint64)
    before = np.searchsorted(runner._adj_keys, qk, side="left") - runner._adj_off[q_node.astype(np.int64)]
    return int(np.minimum(before, w.k).sum())


# ------------------------------------------------------------------ HBM traffic from counter runs

CSRC = os.path.join(ROOT, "paper_2608_16305_amd", "csrc")
# sources that define the hot-site kernels and their launches
TRAFFIC_SOURCES = ("common.h", "gemm.h", "gemm.hip", "gemm_nt.hip", "gemm_nn.hip", "gemm_tn.hip", "gemm_rs.h",
                   "gemm_rs.hip", "lds_dma.h", "attention.hip")


def kernel_fingerprint():
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def traffic_path(w):
    return os.path.join(ROOT, "profiles", f"hot-sites-{w.name}.traffic.json")


def read_traffic(site, w):
    """HBM bytes per launch of `site` from the committed counter record, or None when
    there is none or the kernel sources changed since the counters were taken."""
    p = traffic_path(w)
    if not os.path.exists(p):
        return None
    with open(p) as fh:
        rec = json.load(fh)
    if rec.get("fingerprint") != kernel_fingerprint() or site not in rec.get("sites", {}):
        return None
    return rec["sites"][site]["bytes_per_launch"]


def _site_of(name):
    for site, tag in (("gemm_kv_proj", "KvProj"), ("gemm_kv_dw", "KvDw"), ("gemm_kv_dx", "KvDx")):
        if f"site::{tag}," in name:
            return site
    return None


def _counter_rows(path, counter):
    import csv
    with open(path) as fh:
        rows = [r for r in csv.DictReader(fh) if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def _calibrated(path, counter, probe_bytes):
    """Per-site mean counter value (KiB per dispatch) scaled by the copy-probe factor."""
    rows = _counter_rows(path, counter)
    first_step = next(i for i, r in enumerate(rows) if "mtgnn::(anonymous namespace)::k_agg_" in r["Kernel_Name"] or "mtgnn::k_agg_" in r["Kernel_Name"])
    probes = [r for r in rows[:first_step] if "copyBuffer" in r["Kernel_Name"]][-2:]
    if len(probes) != 2:
        raise SystemExit(f"{path}: the two probe copies before the first step were not found")
    probe_kib = sum(float(r["Counter_Value"]) for r in probes) / 2
    factor = probe_bytes / 1024.0 / probe_kib
    per = {}
    for r in rows[first_step:]:
        site = _site_of(r["Kernel_Name"])
        if site:
            per.setdefault(site, []).append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v)) * factor * 1024.0 for k, v in per.items()}, factor, probe_kib, \
        {k: len(v) for k, v in per.items()}


def write_traffic(args):
    from synth import workload
    w = workload(args.workload)
    probe = args.copy_probe * (1 << 20)
    if probe <= 0:
        raise SystemExit("--traffic-from needs --copy-probe MIB (the probe size of the counter runs)")
    fetch, ff, fkib, nf = _calibrated(args.traffic_from[0], "FETCH_SIZE", probe)
    write, fw, wkib, nw = _calibrated(args.traffic_from[1], "WRITE_SIZE", probe)
    sites = {s: {"fetch_bytes_per_launch": fetch[s], "write_bytes_per_launch": write[s],
                 "bytes_per_launch": fetch[s] + write[s], "dispatches": nf[s]} for s in fetch if s in write}
    rec = {"workload": w.name, "fingerprint": kernel_fingerprint(), "probe_bytes": probe,
           "probe_fetch_kib": fkib, "probe_write_kib": wkib, "fetch_factor": ff, "write_factor": fw,
           "sites": sites}
    os.makedirs(os.path.dirname(traffic_path(w)), exist_ok=True)
    with open(traffic_path(w), "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    n, mib = args.workload, args.copy_probe
    lines = [f"# HBM traffic of the neighbour-slot products on {w.name} (fp32)", "",
             "Two counter passes, each its own run (repository root, MI355X), then the record:", "", "```",
             f"timeout -s KILL 400 rocprofv3 --pmc FETCH_SIZE -f csv -d gpurun_out/pmcF_w{n} -o run -- python -u bench.py "
             f"--workload {n} --steps 2 --warmup 1 --cpu-steps 0 --copy-probe {mib}",
             f"timeout -s KILL 400 rocprofv3 --pmc WRITE_SIZE -f csv -d gpurun_out/pmcW_w{n} -o run -- python -u bench.py "
             f"--workload {n} --steps 2 --warmup 1 --cpu-steps 0 --copy-probe {mib}",
             f"python bench.py --workload {n} --copy-probe {mib} --traffic-from "
             f"gpurun_out/pmcF_w{n}/run_counter_collection.csv gpurun_out/pmcW_w{n}/run_counter_collection.csv", "```", "",
             f"Calibration: `--copy-probe {mib}` copies a {mib} MiB buffer twice just before the first step; the copy "
             f"reads FETCH_SIZE = {fkib:.0f} KiB and WRITE_SIZE = {wkib:.0f} KiB for {probe // 1024} KiB moved each way, "
             f"so FETCH_SIZE is scaled by {ff:.4f} and WRITE_SIZE by {fw:.4f}.", "",
             f"Per launch (mean over the run's dispatches), from `{os.path.basename(traffic_path(w))}`, which bench.py "
             "reads for its `traffic` field while the hash of the kernel sources (`fingerprint`) matches:", "",
             "| site | fetch MB | write MB | total MB | dispatches |", "|---|---|---|---|---|"]
    for k, v in sites.items():
        lines.append(f"| {k} | {v['fetch_bytes_per_launch'] / 1e6:.1f} | {v['write_bytes_per_launch'] / 1e6:.1f} | "
                     f"{v['bytes_per_launch'] / 1e6:.1f} | {v['dispatches']} |")
    with open(os.path.join(ROOT, "profiles", f"hbm-traffic-hot-sites-{w.name}.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps(rec))


def step_counts(runner, s, w, b0, first, count):
    """Mean per-step sizes of the timed steps: updated rows (the memory batch's distinct non-pruned
    endpoints), queries and valid neighbour slots (host-side counts, outside the timed region)."""
    U = Q = P = 0
    for i in range(first, first + count):
        b = b0 + i
        mlo, mhi = (b - 1) * w.batch, b * w.batch
        act = np.ones(mhi - mlo, bool) if s.flags is None else (s.flags[mlo:mhi] & 2) == 0
        U += np.unique(np.concatenate([s.src[mlo:mhi][act], s.dst[mlo:mhi][act]])).size
        elo, ehi = runner.batch_range(b)
        Q += 3 * (ehi - elo if s.flags is None else int(((s.flags[elo:ehi] & 3) == 0).sum()))
        P += valid_slots(runner, s, w, b)
    return {"updated_rows": U / count, "queries": Q / count, "valid_slots": P / count}


def _clean_kernel(name):
    for x in ("mtgnn::", "(anonymous namespace)::", "site::"):
        name = name.replace(x, "")
    return name.split("(")[0]


def kernel_report(args):
    """Per kernel of the step: mean duration (kernel trace), calibrated FETCH_SIZE and WRITE_SIZE bytes per
    dispatch (counter runs), achieved GB/s and its fraction of the 8 TB/s HBM peak."""
    import csv
    from synth import workload
    w = workload(args.workload)
    probe = args.copy_probe * (1 << 20)
    if probe <= 0:
        raise SystemExit("--kernel-report needs --copy-probe MIB (the probe size of the counter runs)")
    trace_csv, fetch_csv, write_csv = args.kernel_report
    dur = {}
    with open(trace_csv) as fh:
        for r in csv.DictReader(fh):
            k = _clean_kernel(r["Kernel_Name"])
            dur.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)

    def counter(path, name):
        rows = _counter_rows(path, name)
        first = next(i for i, r in enumerate(rows) if "k_agg_reset" in r["Kernel_Name"])
        probes = [r for r in rows[:first] if "copyBuffer" in r["Kernel_Name"]][-2:]
        factor = probe / 1024.0 / (sum(float(r["Counter_Value"]) for r in probes) / 2)
        per = {}
        for r in rows[first:]:
            per.setdefault(_clean_kernel(r["Kernel_Name"]), []).append(float(r["Counter_Value"]) * 1024.0 * factor)
        return {k: sum(v) / len(v) for k, v in per.items()}, factor

    fetch, ff = counter(fetch_csv, "FETCH_SIZE")
    write, fw = counter(write_csv, "WRITE_SIZE")
    rows = []
    for k in fetch:
        if k not in write or k not in dur or "copyBuffer" in k:
            continue
        us = sorted(dur[k])[len(dur[k]) // 2]
        by = fetch[k] + write[k]
        rows.append({"kernel": k, "median_us": us, "fetch_MB": fetch[k] / 1e6, "write_MB": write[k] / 1e6,
                     "GBps": by / (us * 1e-6) / 1e9, "hbm_frac": by / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "launches": len(dur[k])})
    rows.sort(key=lambda r: -r["median_us"])
    base = os.path.join(ROOT, "profiles", f"kernel-hbm-{w.name}")
    rec = {"workload": w.name, "fetch_factor": ff, "write_factor": fw, "probe_bytes": probe, "kernels": rows}
    with open(base + ".json", "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    n = args.workload
    lines = [f"# HBM traffic and achieved bandwidth per kernel, {w.name} (MI355X)", "",
             "Three runs of the same step (repository root), then the report:", "", "```",
             f"rocprofv3 --kernel-trace --stats -f csv -d gpurun_out/kt_w{n} -o run -- python -u bench.py --workload {n} "
             f"--steps 10 --warmup 3 --cpu-steps 0",
             f"timeout -s KILL 400 rocprofv3 --pmc FETCH_SIZE -f csv -d gpurun_out/pmcF_w{n} -o run -- python -u bench.py "
             f"--workload {n} --steps 2 --warmup 1 --cpu-steps 0 --copy-probe {args.copy_probe}",
             f"timeout -s KILL 400 rocprofv3 --pmc WRITE_SIZE -f csv -d gpurun_out/pmcW_w{n} -o run -- python -u bench.py "
             f"--workload {n} --steps 2 --warmup 1 --cpu-steps 0 --copy-probe {args.copy_probe}",
             f"python bench.py --workload {n} --copy-probe {args.copy_probe} --kernel-report "
             f"gpurun_out/kt_w{n}/run_kernel_trace.csv gpurun_out/pmcF_w{n}/run_counter_collection.csv "
             f"gpurun_out/pmcW_w{n}/run_counter_collection.csv", "```", "",
             f"Calibration: the {args.copy_probe} MiB probe copy reads FETCH_SIZE x {ff:.4f} and WRITE_SIZE x {fw:.4f} "
             "of the bytes it moves; both counters are scaled by those factors.  Bytes are per dispatch (mean over the "
             "counter runs), durations the median of the kernel-trace run, GB/s = (fetch + write) / duration, and the "
             "fraction is of the 8 TB/s HBM3E peak.  Matrix-product kernels are listed for completeness: their bound "
             "is the MFMA rate, not HBM.", "",
             "| median us | fetch MB | write MB | GB/s | % of HBM peak | launches | kernel |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['median_us']:.1f} | {r['fetch_MB']:.1f} | {r['write_MB']:.1f} | {r['GBps']:.0f} | "
                     f"{100 * r['hbm_frac']:.1f} | {r['launches']} | `{r['kernel'][:100]}` |")
    with open(base + ".md", "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"written": base + ".json", "kernels": len(rows)}))


MFMA_SIMDS = 256 * 4      # MI355X: 256 compute units, 4 SIMDs each
MFMA_CLOCK_GHZ = 2.4      # peak engine clock


def mfma_report(args):
    """Per matrix kernel of the step: median duration (kernel trace) and the mean MFMA-busy cycles per dispatch
    (SQ_VALU_MFMA_BUSY_CYCLES, summed over the SIMDs), as a fraction of all SIMDs' cycles over the duration at
    the peak engine clock (a lower bound when the clock runs below its peak)."""
    import csv
    from synth import workload
    w = workload(args.workload)
    trace_csv, sq_csv = args.mfma_report
    dur = {}
    with open(trace_csv) as fh:
        for r in csv.DictReader(fh):
            dur.setdefault(_clean_kernel(r["Kernel_Name"]), []).append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    rows_c = _counter_rows(sq_csv, "SQ_VALU_MFMA_BUSY_CYCLES")
    first = next(i for i, r in enumerate(rows_c) if "k_agg_reset" in r["Kernel_Name"])
    busy = {}
    for r in rows_c[first:]:
        busy.setdefault(_clean_kernel(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    rows = []
    for k, v in busy.items():
        cyc = sum(v) / len(v)
        if cyc <= 0 or k not in dur:
            continue
        us = sorted(dur[k])[len(dur[k]) // 2]
        rows.append({"kernel": k, "median_us": us, "mfma_busy_cycles": cyc, "launches": len(dur[k]),
                     "mfma_busy_frac": cyc / (MFMA_SIMDS * us * 1e3 * MFMA_CLOCK_GHZ)})
    rows.sort(key=lambda r: -r["median_us"])
    base = os.path.join(ROOT, "profiles", f"mfma-busy-{w.name}")
    with open(base + ".json", "w") as fh:
        json.dump({"workload": w.name, "simds": MFMA_SIMDS, "clock_ghz": MFMA_CLOCK_GHZ, "kernels": rows}, fh, indent=1)
        fh.write("\n")
    n = args.workload
    lines = [f"# MFMA-busy fraction per matrix kernel, {w.name} (MI355X)", "",
             "Two runs of the same step (repository root), then the report:", "", "```",
             f"rocprofv3 --kernel-trace --stats -f csv -d gpurun_out/kt_w{n} -o run -- python -u bench.py --workload {n} "
             f"--steps 10 --warmup 3 --cpu-steps 0",
             f"timeout -s KILL 400 rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES -f csv -d gpurun_out/pmcQ_w{n} "
             f"-o run -- python -u bench.py --workload {n} --steps 2 --warmup 1 --cpu-steps 0",
             f"python bench.py --workload {n} --mfma-report gpurun_out/kt_w{n}/run_kernel_trace.csv "
             f"gpurun_out/pmcQ_w{n}/run_counter_collection.csv", "```", "",
             "SQ_VALU_MFMA_BUSY_CYCLES counts the cycles the matrix cores are busy, summed over the SIMDs (each "
             "v_mfma_f32_16x16x4_f32 adds 32: a kernel's count matches its instruction count times 32).  The "
             "fraction divides the mean per dispatch "
             f"by {MFMA_SIMDS} SIMDs x the median duration x {MFMA_CLOCK_GHZ} GHz; in the step the two streams share "
             "the chip, so a kernel that ran beside another shows less than it would alone.", "",
             "| median us | MFMA-busy cycles (M) | MFMA busy % | launches | kernel |", "|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['median_us']:.1f} | {r['mfma_busy_cycles'] / 1e6:.2f} | {100 * r['mfma_busy_frac']:.1f} | "
                     f"{r['launches']} | `{r['kernel'][:100]}` |")
    with open(base + ".md", "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"written": base + ".json", "kernels": len(rows)}))


def step_report(args):
    """Kernel time per step of a profiled bench run: the totals of rocprofv3's kernel statistics over the step
    intervals between consecutive aggregation launches (the first warmup steps skipped)."""
    import csv
    from synth import workload
    w = workload(args.workload)
    d, bench_json = args.step_report
    with open(os.path.join(d, "run_kernel_trace.csv")) as fh:
        trace = sorted(csv.DictReader(fh), key=lambda r: int(r["Start_Timestamp"]))
    idx = [i for i, r in enumerate(trace) if "k_agg_reset" in r["Kernel_Name"]]
    spans = list(zip(idx[3:-1], idx[4:]))
    if not spans:
        raise SystemExit(f"{d}: too few steps in the trace")
    per = {}
    total = 0.0
    for a, b in spans:
        for r in trace[a:b]:
            us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            k = _clean_kernel(r["Kernel_Name"])
            t, c = per.get(k, (0.0, 0))
            per[k] = (t + us, c + 1)
            total += us
    ns = len(spans)
    with open(bench_json) as fh:
        bench = json.loads(fh.read().strip().splitlines()[-1])
    rl = bench["roofline"]
    n = args.workload
    lines = [f"# Kernel time of one batch step on {w.name} (MI355X)", "", "Command (repository root):", "", "```",
             f"rocprofv3 --kernel-trace --stats -f csv -d gpurun_out/kt_w{n} -o run -- python -u bench.py --workload {n} "
             f"--steps 10 --warmup 3 --cpu-steps 0",
             f"python bench.py --workload {n} --step-report gpurun_out/kt_w{n} BENCH_LINE.json", "```", "",
             f"Per-step figures average the {ns} step intervals between the 4th and the last aggregation launch (the "
             f"warmup's first steps are skipped).  Kernel time per step: {total / ns:.1f} us in "
             f"{sum(c for _, c in per.values()) / ns:.0f} launches (two streams overlap, so the step takes less).", "",
             f"bench.py headline (separate run, `python -u bench.py --workload {n} --cpu-steps 0`): "
             f"{bench['value'] / 1e6:.3f} M events/s, {bench['ms_per_step'] * 1e3:.1f} us per step; step sizes "
             f"{json.dumps(bench.get('step_counts', {}))}; dominant product `{rl['kernel']}` "
             f"{rl['avg_launch_us']:.1f} us per launch, {rl['achieved']:.1f} TFLOP/s = {100 * rl['frac']:.2f}% of "
             f"{rl['peak']} TFLOP/s.", "",
             "| % of kernel time | us/step | launches/step | us/launch | kernel |", "|---|---|---|---|---|"]
    for k, (t, c) in sorted(per.items(), key=lambda kv: -kv[1][0])[:45]:
        lines.append(f"| {100 * t / total:.2f} | {t / ns:.2f} | {c / ns:.2f} | {t / c:.2f} | `{k[:110]}` |")
    path = os.path.join(ROOT, "profiles", f"step-kernels-{w.name}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"written": path, "kernels": len(per)}))


def cpu_baseline(w, s, params, mem, lu, b0, n):
    """The oracle (unchanged) on the host cores, over the first n steps of the same window, once with
    its BLAS pinned to one thread and once with all threads."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import tgn
    # the adjacency lists the sample needs: those of the nodes its steps query (the oracle's own build)
    q_nodes = []
    for i in range(n):
        lo, hi = (b0 + i) * w.batch, (b0 + i + 1) * w.batch
        tar = np.ones(hi - lo, bool) if s.flags is None else (s.flags[lo:hi] & 3) == 0
        q_nodes += [s.src[lo:hi][tar], s.dst[lo:hi][tar], s.neg[lo:hi][tar]]
    adj = tgn.build_adjacency_for(s.src, s.dst, s.t, w.n_nodes, np.unique(np.concatenate(q_nodes)))
    prec = tgn.Prec("bf16" if w.dtype == "bf16" else "f32")

    def run():
        m, l = mem.copy(), lu.copy()
        t0 = time.perf_counter()
        for i in range(n):
            b = b0 + i
            mb = tgn.batch_dict(s, (b - 1) * w.batch, b * w.batch)
            eb = tgn.batch_dict(s, b * w.batch, (b + 1) * w.batch)
            r = tgn.step(prec, w, m, l, params, adj, s.x, mb, eb, None, loss="link")
            m, l = r.mp.mem, r.mp.lu
        return w.batch * n / (time.perf_counter() - t0)

    with threadpool_limits(limits=1):
        one = run()
    allv = run()
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": allv, "unit": "events/s", "cores": threads, "kind": "oracle",
            "single_thread": {"value": one, "cores": 1},
            "sample": f"{n} consecutive steps from batch {b0} of the same workload ({w.batch * n} events), "
                      f"float64 NumPy oracle, timed with its BLAS at all {threads} threads and again at 1; "
                      f"{os.cpu_count()} host CPUs visible"}


if __name__ == "__main__":
    main()
