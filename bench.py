"""Benchmark: batched what-if simulation on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM: dd_graph_load (validate, rank thread chains,
cross-thread edge lists) -> dd_levelize (GPU Kahn phases) ->
dd_apply_transforms (per-variant tables) -> dd_simulate_batch (every
variant's start/finish, makespan reduced in the same kernel).

Prints one JSON line.  `value` = task-variant updates per second of the
whole step (N * V per step).  `roofline` covers the simulation kernel:
algorithmic bytes of one launch over its average duration (HIP events on the
launching stream).  `cpu_baseline` times the oracle on the host cores on a
bounded variant sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def algorithmic_bytes(n, V, n_gathers, n_cls, want_start=False):
    """Bytes one simulate launch must move at minimum:
    per (task, variant): 8 B finish (+8 B start) + 1/8 B removal bit;
    per (gather, variant): 8 B source finish + 1/8 B source removal bit;
    per task: schedule record (node id 4, duration 8, gap 8, class 2, flags 1,
    gather offset 8 = 31 B); per gather: source 4, position 4, class 1, gap 8
    = 17 B; per (class, variant): 16 B scale entry."""
    per_tv = 8.0 + (8.0 if want_start else 0.0) + 1.0 / 8
    per_gv = 8.0 + 1.0 / 8
    return (n * V * per_tv + n_gathers * V * per_gv + n * 31.0 + n_gathers * 17.0
            + n_cls * V * 16.0)


def breakdown_bytes(n_role, n_wait, n, V, n_cls):
    """Bytes one runtime-breakdown call must move at minimum: the removal
    bit of every (task with a role, variant); the finish of every waiting
    call and of its thread predecessor per variant; per task the role and
    class (counting sort) and, for tasks with a role, duration, class, role
    and order entry; the scale table; the output."""
    return (n_role * V / 8.0 + 2.0 * n_wait * V * 8.0 + n * 3.0 + n_role * 19.0
            + n_cls * V * 16.0 + V * 32.0)


def bench_breakdown(di, g, vs, stream, reps):
    """Time dd_runtime_breakdown on one simulated batch (HIP events on the
    launching stream)."""
    import torch
    from paper_2006_03318_amd import batch, binding as B, workloads as W
    role = torch.from_numpy(W.task_roles(g)).to(di.tensors["dur"].device)
    res, gh, handles = batch.simulate(di, stream=stream, keep_handles=True)
    times = []
    nbytes = 0.0
    try:
        outs = [torch.empty((v1 - v0, 4), dtype=torch.int64, device=fin.device)
                for (v0, v1, fin, _s, _m) in res]
        rn = W.task_roles(g)
        n_role, n_wait = int((rn == 1).sum() + (rn == 2).sum()), int((rn == 2).sum())
        for (v0, v1, *_r) in res:
            nbytes += breakdown_bytes(n_role, n_wait, g.n, v1 - v0, di.n_cls)
        for it in range(reps + 2):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for (v0, v1, fin, _s, ms), (_sch, var), out in zip(res, handles, outs):
                B.dd_runtime_breakdown(gh, var, role, fin, ms, out, stream)
            e1.record(stream)
            stream.synchronize()
            if it >= 2:
                times.append(e0.elapsed_time(e1))
    finally:
        for sch, var in handles:
            B.dd_sched_free(sch)
            B.dd_variants_free(var)
        B.dd_graph_free(gh)
    ms_call = float(np.mean(times))
    achieved = nbytes / (ms_call / 1e3) / 1e9
    pairs = float(n_role) * vs.n_variants
    return {"kernel": "k_bd_accum", "calls_timed": reps, "avg_call_ms": round(ms_call, 4),
            "tasks_with_role": n_role, "waiting_calls": n_wait,
            "task_variant_pairs_per_s": round(pairs / (ms_call / 1e3), 1),
            "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": None, "algorithmic_bytes_per_call": int(nbytes)}}


def policy_bytes(n, V, n_edges_out):
    """Bytes one schedule-rule call must move at minimum: per (task,
    variant) the finish written (8 B), the reference count and start written
    at set-up (12 B) and the task's frontier metadata read when it becomes
    ready (thread 4, priority 4, push/pull flag 1, removal bit 1/8); per
    (out-edge, variant) one read-modify-write of the child's count and start
    (2 x 12 B); per task its record (32 B), duration and gap (16 B) and
    out-edges (4 B each), read once per variant."""
    per_tv = 8.0 + 12.0 + 9.0 + 1.0 / 8 + 48.0
    return n * V * per_tv + n_edges_out * V * (24.0 + 4.0)


def bench_policy(stream, reps, cpu_workers):
    """Time dd_simulate_policy (both rules) on the VGG-19 parameter-server
    workload with P3's sliced pushes and pulls, and time the oracle on the
    same variants."""
    import torch
    from paper_2006_03318_amd import binding as B, workloads as W
    from oracle import oracle as O
    g, vs, pp, prio = W.p3_workload(iters=32, variants=2048)
    dev = torch.device("cuda:0")

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    gl = B.dd_graph_load_ex(g.n, g.n_threads, t(g.in_ptr), t(g.in_src), t(g.edge_cls),
                            t(g.thread_prev), t(g.thread_id), t(g.dur), t(g.gap), t(g.node_cls),
                            B.DD_LOAD_SHARED_THREADS, stream)
    V = vs.n_variants
    out = {}
    try:
        var = B.dd_apply_transforms(gl, V, int(vs.scale.shape[0]), t(vs.scale), t(vs.remove_bits),
                                    t(vs.edge_on[:, 0]), stream)
        fin = torch.empty((g.n, V), dtype=torch.int64, device=dev)
        ms = torch.empty((V,), dtype=torch.int64, device=dev)
        dpp, dprio = t(pp), t(prio)
        for policy, name in ((B.DD_POLICY_EARLIEST, "earliest"), (B.DD_POLICY_PRIORITY, "p3")):
            times = []
            for it in range(reps + 1):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                B.dd_simulate_policy(gl, var, policy, dpp, dprio, fin, None, ms, stream)
                e1.record(stream)
                stream.synchronize()
                if it >= 1:
                    times.append(e0.elapsed_time(e1))
            out[name] = (float(np.mean(times)), ms.cpu().numpy().copy())
        B.dd_variants_free(var)
    finally:
        B.dd_graph_free(gl)
    cores = max(1, min(len(os.sched_getaffinity(0)), cpu_workers))
    t0 = time.perf_counter()
    _, _, oms = O.run_policy(g, vs, 1, pp, prio, want_start=False, want_finish=False,
                             workers=cores)
    cpu_s = time.perf_counter() - t0
    ms_call, gms = out["p3"]
    n_out = g.n_edges + int((g.thread_prev >= 0).sum())
    nbytes = policy_bytes(g.n, V, n_out)
    achieved = nbytes / (ms_call / 1e3) / 1e9
    steps = float(g.n) * V
    return {"kernel": "k_sim_event", "workload": "%s: %d tasks (%d push/pull slices on 2 "
                                                 "shared channels) x %d variants" %
                                                 (g.name, g.n, int(pp.sum()), V),
            "calls_timed": reps,
            "avg_call_ms": {"p3": round(ms_call, 3), "earliest": round(out["earliest"][0], 3)},
            "task_variant_steps_per_s": round(steps / (ms_call / 1e3), 1),
            "ns_per_step_per_variant": round(ms_call * 1e6 / g.n, 1),
            "parity_all_makespans_equal": bool(np.array_equal(gms, oms)),
            "p3_over_earliest_mean_makespan": round(float(np.mean(gms / out["earliest"][1])), 4),
            "cpu_oracle": {"value": round(steps / cpu_s, 1), "unit": "task-variant steps/s",
                           "cores": cores, "kind": "oracle",
                           "sample": "all %d variants (%.2f s wall)" % (V, cpu_s)},
            "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": None, "algorithmic_bytes_per_call": int(nbytes)}}


def kernel_source_digest():
    """sha256 over the sources the simulation kernel is compiled from and
    the build script (it holds the kernel's compile flags)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("csrc/k_simulate.hip", "csrc/dd_internal.h", "csrc/dd_common.h", "build.py"):
        with open(os.path.join(ROOT, "paper_2006_03318_amd", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(config, n, V):
    """HBM bytes per launch from the committed counter summary of this
    workload (FETCH_SIZE + WRITE_SIZE, each scaled by the plain copy's), or
    None when there is none or the kernel's sources changed since."""
    path = os.path.join(ROOT, "profiles", "k_sim_pipe_transformer_x32_counters.md")
    if config != 5 or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("traffic_bytes_per_launch:"):
            for tok in line.split()[1:]:
                k, _, v = tok.partition("=")
                fields[k] = v
            break
    if fields.get("source_sha256") != kernel_source_digest():
        return None
    if fields.get("tasks") != str(n) or fields.get("variants") != str(V):
        return None
    return int(fields["bytes"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--variants", type=int, default=None)
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="variants the oracle runs for the CPU baseline (-1 = all, 0 = skip)")
    ap.add_argument("--cpu-workers", type=int, default=16,
                    help="oracle worker threads at most (the host share of one GPU is 16 "
                         "cores)")
    ap.add_argument("--breakdown-reps", type=int, default=5,
                    help="timed dd_runtime_breakdown calls after the steps (0 = skip)")
    ap.add_argument("--policy-reps", type=int, default=3,
                    help="timed dd_simulate_policy calls per rule on the P3 workload (0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device three times: the plain copy "
                         "whose byte counters scale the simulation kernel's")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the simulation shards over variants with no "
              "exchange between shards, and runs on more than one GPU are not part of "
              "this benchmark (--gpus %d not supported)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2006_03318_amd import batch, binding as B, workloads as W

    assert torch.cuda.is_available(), "bench needs a GPU"
    if args.copy_calibration > 0:
        nb = args.copy_calibration << 20
        src = torch.ones(nb // 8, dtype=torch.int64, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": nb, "copy_bytes_written": nb, "copies": 3}))
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    t0 = time.time()
    g, vs = W.config(args.config, variants=args.variants)
    gen_s = time.time() - t0
    print("[bench] %s: %d tasks, %d dependency edges, %d threads, %d variants "
          "(generated in %.1f s)" % (g.name, g.n, g.n_edges, g.n_threads, vs.n_variants,
                                     gen_s), file=sys.stderr, flush=True)
    di = batch.to_device(g, vs, device=dev)
    outs = []
    for (v0, v1, *_r) in di.batches:
        Vb = v1 - v0
        outs.append((torch.empty((g.n, Vb), dtype=torch.int64, device=dev), None,
                     torch.empty((Vb,), dtype=torch.int64, device=dev)))
    torch.cuda.synchronize()

    E = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    rows = {"load": [], "levelize": [], "transforms": [], "simulate": []}
    info = {}
    binfo = [None] * len(di.batches)      # schedule shape of each batch

    def step(record):
        ev = [E() for _ in range(2 + 3 * len(di.batches))]
        ev[0].record(stream)
        gh = batch.load_graph(di, stream)
        ev[1].record(stream)
        k = 2
        hs = []
        for bi, (v0, v1, mask, scale, rm, eon) in enumerate(di.batches):
            sch, nsteps = B.dd_levelize(gh, mask, B.DD_PHASES, stream)
            ev[k].record(stream)
            var = B.dd_apply_transforms(gh, v1 - v0, di.n_cls, scale, rm, eon, stream)
            ev[k + 1].record(stream)
            fin, st, ms = outs[bi]
            B.dd_simulate_batch(gh, sch, var, fin, st, ms, stream)
            ev[k + 2].record(stream)
            if binfo[bi] is None:
                binfo[bi] = B.dd_sched_info(sch)
                binfo[bi]["plan"] = B.dd_simulate_plan(sch, var)
            if not info:
                info.update(binfo[bi])
            hs.append((sch, var))
            k += 3
        for sch, var in hs:
            B.dd_sched_free(sch)
            B.dd_variants_free(var)
        B.dd_graph_free(gh)
        if record:
            stream.synchronize()
            rows["load"].append(ev[0].elapsed_time(ev[1]))
            k = 2
            prev = ev[1]
            lv = tr = sm = 0.0
            for _ in di.batches:
                lv += prev.elapsed_time(ev[k])
                tr += ev[k].elapsed_time(ev[k + 1])
                sm += ev[k + 1].elapsed_time(ev[k + 2])
                prev = ev[k + 2]
                k += 3
            rows["levelize"].append(lv)
            rows["transforms"].append(tr)
            rows["simulate"].append(sm)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(True)
        print("[bench] step %d/%d done" % (i + 1, args.steps), file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    NV = g.n * vs.n_variants
    value = NV / (ms_per_step / 1e3)

    # simulate time per step = sum over the batches' launches; bytes likewise
    sim_ms = float(np.mean(rows["simulate"]))
    nbytes = sum(algorithmic_bytes(g.n, v1 - v0, bi_["n_gathers"], di.n_cls)
                 for (v0, v1, *_r), bi_ in zip(di.batches, binfo))
    achieved = nbytes / (sim_ms / 1e3) / 1e9
    # the few-variant path (negative plan) launches a kernel per step of
    # more than one chunk (plus one that clears its look-back slots); its
    # "launch" here is the whole simulate call of a batch
    split = all(b["plan"] < 0 for b in binfo)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": None if split else measured_traffic(args.config, g.n, vs.n_variants),
                "kernel": "k_sim_phase" if split else "k_sim_pipe",
                "algorithmic_bytes_per_launch": int(nbytes),
                "avg_launch_ms": round(sim_ms / len(di.batches), 4),
                "launches_per_step": len(di.batches),
                "variants_per_workgroup": [b["plan"] for b in binfo]}

    # the runtime breakdown (CPU-only / GPU-only / CPU+GPU parallel) of every
    # variant, after the timed steps
    bd = None
    if args.breakdown_reps > 0:
        bd = bench_breakdown(di, g, vs, stream, args.breakdown_reps)

    # the schedule-rule path (Sec. 4.4 "Schedule", the P3 model) on its own
    # workload, after the timed steps
    pol = None
    if args.policy_reps > 0:
        pol = bench_policy(stream, args.policy_reps, args.cpu_workers)

    # parity sample + CPU baseline: the oracle on the first variants
    cpu = None
    parity = None
    if args.cpu_sample != 0:
        from oracle import oracle as O
        O.build(force=False)
        ns = vs.n_variants if args.cpu_sample < 0 else min(args.cpu_sample, vs.n_variants)
        avail = len(os.sched_getaffinity(0))
        cores = max(1, min(avail, args.cpu_workers))
        t0 = time.perf_counter()
        _, _, oms, _ = O.run(g, vs, variants=range(ns), want_start=False, want_finish=False,
                             workers=cores)
        cpu_s = time.perf_counter() - t0
        # one core: a bounded sample of about two seconds of oracle work
        per_core = g.n * ns / cpu_s / cores          # rate estimate per worker
        n1 = max(1, min(ns, int(2.0 * per_core / max(1, g.n))))
        t1 = time.perf_counter()
        O.run(g, vs, variants=range(n1), want_start=False, want_finish=False, workers=1)
        one_s = time.perf_counter() - t1
        cpu = {"value": round(g.n * ns / cpu_s, 1), "unit": "node-variant updates/s",
               "cores": cores, "kind": "oracle",
               "sample": "%s%d of %d variants, all %d tasks (%.1f s wall on %d worker threads)"
                         % ("" if ns == vs.n_variants else "first ", ns, vs.n_variants, g.n,
                            cpu_s, cores),
               "nproc": os.cpu_count(), "affinity_cpus": avail,
               "worker_cap": "at most %d worker threads: the host share of one GPU"
                             % args.cpu_workers,
               "single_core_value": round(g.n * n1 / one_s, 1),
               "single_core_sample": "first %d variants on 1 worker thread (%.2f s)"
                                     % (n1, one_s)}
        gms = np.concatenate([m.cpu().numpy() for (_, _, m) in outs])[:ns]
        parity = bool(np.array_equal(gms, oms))

    out = {
        "metric": "simulated node-variant updates/sec + achieved HBM GB/s (dd_simulate_batch)",
        "value": round(value, 1),
        "unit": "node-variant updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic (seeded trace-shaped task graph, random-variant tables)",
        "config": {"workload": "%s sweep: %d tasks x %d variants, %d dependency edges, "
                               "%d threads" % (g.name, g.n, vs.n_variants, g.n_edges,
                                               g.n_threads),
                   "tasks": g.n, "variants": vs.n_variants, "phases": info.get("n_steps"),
                   "gathers": info.get("n_gathers")},
        "breakdown_ms": {k: round(float(np.mean(v)), 3) for k, v in rows.items()},
        "simulate_only_updates_per_s": round(NV / (sim_ms / 1e3), 1),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "runtime_breakdown": bd,
        "schedule_policy": pol,
        "parity_sample_makespans_equal": parity,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
