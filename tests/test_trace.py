"""The trace front end (Sec. 4.2 tasks and dependencies, Sec. 4.3 layer
mapping) on rocprofv3 CSV traces.

* a hand-written trace whose graph is derived by hand: task order, threads,
  thread order, durations, gaps, kinds, every dependency type and layers;
* round trips: a timeline the simulation itself produced, written out as a
  rocprofv3 trace and read back, is reproduced exactly by the rebuilt graph
  (every finish time, every start but the synchronization calls', whose
  start in the model is the end of their wait);
* a real trace of a small CNN training on an MI355X (two steady-state
  iterations): its structure, and the simulated iteration time against the
  measured one.
"""
import csv
import os
import tempfile

import numpy as np
import pytest

from paper_2006_03318_amd import recipes as R
from paper_2006_03318_amd import trace as TR
from paper_2006_03318_amd import workloads as W
from tests import helpers as H

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_toy_trace_by_hand():
    tg = TR.build_graph(TR.read_rocprof_csv(os.path.join(GOLD, "trace_toy")))
    g = tg.graph
    assert tg.names == ["(thread start)", "hipGetDevice", "hipLaunchKernel", "hipLaunchKernel",
                        "miopenSp3AsmConv_v30_fp32_stride1", "hipMemcpyAsync",
                        "hipDeviceSynchronize", "hipLaunchKernel",
                        "void at::native::vectorized_elementwise_kernel<4, relu_functor>",
                        "MEMORY_COPY_HOST_TO_DEVICE", "Cijk_Ailk_Bljk_S_B_MT32x16x64",
                        "hipMemcpyWithStream:issue", "MEMORY_COPY_DEVICE_TO_HOST",
                        "hipMemcpyWithStream:return"]
    # threads: host 100, host 200, then the stream; host 200 starts with a
    # zero-length task whose gap reaches its first call
    assert tg.cpu_threads == [100, 200] and tg.gpu_streams == [("Agent 1", 0)]
    assert g.thread_id.tolist() == [1, 0, 0, 0, 2, 0, 0, 1, 2, 2, 2, 0, 2, 0]
    assert g.thread_prev.tolist() == [-1, -1, 1, 2, -1, 3, 5, 0, 4, 8, 9, 6, 10, 11]
    assert tg.measured_start.tolist() == [0, 0, 5, 18, 20, 30, 40, 45, 50, 61, 71, 80, 90, 110]
    # the synchronize keeps what followed its wait: 1075 - 1070
    assert g.dur.tolist() == [0, 2, 10, 8, 30, 4, 5, 7, 10, 9, 8, 10, 20, 10]
    # CPU gaps up to the next call of the thread; none after an issue part
    assert g.gap.tolist() == [45, 3, 3, 4, 0, 6, 5, 0, 0, 0, 0, 0, 0, 0]
    K = W
    assert g.kind.tolist() == [K.K_API, K.K_API, K.K_LAUNCH, K.K_LAUNCH, K.K_CONV, K.K_LAUNCH,
                               K.K_SYNC, K.K_LAUNCH, K.K_ELEM, K.K_MEMCPY, K.K_GEMM, K.K_SYNC,
                               K.K_MEMCPY, K.K_SYNC]
    dst = np.repeat(np.arange(g.n), np.diff(g.in_ptr))
    edges = sorted(zip(g.in_src.tolist(), dst.tolist()))
    # correlation 2->4, 3->8, 5->9, 7->10, 11->12; the synchronize waits on
    # the copy issued last before it (9 -> 6); the blocking copy returns
    # after its copy (12 -> 13)
    assert edges == sorted([(2, 4), (3, 8), (5, 9), (7, 10), (11, 12), (9, 6), (12, 13)])
    assert g.launch_of.tolist() == [-1, -1, -1, -1, 2, -1, -1, -1, 3, 5, 7, -1, 11, -1]
    assert tg.layer_names == ["fwd layer0:Conv2d", "fwd layer1:ReLU", "bwd layer0:Conv2d"]
    assert g.layer.tolist() == [-1, -1, 0, 1, 0, -1, -1, 2, 1, -1, 2, -1, -1, -1]
    assert g.op[4] == W.OP_CONV and g.op[8] == W.OP_RELU and (g.iteration == 0).all()


def test_toy_trace_simulates(oracle_mod):
    """Worked by hand: kernels start when their call and gap are done (the
    convolution at 5 + 10 + 3 = 18, two ns before the trace has it: the
    launch latency the model does not carry), the synchronize when the
    copy issued before it ends (67), the blocking copy's return part when
    its copy ends (107)."""
    tg = TR.build_graph(TR.read_rocprof_csv(os.path.join(GOLD, "trace_toy")))
    S, F, M, _ = oracle_mod.run(tg.graph, H.variants(tg.graph, V=1))
    assert S[0].tolist() == [0, 0, 5, 18, 18, 30, 67, 45, 48, 58, 67, 77, 87, 107]
    assert M[0] == 117 and tg.measured_span == 120


# --------------------------------------------------------------------------
# round trips
_NAMES = {W.K_GEMM: "Cijk_Alik_Bljk_S_MT64", W.K_ELEM: "vectorized_elementwise_kernel<add>",
          W.K_CONV: "miopenSp3AsmConv_fp32", W.K_GPU_OTHER: "batched_transpose_32x16",
          W.K_OPT: "multi_tensor_apply_kernel<sgd>"}


def _random_program(rng, n_ops, n_streams):
    """One host thread issuing kernels and asynchronous copies on several
    streams, with device synchronizations and blocking copies."""
    b = W._Builder(1 + n_streams)
    streams = list(range(1, 1 + n_streams))
    blocking = []
    for _ in range(n_ops):
        r = rng.random()
        s = int(rng.choice(streams))
        if r < 0.7:
            kind = int(rng.choice(list(_NAMES)))
            b.launch(0, s, kind, int(rng.integers(0, 4)))
        elif r < 0.8:
            b.launch(0, s, W.K_MEMCPY, -1)
        elif r < 0.9:
            b.sync(0, streams, -1)
        else:
            issue = b.task(0, W.K_SYNC, -1)
            cp = b.task(s, W.K_MEMCPY, -1, launch_of=issue)
            b.edge(issue, cp)
            ret = b.task(0, W.K_SYNC, -1)
            b.edge(cp, ret)
            blocking.append((issue, cp, ret))
    t = W._template(b, 4)
    g = W._tile(t, 1, rng, {k: 20_000 for k in _NAMES}, (5_000, 50_000), "roundtrip")
    for issue, _, _ in blocking:
        g.gap[issue] = 0
    # a trace cannot see host work after the thread's last call
    cpu = np.nonzero(g.thread_id == 0)[0]
    g.gap[cpu[-1]] = 0
    return g, blocking


def _write_trace(d, g, S, blocking):
    """The simulated timeline as rocprofv3 CSV files."""
    F = S + g.dur
    R = F + g.gap
    n = g.n
    corr = np.arange(n) + 1000
    role = {}
    for issue, cp, ret in blocking:
        role[issue] = ("issue", cp, ret)
        role[ret] = ("skip",)
    api, ker, cps = [], [], []
    cpu = np.nonzero(g.thread_id == 0)[0]
    arrival = {}
    for u in cpu:
        p = g.thread_prev[u]
        arrival[u] = int(R[p]) if p >= 0 else 0
    child = {int(g.launch_of[k]): k for k in range(n) if g.launch_of[k] >= 0}
    for u in cpu:
        u = int(u)
        if role.get(u, ("",))[0] == "skip":
            continue
        if role.get(u, ("",))[0] == "issue":
            _, cp, ret = role[u]
            api.append(("hipMemcpyWithStream", corr[cp], arrival[u], int(F[ret])))
        elif g.kind[u] == W.K_SYNC:
            api.append(("hipDeviceSynchronize", corr[u], arrival[u], int(F[u])))
        else:
            k = child[u]
            api.append(("hipMemcpyAsync" if g.kind[k] == W.K_MEMCPY else "hipLaunchKernel",
                        corr[k], int(S[u]), int(F[u])))
    for k in range(n):
        if g.thread_id[k] == 0:
            continue
        if g.kind[k] == W.K_MEMCPY:
            blk = any(k == cp for _, cp, _ in blocking)
            cps.append(("MEMORY_COPY_DEVICE_TO_HOST" if blk else "MEMORY_COPY_HOST_TO_DEVICE",
                        int(g.thread_id[k]), corr[k], int(S[k]), int(F[k])))
        else:
            ker.append((int(g.thread_id[k]), _NAMES[int(g.kind[k])], corr[k], int(S[k]),
                        int(F[k])))
    with open(os.path.join(d, "run_hip_api_trace.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Domain", "Function", "Process_Id", "Thread_Id", "Correlation_Id",
                    "Start_Timestamp", "End_Timestamp"])
        for fn, c, a, b in api:
            w.writerow(["HIP_RUNTIME_API_EXT", fn, 7, 7, int(c), a, b])
    with open(os.path.join(d, "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id",
                    "Kernel_Id", "Kernel_Name", "Correlation_Id", "Start_Timestamp",
                    "End_Timestamp"])
        for i, (s, nm, c, a, b) in enumerate(ker):
            w.writerow(["KERNEL_DISPATCH", "Agent 1", 1, s, 7, i, 1, nm, int(c), a, b])
    with open(os.path.join(d, "run_memory_copy_trace.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Kind", "Direction", "Stream_Id", "Source_Agent_Id", "Destination_Agent_Id",
                    "Correlation_Id", "Start_Timestamp", "End_Timestamp"])
        for dr, s, c, a, b in cps:
            src, dst = ("Agent 1", "Agent 0") if "TO_HOST" in dr else ("Agent 0", "Agent 1")
            w.writerow(["MEMORY_COPY", dr, s, src, dst, int(c), a, b])


@pytest.mark.parametrize("seed", range(12))
def test_round_trip_reproduces_the_timeline(oracle_mod, seed):
    rng = np.random.default_rng(9100 + seed)
    g, blocking = _random_program(rng, int(rng.integers(5, 120)), int(rng.integers(1, 4)))
    S, F, M, _ = oracle_mod.run(g, H.variants(g, V=1))
    d = tempfile.mkdtemp(prefix="dd_trace_")
    _write_trace(d, g, S[0], blocking)
    tg = TR.build_graph(TR.read_rocprof_csv(d))
    g2 = tg.graph
    assert g2.n == g.n
    S2, F2, M2, _ = oracle_mod.run(g2, H.variants(g2, V=1))
    assert M2[0] == M[0]
    assert (F2[0] == tg.measured_end).all()
    plain = g2.kind != W.K_SYNC
    assert (S2[0][plain] == tg.measured_start[plain]).all()
    # the rebuilt graph has the program's dependencies: one correlation edge
    # per device task, each sync waits on every stream that has work
    gpu = g2.thread_id >= 1
    assert (g2.launch_of[gpu] >= 0).all() and (g2.launch_of[~gpu] < 0).all()


# --------------------------------------------------------------------------
def _cnn():
    return TR.build_graph(TR.read_rocprof_csv(os.path.join(GOLD, "rocprof_cnn")),
                          iterations=[2, 3])


def test_real_trace_structure():
    tg = _cnn()
    g = tg.graph
    gpu = np.isin(g.kind, W.GPU_KINDS + (W.K_MEMCPY,))
    assert int(np.isin(g.kind, W.GPU_KINDS).sum()) == 88          # 44 kernels per iteration
    assert (g.launch_of[gpu] >= 0).all()                           # every GPU task has its call
    assert len(tg.cpu_threads) == 2 and len(tg.gpu_streams) == 1   # main and autograd threads
    assert set(np.unique(g.iteration).tolist()) == {2, 3}
    # the layer ranges cover the forward and backward kernels of all layers
    names = {tg.layer_names[l] for l in g.layer[np.isin(g.kind, W.GPU_KINDS) & (g.layer >= 0)]}
    assert {"fwd layer0:Conv2d", "bwd layer3:Conv2d", "fwd layer8:Linear", "bwd layer8:Linear"} <= names
    conv = np.isin(g.kind, (W.K_CONV,))
    assert conv.sum() >= 4 and (g.op[conv] == W.OP_CONV).all()
    assert ((g.kind == W.K_GEMM).sum()) >= 4
    # blocking copies of the inputs and of the loss value: issue and return parts
    assert sum(n.endswith(":issue") for n in tg.names) == 6
    assert (g.gap >= 0).all() and (g.dur >= 0).all()


def test_real_trace_iteration_time(oracle_mod):
    """The unmodified graph's simulated time against the measured one (the
    accuracy question of Sec. 6: this small model is bound by its CPU
    threads, where the gaps carry the measured host time)."""
    tg = _cnn()
    g = tg.graph
    S, F, M, _ = oracle_mod.run(g, H.variants(g, V=1))
    err = abs(int(M[0]) - tg.measured_span) / tg.measured_span
    assert err <= 0.01, err
    # what-if sweeps run on it like on any graph: AMP cannot lengthen it,
    # halving the launch cost shortens a CPU-bound iteration
    g2, vs = R.compile_sweep(g, [[], [R.AMP()], [R.ScaleLaunch(1, 2)]])
    _, _, M2, _ = oracle_mod.run(g2, vs)
    assert M2[1] <= M2[0] and M2[2] < M2[0]
