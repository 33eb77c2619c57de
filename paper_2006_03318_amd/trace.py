"""Trace -> task graph: the dependency-graph construction of Sec. 4.2 and the
task-to-layer mapping of Sec. 4.3, from rocprofv3 CSV output on ROCm.

Input: the files rocprofv3 writes with
    --kernel-trace --hip-runtime-trace --memory-copy-trace --marker-trace
    --output-format csv -d DIR -o PREFIX
(PREFIX_kernel_trace.csv, PREFIX_hip_api_trace.csv,
PREFIX_memory_copy_trace.csv, PREFIX_marker_api_trace.csv; the last two are
optional).  Output: a `workloads.TaskGraph` the C-ABI and the recipe
compiler take, with the measured timeline of every task.

Tasks (Sec. 4.2.1): every HIP runtime call is a CPU task on its host thread;
every kernel dispatch and memory copy is a GPU task on its stream (agent,
stream id).  Duration = end - start.  A CPU task's gap is the time from its
end to the start of the next task on its thread (the non-HIP CPU work the
trace cannot see); GPU tasks have no gap.

Dependencies (Sec. 4.2.2):
  * order of the tasks of one CPU thread, and of one GPU stream (by start);
  * correlation: the call that issued a GPU task -> that task (same
    correlation id);
  * synchronization: a call that waits for the device (device, stream or
    event synchronize) depends on the last GPU task of every stream issued by
    a call that started before it;
  * blocking copies (hipMemcpy, hipMemcpyWithStream, the D2H direction of
    hipMemcpyAsync, ...): the call waits for its own copy.
  Communication tasks are not in a one-GPU trace; the Distributed recipe
  adds them.

Readings where the trace or the paper leaves a choice (each is listed in
the design notes):
  * a synchronization call's duration is the part after the work it waited
    for ended (the wait itself is the dependency): end - max(start, latest
    end among the awaited GPU tasks);
  * a blocking copy call becomes two CPU tasks on its thread: the issue part
    (from its start until its copy began, with the correlation edge to the
    copy) and the return part (after the copy ended until the call
    returned, depending on the copy); the gap follows the return part;
  * the CSV carries no stream or event arguments, so every synchronize waits
    on all streams;
  * layers: the innermost marker range (roctx, e.g. torch.cuda.nvtx) on a
    CPU task's thread that contains its start gives its layer; a GPU task
    takes the layer of the call that issued it.  Ranges named
    "iteration <k>" give the iteration instead;
  * a host thread whose first call in the window comes after the window's
    first task starts with a zero-length task whose gap is that offset (what
    started the thread is not a traced dependency).

Host-only and plain Python/numpy: the graph is built once per trace.
"""
from __future__ import annotations

import csv
import dataclasses
import os
import re
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import workloads as W

# HIP runtime calls that issue device work (their correlated GPU tasks follow)
ISSUE_CALLS = {
    "hipLaunchKernel", "hipExtModuleLaunchKernel", "hipModuleLaunchKernel",
    "hipExtLaunchKernel", "hipLaunchCooperativeKernel", "hipExtLaunchKernelGGL",
    "hipLaunchKernelExC", "hipGraphLaunch", "hipMemcpyAsync", "hipMemsetAsync",
    "hipMemsetD8Async", "hipMemsetD16Async", "hipMemsetD32Async", "hipMemcpy2DAsync",
    "hipMemcpy3DAsync", "hipMemcpyHtoDAsync", "hipMemcpyDtoHAsync", "hipMemcpyDtoDAsync",
    "hipMemcpyPeerAsync", "hipMemcpyToSymbolAsync", "hipMemcpyFromSymbolAsync",
}
# calls that return only after their own device work is done
BLOCKING_COPY_CALLS = {
    "hipMemcpy", "hipMemcpyWithStream", "hipMemcpyHtoD", "hipMemcpyDtoH", "hipMemcpyDtoD",
    "hipMemcpy2D", "hipMemcpy3D", "hipMemset", "hipMemsetD8", "hipMemsetD16", "hipMemsetD32",
    "hipMemcpyToSymbol", "hipMemcpyFromSymbol", "hipMemcpyPeer",
}
# calls that wait for earlier device work
SYNC_CALLS = {"hipDeviceSynchronize", "hipStreamSynchronize", "hipEventSynchronize",
              "hipCtxSynchronize"}

_ITER_RE = re.compile(r"^iteration\s+(\d+)$")


@dataclasses.dataclass
class TraceGraph:
    """A graph built from a trace, with what the trace measured."""
    graph: W.TaskGraph
    names: List[str]                 # call or kernel name of every task
    layer_names: List[str]           # layer ids -> marker range names
    measured_start: np.ndarray       # int64 [n], ns from the window start
    measured_end: np.ndarray
    cpu_threads: List[int]           # host thread id of each CPU execution thread
    gpu_streams: List[Tuple[str, int]]   # (agent, stream id) of each GPU execution thread

    @property
    def measured_span(self) -> int:
        return int(self.measured_end.max() - self.measured_start.min()) if self.graph.n else 0


def _read(path: str) -> List[dict]:
    if not os.path.exists(path):
        return []
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def read_rocprof_csv(directory: str, prefix: str = "run") -> Dict[str, List[dict]]:
    """The four CSV tables (missing ones are empty)."""
    p = lambda s: os.path.join(directory, "%s_%s.csv" % (prefix, s))   # noqa: E731
    t = {"kernel": _read(p("kernel_trace")), "api": _read(p("hip_api_trace")),
         "memcpy": _read(p("memory_copy_trace")), "marker": _read(p("marker_api_trace"))}
    if not t["api"]:
        raise ValueError("no HIP API trace in %s (prefix %s)" % (directory, prefix))
    return t


def kernel_kind(name: str) -> Tuple[int, int]:
    """(task kind, operator tag) of a GPU kernel from its name (the Select by
    keyword of Sec. 4.4)."""
    s = name.lower()
    op = W.OP_NONE
    if "relu" in s or "threshold" in s:
        op = W.OP_RELU
    elif "batchnorm" in s or "batch_norm" in s:
        op = W.OP_BN
    elif "conv" in s or "igemm" in s or "winograd" in s:
        op = W.OP_CONV
    if s.startswith("cijk_") or ("gemm" in s and "igemm" not in s) or "matmul" in s:
        return W.K_GEMM, op
    if op == W.OP_CONV:
        return W.K_CONV, op
    if "multi_tensor_apply" in s or "adam" in s or "sgd" in s:
        return W.K_OPT, op
    if "elementwise" in s or "pointwise" in s or op in (W.OP_RELU, W.OP_BN):
        return W.K_ELEM, op
    return W.K_GPU_OTHER, op


def _layer_op(layer_name: str) -> int:
    s = layer_name.lower()
    if "conv" in s:
        return W.OP_CONV
    if "batchnorm" in s:
        return W.OP_BN
    if "relu" in s:
        return W.OP_RELU
    return W.OP_NONE


def build_graph(tables: Dict[str, List[dict]], window: Optional[Tuple[int, int]] = None,
                iterations: Optional[Sequence[int]] = None) -> TraceGraph:
    """Build the graph of the calls that start inside `window` (absolute ns,
    default everything), or inside the marker ranges "iteration <k>" for k in
    `iterations`, with the GPU tasks they issued."""
    api = tables["api"]
    markers = tables.get("marker", [])
    if iterations is not None:
        spans = []
        for m in markers:
            mm = _ITER_RE.match(m["Function"].strip())
            if mm and int(mm.group(1)) in set(iterations):
                spans.append((int(m["Start_Timestamp"]), int(m["End_Timestamp"])))
        if not spans:
            raise ValueError("no marker range for iterations %s" % list(iterations))
        window = (min(a for a, _ in spans), max(b for _, b in spans))
    lo, hi = window if window is not None else (-(1 << 62), 1 << 62)

    # ---- CPU calls in the window ----
    calls = [r for r in api if lo <= int(r["Start_Timestamp"]) <= hi]
    calls.sort(key=lambda r: (int(r["Start_Timestamp"]), int(r["Correlation_Id"])))
    corr_call = {int(r["Correlation_Id"]): i for i, r in enumerate(calls)}
    # ---- GPU work they issued ----
    gpu = []
    for r in tables["kernel"]:
        c = int(r["Correlation_Id"])
        if c in corr_call:
            gpu.append(("kernel", r, c, (r["Agent_Id"], int(r["Stream_Id"]))))
    for r in tables.get("memcpy", []):
        c = int(r["Correlation_Id"])
        if c in corr_call:
            gpu.append(("copy", r, c, (r["Destination_Agent_Id"]
                                       if "HOST_TO_DEVICE" in r["Direction"] or
                                       "DEVICE_TO_DEVICE" in r["Direction"]
                                       else r["Source_Agent_Id"], int(r["Stream_Id"]))))
    gpu.sort(key=lambda x: (int(x[1]["Start_Timestamp"]), x[2]))
    own: Dict[int, List[int]] = {}
    for j, (_, _, c, _) in enumerate(gpu):
        own.setdefault(corr_call[c], []).append(j)

    # ---- tasks: CPU calls (blocking copies split in two), then GPU tasks ----
    # each entry: (start, end, thread key, kind, name, call index or -1, gpu index or -1, part)
    T = []
    for i, r in enumerate(calls):
        f = r["Function"]
        s, e = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        key = ("cpu", int(r["Thread_Id"]))
        blocking = f in BLOCKING_COPY_CALLS or (
            f in ("hipMemcpyAsync", "hipMemcpyDtoHAsync") and any(
                gpu[j][0] == "copy" and "DEVICE_TO_HOST" in gpu[j][1]["Direction"]
                for j in own.get(i, [])))
        if blocking and i in own:
            g0 = min(int(gpu[j][1]["Start_Timestamp"]) for j in own[i])
            g1 = max(int(gpu[j][1]["End_Timestamp"]) for j in own[i])
            mid = min(max(g0, s), e)
            T.append([s, mid, key, W.K_SYNC, f + ":issue", i, -1, 1])
            T.append([max(g1, mid) if max(g1, mid) <= e else e, e, key, W.K_SYNC, f + ":return",
                      i, -1, 2])
        else:
            kind = W.K_SYNC if f in SYNC_CALLS else (W.K_LAUNCH if f in ISSUE_CALLS or i in own
                                                     else W.K_API)
            T.append([s, e, key, kind, f, i, -1, 0])
    for j, (typ, r, c, skey) in enumerate(gpu):
        s, e = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        if typ == "kernel":
            kind, op = kernel_kind(r["Kernel_Name"])
            name = r["Kernel_Name"]
        else:
            kind, op, name = W.K_MEMCPY, W.OP_NONE, r["Direction"]
        T.append([s, e, ("gpu",) + skey, kind, name, -1, j, 0])
    # a host thread whose first call comes after the window's start gets a
    # zero-length first task at the start, with the offset as its gap (what
    # set that thread going -- e.g. the main thread starting the backward
    # pass -- is not among the traced dependencies)
    if T:
        t_min = min(t[0] for t in T)
        first: Dict[tuple, int] = {}
        for t in T:
            if t[2][0] == "cpu":
                first[t[2]] = min(first.get(t[2], t[0]), t[0])
        for key, s0 in sorted(first.items()):
            if s0 > t_min:
                T.append([t_min, t_min, key, W.K_API, "(thread start)", -1, -1, 3])
    # ids in trace order
    order = sorted(range(len(T)), key=lambda k: (T[k][0], T[k][1], k))
    T = [T[k] for k in order]
    n = len(T)
    start = np.array([t[0] for t in T], np.int64)
    end = np.array([max(t[1], t[0]) for t in T], np.int64)
    # threads: CPU threads first, then GPU streams
    keys = sorted({t[2] for t in T}, key=lambda k: (k[0] != "cpu", k))
    tix = {k: i for i, k in enumerate(keys)}
    thread = np.array([tix[t[2]] for t in T], np.int32)
    kind = np.array([t[3] for t in T], np.uint8)
    is_cpu = np.array([t[2][0] == "cpu" for t in T], bool)

    # sequential order per thread (by start, then end, then trace order)
    prev = np.full(n, -1, np.int32)
    nxt = np.full(n, -1, np.int64)
    for k in range(len(keys)):
        ids = np.nonzero(thread == k)[0]
        ids = ids[np.lexsort((ids, end[ids], start[ids]))]
        prev[ids[1:]] = ids[:-1]
        nxt[ids[:-1]] = ids[1:]
    dur = end - start
    gap = np.zeros(n, np.int64)
    has_next = is_cpu & (nxt >= 0)
    gap[has_next] = np.maximum(0, start[nxt[has_next]] - end[has_next])
    # the issue part of a blocking copy hands over to its return part with no
    # CPU work between them: the wait is the dependency on the copy
    part = np.array([t[7] for t in T], np.int8)
    gap[part == 1] = 0
    # a thread-start task waits until its thread's first call
    for u in np.nonzero(part == 3)[0]:
        gap[u] = start[nxt[u]] - start[u]

    # id of each call's task(s) and of each GPU task
    call_task: Dict[int, List[int]] = {}
    gpu_task = np.full(len(gpu), -1, np.int64)
    for u, t in enumerate(T):
        if t[5] >= 0:
            call_task.setdefault(t[5], []).append(u)
        if t[6] >= 0:
            gpu_task[t[6]] = u
    edges: List[Tuple[int, int]] = []
    launch_of = np.full(n, -1, np.int64)
    # correlation: the call (its issue part) -> its GPU tasks
    for i, js in own.items():
        src = min(call_task[i], key=lambda u: T[u][7] if T[u][7] else 0)
        for j in js:
            edges.append((src, int(gpu_task[j])))
            launch_of[gpu_task[j]] = src
    # blocking copies: the return part waits for the call's own copies
    for i, us in call_task.items():
        ret = [u for u in us if T[u][7] == 2]
        for u in ret:
            for j in own.get(i, []):
                edges.append((int(gpu_task[j]), u))
    # synchronization: the last GPU task of every stream issued before the call
    gpu_ids = np.nonzero(~is_cpu)[0]
    issue_start = np.full(n, np.iinfo(np.int64).max, np.int64)
    for u in gpu_ids:
        if launch_of[u] >= 0:
            issue_start[u] = start[launch_of[u]]
    streams = sorted({int(thread[u]) for u in gpu_ids})
    by_stream = {k: gpu_ids[thread[gpu_ids] == k] for k in streams}
    for k in streams:                 # stream order = issue order
        ids = by_stream[k]
        by_stream[k] = ids[np.lexsort((ids, issue_start[ids]))]
    for u in range(n):
        if not (is_cpu[u] and T[u][4] in SYNC_CALLS):
            continue
        waited_end = -1
        for k in streams:
            ids = by_stream[k]
            pos = np.searchsorted(issue_start[ids], start[u], side="left") - 1
            if pos >= 0:
                w = int(ids[pos])
                edges.append((w, u))
                waited_end = max(waited_end, int(end[w]))
        # the call's own time is what follows the wait
        if waited_end > start[u]:
            dur[u] = max(0, int(end[u]) - waited_end)
    # in-edge CSR (sources sorted by trace order)
    if edges:
        e = np.array(sorted(set(edges), key=lambda x: (x[1], x[0])), np.int64)
    else:
        e = np.zeros((0, 2), np.int64)
    in_ptr = np.zeros(n + 1, np.int64)
    np.add.at(in_ptr, e[:, 1] + 1, 1)
    in_ptr = np.cumsum(in_ptr)

    # ---- layers and iterations from marker ranges (Sec. 4.3) ----
    layer = np.full(n, -1, np.int32)
    iteration = np.zeros(n, np.int32)
    op = np.zeros(n, np.uint8)
    layer_names: List[str] = []
    lid: Dict[str, int] = {}
    by_thread: Dict[int, List[Tuple[int, int, str]]] = {}
    for m in markers:
        by_thread.setdefault(int(m["Thread_Id"]), []).append(
            (int(m["Start_Timestamp"]), int(m["End_Timestamp"]), m["Function"].strip()))
    for u in range(n):
        if not is_cpu[u]:
            continue
        rs = by_thread.get(T[u][2][1], [])
        best = None
        for (a, b, nm) in rs:
            if a <= start[u] <= b and not _ITER_RE.match(nm):
                if best is None or (b - a) < (best[1] - best[0]):
                    best = (a, b, nm)
        if best is not None:
            if best[2] not in lid:
                lid[best[2]] = len(layer_names)
                layer_names.append(best[2])
            layer[u] = lid[best[2]]
    # iteration: the latest "iteration <k>" range started (on any thread:
    # backward passes may run on another host thread) before the call
    it_spans = sorted((a, int(_ITER_RE.match(nm).group(1))) for rs in by_thread.values()
                      for (a, b, nm) in rs if _ITER_RE.match(nm))
    if it_spans:
        a_s = np.array([a for a, _ in it_spans], np.int64)
        k_s = np.array([k for _, k in it_spans], np.int32)
        for u in range(n):
            if is_cpu[u]:
                pos = np.searchsorted(a_s, start[u], side="right") - 1
                if pos >= 0:
                    iteration[u] = k_s[pos]
    for u in gpu_ids:
        lo_ = launch_of[u]
        if lo_ >= 0:
            layer[u] = layer[lo_]
            iteration[u] = iteration[lo_]
    for u in range(n):
        if not is_cpu[u] and T[u][3] != W.K_MEMCPY:
            op[u] = kernel_kind(T[u][4])[1]
            if op[u] == W.OP_NONE and layer[u] >= 0:
                op[u] = _layer_op(layer_names[layer[u]])
    t0 = int(start.min()) if n else 0
    g = W.TaskGraph(n, len(keys), in_ptr, e[:, 0].astype(np.int32), np.zeros(e.shape[0], np.uint8),
                    prev, thread, dur, gap, np.zeros(n, np.uint16), 1, 1, kind, layer,
                    launch_of, "trace", op=op, iteration=iteration)
    return TraceGraph(g, [t[4] for t in T], layer_names, start - t0, end - t0,
                      [k[1] for k in keys if k[0] == "cpu"],
                      [(k[1], k[2]) for k in keys if k[0] == "gpu"])
