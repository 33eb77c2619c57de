"""Small builders shared by the tests (no simulation arithmetic here)."""
from __future__ import annotations

import numpy as np

from paper_2006_03318_amd.workloads import TaskGraph, VariantSet, pack_bits


def graph(n_threads, thread, edges, dur, gap, cls=None, edge_cls=None, n_cls=None,
          n_edge_cls=None, thread_order=None):
    """Tasks 0..n-1 on `thread[i]`; thread order = id order unless
    `thread_order` (list of per-thread id lists) is given; edges (src, dst)."""
    n = len(thread)
    thread = np.asarray(thread, np.int32)
    prev = np.full(n, -1, np.int32)
    if thread_order is None:
        last = {}
        for i in range(n):
            t = int(thread[i])
            if t in last:
                prev[i] = last[t]
            last[t] = i
    else:
        for lst in thread_order:
            for a, b in zip(lst[:-1], lst[1:]):
                prev[b] = a
    edges = list(edges)
    ec = list(edge_cls) if edge_cls is not None else [0] * len(edges)
    order = sorted(range(len(edges)), key=lambda i: edges[i][1])
    in_ptr = np.zeros(n + 1, np.int64)
    for s, d in edges:
        in_ptr[d + 1] += 1
    in_ptr = np.cumsum(in_ptr)
    src = np.array([edges[i][0] for i in order], np.int32)
    ecls = np.array([ec[i] for i in order], np.uint8)
    cls = np.zeros(n, np.uint16) if cls is None else np.asarray(cls, np.uint16)
    return TaskGraph(n, n_threads, in_ptr, src, ecls, prev, thread,
                     np.asarray(dur, np.int64), np.asarray(gap, np.int64), cls,
                     int(n_cls or (int(cls.max()) + 1 if n else 1)),
                     int(n_edge_cls or (int(ecls.max()) + 1 if ecls.size else 1)),
                     np.zeros(n, np.uint8), np.full(n, -1, np.int32), np.full(n, -1, np.int64))


def variants(g: TaskGraph, scales=None, removed=None, edge_on=None, V=None):
    """scales: list over variants of {cls: (p, q)}; removed: list over
    variants of task-id lists; edge_on: list of class masks."""
    V = V or max(len(scales or [0]), len(removed or [0]), len(edge_on or [0]))
    C = g.n_node_cls
    s = np.ones((C, V, 2), np.int32)
    for v, sc in enumerate(scales or []):
        for c, pq in sc.items():
            s[c, v] = pq
    bits = np.zeros((g.n, V), bool)
    for v, rm in enumerate(removed or []):
        for u in rm:
            bits[u, v] = True
    eo = np.full((V, 1), np.uint64((1 << 64) - 1), np.uint64)
    for v, m in enumerate(edge_on or []):
        eo[v, 0] = np.uint64(m)
    return VariantSet(V, s, pack_bits(bits), eo, [(0, V, (1 << 64) - 1)])
