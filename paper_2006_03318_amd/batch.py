"""Sequencing of C-ABI calls for one workload: load the graph, levelize once
per edge-class batch, build the transform tables and simulate.  Only calls
the library through `binding`; torch provides device memory and the stream.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

from . import binding as B


@dataclasses.dataclass
class DeviceInputs:
    """Graph and variant tables already resident in device memory."""
    n: int
    n_threads: int
    tensors: dict
    batches: List[tuple]        # (v0, v1, edge-class mask, scale, rm_bits, edge_on)
    n_cls: int
    n_variants: int


def to_device(g, vs, device="cuda") -> DeviceInputs:
    import torch

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)
    ten = dict(in_ptr=t(g.in_ptr.astype(np.int64)), in_src=t(g.in_src.astype(np.int32)),
               edge_cls=t(g.edge_cls.astype(np.uint8)),
               thread_prev=t(g.thread_prev.astype(np.int32)),
               thread_id=t(g.thread_id.astype(np.int32)), dur=t(g.dur.astype(np.int64)),
               gap=t(g.gap.astype(np.int64)), node_cls=t(g.node_cls.astype(np.uint16)))
    batches = []
    for (v0, v1, mask) in vs.batches:
        sub = vs if (v0 == 0 and v1 == vs.n_variants) else vs.subset(v0, v1)
        batches.append((v0, v1, mask, t(sub.scale.astype(np.int32)),
                        t(sub.remove_bits.astype(np.uint32)),
                        t(sub.edge_on[:, 0].astype(np.uint64))))
    return DeviceInputs(g.n, g.n_threads, ten, batches, int(vs.scale.shape[0]), vs.n_variants)


def load_graph(di: DeviceInputs, stream=None):
    x = di.tensors
    return B.dd_graph_load(di.n, di.n_threads, x["in_ptr"], x["in_src"], x["edge_cls"],
                           x["thread_prev"], x["thread_id"], x["dur"], x["gap"], x["node_cls"],
                           stream)


def simulate(di: DeviceInputs, mode=B.DD_PHASES, want_start=False, stream=None,
             outputs: Optional[list] = None, keep_handles=False, variants_per_wg: int = 0):
    """Run every batch; returns a list of (v0, v1, finish[N][Vb], start, makespan[Vb]).
    variants_per_wg: 0 = the library's launch shape, else 1/2/4/8/16, or -1/-2/-4/-8 for
    the few-variant path (one launch per step) with that many variants per workgroup."""
    import torch
    dev = di.tensors["dur"].device
    g = load_graph(di, stream)
    res = []
    handles = []
    try:
        for bi, (v0, v1, mask, scale, rm, eon) in enumerate(di.batches):
            Vb = v1 - v0
            sch, _ = B.dd_levelize(g, mask, mode, stream)
            var = B.dd_apply_transforms(g, Vb, di.n_cls, scale, rm, eon, stream)
            if outputs is not None:
                fin, st, ms = outputs[bi]
            else:
                fin = torch.empty((di.n, Vb), dtype=torch.int64, device=dev)
                st = torch.empty((di.n, Vb), dtype=torch.int64, device=dev) if want_start else None
                ms = torch.empty((Vb,), dtype=torch.int64, device=dev)
            if variants_per_wg:
                B.dd_simulate_batch_vs(g, sch, var, fin, st, ms, variants_per_wg, stream)
            else:
                B.dd_simulate_batch(g, sch, var, fin, st, ms, stream)
            res.append((v0, v1, fin, st, ms))
            handles.append((sch, var))
    finally:
        if not keep_handles:
            for sch, var in handles:
                B.dd_sched_free(sch)
                B.dd_variants_free(var)
            B.dd_graph_free(g)
    if keep_handles:
        return res, g, handles
    return res


def simulate_policy(g, vs, policy, pp=None, prio=None, shared=True, want_start=False,
                    stream=None, device="cuda"):
    """All variants under a schedule rule (dd_simulate_policy): the graph is
    loaded with DD_LOAD_SHARED_THREADS when `shared`, the full variant table
    goes in one handle.  Returns (finish[N][V], start or None, makespan[V])."""
    import torch

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)
    gl = B.dd_graph_load_ex(g.n, g.n_threads, t(g.in_ptr.astype(np.int64)),
                            t(g.in_src.astype(np.int32)), t(g.edge_cls.astype(np.uint8)),
                            t(g.thread_prev.astype(np.int32)), t(g.thread_id.astype(np.int32)),
                            t(g.dur.astype(np.int64)), t(g.gap.astype(np.int64)),
                            t(g.node_cls.astype(np.uint16)),
                            B.DD_LOAD_SHARED_THREADS if shared else 0, stream)
    var = None
    try:
        V = vs.n_variants
        var = B.dd_apply_transforms(gl, V, int(vs.scale.shape[0]), t(vs.scale.astype(np.int32)),
                                    t(vs.remove_bits.astype(np.uint32)),
                                    t(vs.edge_on[:, 0].astype(np.uint64)), stream)
        fin = torch.empty((g.n, V), dtype=torch.int64, device=device)
        st = torch.empty((g.n, V), dtype=torch.int64, device=device) if want_start else None
        ms = torch.empty((V,), dtype=torch.int64, device=device)
        B.dd_simulate_policy(gl, var, policy,
                             None if pp is None else t(np.asarray(pp, np.uint8)),
                             None if prio is None else t(np.asarray(prio, np.int32)),
                             fin, st, ms, stream)
    finally:
        if var is not None:
            B.dd_variants_free(var)
        B.dd_graph_free(gl)
    return fin, st, ms
