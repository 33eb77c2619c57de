"""The oracle: TEST INFRASTRUCTURE ONLY.

ctypes wrapper over dd_oracle.c, a plain CPU implementation of the paper's
simulation algorithm (Sec. 4.1, Algorithm 1) applied per variant after the
shrink/scale and Remove transformations (Sec. 4.4).  Only tests/, the smoke
check and the benchmark's CPU-baseline leg may import this module.  It
shares no code with the GPU path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dd_oracle.c")
_LIB = os.path.join(_HERE, "_build", "libdd_oracle.so")

OK, EINVAL, ECYCLE, ENOMEM = 0, 1, 2, 5


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C, -O2, pthreads)."""
    if force or not os.path.exists(_LIB):
        os.makedirs(os.path.dirname(_LIB), exist_ok=True)
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Graph(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("n_threads", ctypes.c_int32),
                ("in_ptr", ctypes.c_void_p), ("in_src", ctypes.c_void_p),
                ("edge_cls", ctypes.c_void_p), ("thread_prev", ctypes.c_void_p),
                ("thread_id", ctypes.c_void_p), ("dur", ctypes.c_void_p),
                ("gap", ctypes.c_void_p), ("node_cls", ctypes.c_void_p)]


class _Variants(ctypes.Structure):
    _fields_ = [("n_variants", ctypes.c_int32), ("n_cls", ctypes.c_int32),
                ("scale", ctypes.c_void_p), ("rm_bits", ctypes.c_void_p),
                ("edge_words", ctypes.c_int32), ("edge_on", ctypes.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
        _lib.ddo_run.restype = ctypes.c_int
        _lib.ddo_run.argtypes = [ctypes.POINTER(_Graph), ctypes.POINTER(_Variants),
                                 ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                 ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]
        _lib.ddo_breakdown.restype = ctypes.c_int
        _lib.ddo_breakdown.argtypes = [ctypes.POINTER(_Graph), ctypes.POINTER(_Variants),
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]
        _lib.ddo_run_policy.restype = ctypes.c_int
        _lib.ddo_run_policy.argtypes = [ctypes.POINTER(_Graph), ctypes.POINTER(_Variants),
                                        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]
        _lib.ddo_steps.restype = ctypes.c_int
        _lib.ddo_steps.argtypes = [ctypes.POINTER(_Graph), ctypes.c_uint64, ctypes.c_void_p,
                                   ctypes.c_void_p]
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__("oracle status %d" % code)
        self.code = code


def _graph_struct(g):
    arrs = dict(in_ptr=np.ascontiguousarray(g.in_ptr, np.int64),
                in_src=np.ascontiguousarray(g.in_src, np.int32),
                edge_cls=np.ascontiguousarray(g.edge_cls, np.uint8),
                thread_prev=np.ascontiguousarray(g.thread_prev, np.int32),
                thread_id=np.ascontiguousarray(g.thread_id, np.int32),
                dur=np.ascontiguousarray(g.dur, np.int64),
                gap=np.ascontiguousarray(g.gap, np.int64),
                node_cls=np.ascontiguousarray(g.node_cls, np.uint16))
    gs = _Graph(int(g.n), int(g.n_threads), *[_p(arrs[k]) for k in
                ("in_ptr", "in_src", "edge_cls", "thread_prev", "thread_id", "dur", "gap",
                 "node_cls")])
    return gs, arrs


def steps(g, mask: int = (1 << 64) - 1):
    """Kahn levels and phases of every task (edge classes in `mask`)."""
    lib = _load()
    gs, keep = _graph_struct(g)
    level = np.zeros(max(g.n, 1), np.int32)
    phase = np.zeros(max(g.n, 1), np.int32)
    rc = lib.ddo_steps(ctypes.byref(gs), ctypes.c_uint64(mask & (2 ** 64 - 1)), _p(level),
                       _p(phase))
    if rc != OK:
        raise OracleError(rc)
    return level[:g.n], phase[:g.n]


def run(g, vs, variants: Optional[Sequence[int]] = None, mode: int = 0, tie: int = 0,
        want_start: bool = True, want_finish: bool = True, workers: Optional[int] = None):
    """Simulate the listed variants (default: all).

    Returns (start, finish, makespan, bindings): start/finish int64
    [len(variants)][N] (or None), makespan and bindings int64 [len(variants)].
    mode 0: removed tasks kept with zero duration and gap; mode 1: unlinked.
    tie: 0/1/2 = rule schedule() uses among equal starts.
    """
    lib = _load()
    arrs = dict(in_ptr=np.ascontiguousarray(g.in_ptr, np.int64),
                in_src=np.ascontiguousarray(g.in_src, np.int32),
                edge_cls=np.ascontiguousarray(g.edge_cls, np.uint8),
                thread_prev=np.ascontiguousarray(g.thread_prev, np.int32),
                thread_id=np.ascontiguousarray(g.thread_id, np.int32),
                dur=np.ascontiguousarray(g.dur, np.int64),
                gap=np.ascontiguousarray(g.gap, np.int64),
                node_cls=np.ascontiguousarray(g.node_cls, np.uint16))
    gs = _Graph(int(g.n), int(g.n_threads), *[_p(arrs[k]) for k in
                ("in_ptr", "in_src", "edge_cls", "thread_prev", "thread_id", "dur", "gap",
                 "node_cls")])
    scale = np.ascontiguousarray(vs.scale, np.int32)
    rb = np.ascontiguousarray(vs.remove_bits, np.uint32)
    eo = np.ascontiguousarray(vs.edge_on, np.uint64)
    vv = _Variants(int(vs.n_variants), int(scale.shape[0]), _p(scale), _p(rb),
                   int(eo.shape[1]), _p(eo))
    if variants is None:
        variants = range(vs.n_variants)
    vl = np.ascontiguousarray(np.array(list(variants), np.int32))
    L = vl.shape[0]
    start = np.zeros((L, g.n), np.int64) if want_start else None
    finish = np.zeros((L, g.n), np.int64) if want_finish else None
    ms = np.zeros(L, np.int64)
    nb = np.zeros(L, np.int64)
    if workers is None:
        workers = max(1, min(len(os.sched_getaffinity(0)), 16))
    rc = lib.ddo_run(ctypes.byref(gs), ctypes.byref(vv), _p(vl), L, mode, tie,
                     _p(start), _p(finish), _p(ms), _p(nb), int(workers))
    if rc != OK:
        raise OracleError(rc)
    return start, finish, ms, nb


def breakdown(g, vs, role, variants: Optional[Sequence[int]] = None,
              workers: Optional[int] = None):
    """Runtime breakdown (Sec. 6.2, Fig. 6) of the listed variants from the
    oracle's own simulation: int64 [len(variants)][4] = total, CPU-only,
    GPU-only, CPU+GPU parallel.  role: uint8 [N], 1 = GPU kernel, 2 = CPU call
    that waits for the GPU (synchronization, device-to-host copy), 0 = other."""
    lib = _load()
    gs, keep = _graph_struct(g)
    scale = np.ascontiguousarray(vs.scale, np.int32)
    rb = np.ascontiguousarray(vs.remove_bits, np.uint32)
    eo = np.ascontiguousarray(vs.edge_on, np.uint64)
    vv = _Variants(int(vs.n_variants), int(scale.shape[0]), _p(scale), _p(rb),
                   int(eo.shape[1]), _p(eo))
    if variants is None:
        variants = range(vs.n_variants)
    vl = np.ascontiguousarray(np.array(list(variants), np.int32))
    rl = np.ascontiguousarray(role, np.uint8)
    L = vl.shape[0]
    ms = np.zeros(L, np.int64)
    out = np.zeros((L, 4), np.int64)
    if workers is None:
        workers = max(1, min(len(os.sched_getaffinity(0)), 16))
    rc = lib.ddo_breakdown(ctypes.byref(gs), ctypes.byref(vv), _p(rl), _p(vl), L, _p(ms),
                           _p(out), int(workers))
    if rc != OK:
        raise OracleError(rc)
    return out


POLICY_EARLIEST, POLICY_PRIORITY = 0, 1


def run_policy(g, vs, policy: int, pp=None, prio=None, variants: Optional[Sequence[int]] = None,
               want_start: bool = True, want_finish: bool = True,
               workers: Optional[int] = None):
    """Simulate the listed variants with an overridden schedule() (Sec. 4.4,
    "Schedule"); threads may hold several chains.  policy 0: earliest time
    max(P[t], start), first in trace order among equals; policy 1: P3's
    priority rule over push/pull tasks (pp[u] != 0) with priority prio[u].
    Returns (start, finish, makespan) like run()."""
    lib = _load()
    gs, keep = _graph_struct(g)
    scale = np.ascontiguousarray(vs.scale, np.int32)
    rb = np.ascontiguousarray(vs.remove_bits, np.uint32)
    eo = np.ascontiguousarray(vs.edge_on, np.uint64)
    vv = _Variants(int(vs.n_variants), int(scale.shape[0]), _p(scale), _p(rb),
                   int(eo.shape[1]), _p(eo))
    if variants is None:
        variants = range(vs.n_variants)
    vl = np.ascontiguousarray(np.array(list(variants), np.int32))
    L = vl.shape[0]
    ppa = None if pp is None else np.ascontiguousarray(pp, np.uint8)
    pra = None if prio is None else np.ascontiguousarray(prio, np.int32)
    start = np.zeros((L, g.n), np.int64) if want_start else None
    finish = np.zeros((L, g.n), np.int64) if want_finish else None
    ms = np.zeros(L, np.int64)
    if workers is None:
        workers = max(1, min(len(os.sched_getaffinity(0)), 16))
    rc = lib.ddo_run_policy(ctypes.byref(gs), ctypes.byref(vv), _p(vl), L, int(policy),
                            _p(ppa), _p(pra), _p(start), _p(finish), _p(ms), int(workers))
    if rc != OK:
        raise OracleError(rc)
    return start, finish, ms
