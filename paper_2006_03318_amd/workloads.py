"""Seeded synthetic trace-shaped task graphs and variant tables.

This module only *describes* inputs: tasks (CPU launch / sync tasks, GPU
kernels, memcpys, communication tasks), the execution thread of each task
and its order on that thread, dependency edges, integer-nanosecond durations
and gaps, and per-variant transform tables (rational duration scales,
removal bits, active edge classes).  It contains no simulation arithmetic:
no start, finish or release time is ever computed here.  Both the oracle
and the GPU path read the same objects.

Shapes follow the paper's description of training traces: one or two CPU
threads issuing every kernel through a launch call, one main compute stream,
a memcpy stream, an optional auxiliary stream joined through events, and a
communication channel for gradient all-reduces (Sec. 3 ("Key Ideas"),
Sec. 4.2.1 task types, Sec. 4.2.2 dependency types).  Durations follow the
recipe stated in the design notes: kernels lognormal(median, sigma=1),
CPU launch calls U[5,15] us, CPU gaps U[0,3] us, device and communication
gaps 0, all int64 ns.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# task kinds (metadata only; the simulation sees threads, edges, classes)
K_LAUNCH, K_SYNC, K_GEMM, K_ELEM, K_AUX, K_WU, K_MEMCPY, K_COMM, K_CONV, \
    K_GPU_OTHER, K_OPT, K_EMB = range(12)
# operator tags of CNN kernels (the layer types the batchnorm recipe selects)
# and of the copies a memory-offloading recipe inserts
OP_NONE, OP_CONV, OP_BN, OP_RELU, OP_OTHER, OP_OFFLOAD, OP_PREFETCH = range(7)
N_KINDS = 12          # kinds the synthetic generators emit (the class numbering uses it)
GPU_KINDS = (K_GEMM, K_ELEM, K_AUX, K_WU, K_CONV, K_GPU_OTHER, K_OPT, K_EMB)
CPU_KINDS = (K_LAUNCH, K_SYNC)
K_API = 12            # a traced runtime call that neither issues nor waits for device work

SEED_BASE = 2006033180


@dataclasses.dataclass
class TaskGraph:
    """A dependency graph G(V, E) in the layout the C-ABI accepts.

    in_ptr/in_src/edge_cls: CSR of dependency in-edges (src -> dst).
    thread_prev: previous task on the same execution thread (-1 = first).
    thread_id: execution thread of each task.
    dur, gap: int64 ns.  node_cls: transform class of each task.
    """
    n: int
    n_threads: int
    in_ptr: np.ndarray
    in_src: np.ndarray
    edge_cls: np.ndarray
    thread_prev: np.ndarray
    thread_id: np.ndarray
    dur: np.ndarray
    gap: np.ndarray
    node_cls: np.ndarray
    n_node_cls: int
    n_edge_cls: int
    kind: np.ndarray
    layer: np.ndarray
    launch_of: np.ndarray          # for device tasks: the CPU call that issued it, else -1
    name: str = ""
    op: Optional[np.ndarray] = None         # operator tag of GPU kernels (OP_*), 0 = none
    iteration: Optional[np.ndarray] = None  # training iteration of each task

    @property
    def n_edges(self) -> int:
        return int(self.in_ptr[-1])

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.in_ptr, self.in_src, self.edge_cls, self.thread_prev,
                  self.thread_id, self.dur, self.gap, self.node_cls):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()[:16]


@dataclasses.dataclass
class VariantSet:
    """Per-variant transform tables.

    scale: int32 [n_cls][V][2] = (p, q): duration of a task of class c in
      variant v becomes floor(d * p / q).
    remove_bits: uint32 [N][ceil(V/32)]; bit (v % 32) of word v // 32 set
      means the task is removed in variant v.
    edge_on: uint64 [V][ceil(K/64)]; bit k set means edges of class k are
      present in variant v.
    batches: list of (v0, v1, active_class_mask): variant ranges that share
      one levelization (their active edge classes have an acyclic union).
    """
    n_variants: int
    scale: np.ndarray
    remove_bits: np.ndarray
    edge_on: np.ndarray
    batches: List[Tuple[int, int, int]]

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.scale, self.remove_bits, self.edge_on):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()[:16]

    def subset(self, v0: int, v1: int) -> "VariantSet":
        """Variants [v0, v1) as their own set (bit columns re-packed)."""
        V = v1 - v0
        W = (V + 31) // 32
        bits = unpack_bits(self.remove_bits, self.n_variants)[:, v0:v1]
        rb = pack_bits(bits)
        assert rb.shape[1] == W
        return VariantSet(V, np.ascontiguousarray(self.scale[:, v0:v1]), rb,
                          np.ascontiguousarray(self.edge_on[v0:v1]),
                          [(0, V, self.batches[0][2])])


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """bool [N][V] -> uint32 [N][ceil(V/32)], bit v%32 of word v//32."""
    N, V = bits.shape
    W = (V + 31) // 32
    padded = np.zeros((N, W * 32), dtype=np.uint8)
    padded[:, :V] = bits
    b8 = np.packbits(padded, axis=1, bitorder="little")
    return np.ascontiguousarray(b8).view("<u4").reshape(N, W).astype(np.uint32)


def unpack_bits(words: np.ndarray, V: int) -> np.ndarray:
    N = words.shape[0]
    b8 = np.ascontiguousarray(words.astype("<u4")).view(np.uint8).reshape(N, -1)
    return np.unpackbits(b8, axis=1, bitorder="little")[:, :V].astype(bool)


# ---------------------------------------------------------------------------
class _Builder:
    """Emits tasks in trace (program) order.  Node ids are emission order."""

    def __init__(self, n_threads: int):
        self.n_threads = n_threads
        self.thread: List[int] = []
        self.kind: List[int] = []
        self.layer: List[int] = []
        self.launch_of: List[int] = []
        self.cls_override: List[int] = []
        self.op: List[int] = []
        self.edges: List[Tuple[int, int, int]] = []
        self.last: dict = {}

    def task(self, thread: int, kind: int, layer: int, launch_of: int = -1,
             cls_override: int = -1, op: int = OP_NONE) -> int:
        i = len(self.thread)
        self.thread.append(thread)
        self.kind.append(kind)
        self.layer.append(layer)
        self.launch_of.append(launch_of)
        self.cls_override.append(cls_override)
        self.op.append(op)
        self.last[thread] = i
        return i

    def edge(self, src: int, dst: int, ecls: int = 0):
        self.edges.append((src, dst, ecls))

    def launch(self, cpu: int, stream: int, kind: int, layer: int,
               cls_override: int = -1, op: int = OP_NONE) -> Tuple[int, int]:
        """A CPU launch call followed by the device task it issues
        (correlation dependency, Sec. 4.2.2)."""
        l = self.task(cpu, K_LAUNCH, layer)
        k = self.task(stream, kind, layer, launch_of=l, cls_override=cls_override, op=op)
        self.edge(l, k)
        return l, k

    def sync(self, cpu: int, streams, layer: int) -> int:
        """CPU synchronization call: waits for the last task on each stream."""
        srcs = [self.last[s] for s in streams if s in self.last]
        t = self.task(cpu, K_SYNC, layer)
        for s in srcs:
            self.edge(s, t)
        return t


@dataclasses.dataclass
class _Template:
    thread: np.ndarray
    kind: np.ndarray
    layer: np.ndarray
    launch_of: np.ndarray
    cls_override: np.ndarray
    op: np.ndarray
    esrc: np.ndarray
    edst: np.ndarray
    ecls: np.ndarray
    n_threads: int
    n_layers: int


def _template(b: _Builder, n_layers: int) -> _Template:
    e = np.array(b.edges, dtype=np.int64).reshape(-1, 3)
    return _Template(np.array(b.thread, np.int32), np.array(b.kind, np.uint8),
                     np.array(b.layer, np.int32), np.array(b.launch_of, np.int64),
                     np.array(b.cls_override, np.int32), np.array(b.op, np.uint8),
                     e[:, 0], e[:, 1], e[:, 2].astype(np.uint8), b.n_threads, n_layers)


_KERNEL_MEDIAN_NS = {K_GEMM: 400_000, K_ELEM: 20_000, K_AUX: 20_000, K_WU: 20_000,
                     K_CONV: 50_000, K_GPU_OTHER: 50_000, K_OPT: 50_000, K_EMB: 30_000}


def _durations(rng, kind: np.ndarray, medians: dict, memcpy_range, comm_ns=None):
    n = kind.shape[0]
    dur = np.zeros(n, np.int64)
    gap = np.zeros(n, np.int64)
    cpu = np.isin(kind, CPU_KINDS)
    dur[cpu] = rng.integers(5_000, 15_001, size=int(cpu.sum()))
    gap[cpu] = rng.integers(0, 3_001, size=int(cpu.sum()))
    for k, med in medians.items():
        m = kind == k
        c = int(m.sum())
        if c:
            z = rng.standard_normal(c)
            dur[m] = np.maximum(1, np.rint(med * np.exp(1.0 * z))).astype(np.int64)
    m = kind == K_MEMCPY
    if m.any():
        dur[m] = rng.integers(memcpy_range[0], memcpy_range[1] + 1, size=int(m.sum()))
    if comm_ns is not None:
        m = kind == K_COMM
        dur[m] = comm_ns
    return dur, gap


def _tile(t: _Template, iters: int, rng, medians, memcpy_range, name: str,
          comm_ns=None) -> TaskGraph:
    """Chain `iters` copies of one iteration: thread order continues across
    iterations; dependency edges stay inside an iteration."""
    n1 = t.thread.shape[0]
    N = n1 * iters
    thread = np.tile(t.thread, iters)
    kind = np.tile(t.kind, iters)
    layer = np.tile(t.layer, iters)
    off = (np.arange(iters, dtype=np.int64) * n1)
    lo = np.where(t.launch_of[None, :] >= 0, t.launch_of[None, :] + off[:, None], -1).reshape(-1)
    # thread order: previous task on the same thread, across iteration borders
    prev = np.full(N, -1, np.int32)
    order = np.argsort(thread, kind="stable")
    th_sorted = thread[order]
    same = th_sorted[1:] == th_sorted[:-1]
    prev[order[1:][same]] = order[:-1][same].astype(np.int32)
    # edges
    esrc = (t.esrc[None, :] + off[:, None]).reshape(-1)
    edst = (t.edst[None, :] + off[:, None]).reshape(-1)
    ecls = np.tile(t.ecls, iters)
    ordr = np.argsort(edst, kind="stable")
    esrc, edst, ecls = esrc[ordr], edst[ordr], ecls[ordr]
    in_ptr = np.zeros(N + 1, np.int64)
    np.add.at(in_ptr, edst + 1, 1)
    in_ptr = np.cumsum(in_ptr)
    dur, gap = _durations(rng, kind, medians, memcpy_range, None)
    if comm_ns is not None:
        m = kind == K_COMM
        dur[m] = np.tile(comm_ns, iters)
    L1 = t.n_layers + 1
    node_cls = (np.where(layer >= 0, layer, t.n_layers) * N_KINDS + kind).astype(np.int64)
    co = np.tile(t.cls_override, iters)
    node_cls = np.where(co >= 0, L1 * N_KINDS + co, node_cls)
    n_cls = int(L1 * N_KINDS + max(0, int(t.cls_override.max()) + 1))
    return TaskGraph(N, t.n_threads, in_ptr, esrc.astype(np.int32), ecls.astype(np.uint8),
                     prev, thread.astype(np.int32), dur, gap, node_cls.astype(np.uint16),
                     n_cls, int(ecls.max()) + 1 if ecls.size else 1, kind, layer, lo, name,
                     op=np.tile(t.op, iters),
                     iteration=np.repeat(np.arange(iters, dtype=np.int32), n1))


# ---------------------------------------------------------------------------
# workload structures
CPU, S0, MEMCPY_S, AUX_S = 0, 1, 2, 3


def _cnn_iteration(n_layers=20) -> _Template:
    """Small CNN: per layer 3 fwd + 6 bwd kernels (1 fwd + 2 bwd conv-like)
    and 1 optimizer kernel, each issued by a CPU launch; one H2D memcpy at
    the start; one end-of-iteration synchronization."""
    b = _Builder(3)
    _, mc = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)
    first = True
    fwd_ops = (OP_CONV, OP_BN, OP_RELU)
    bwd_ops = (OP_CONV, OP_CONV, OP_RELU, OP_BN, OP_OTHER, OP_OTHER)   # data and weight grads first
    for l in range(n_layers):
        for j in range(3):
            _, k = b.launch(CPU, S0, K_CONV if j == 0 else K_GPU_OTHER, l, op=fwd_ops[j])
            if first:
                b.edge(mc, k)   # input batch must arrive before the first kernel
                first = False
    for l in reversed(range(n_layers)):
        for j in range(6):
            b.launch(CPU, S0, K_CONV if bwd_ops[j] == OP_CONV else K_GPU_OTHER, l, op=bwd_ops[j])
    for l in range(n_layers):
        b.launch(CPU, S0, K_OPT, l)
    b.sync(CPU, [S0, MEMCPY_S], -1)
    return _template(b, n_layers)


def _transformer_iteration(n_layers=24, n_wu=554, comm=False, bucket_bytes=25 << 20,
                           layer_grad_bytes=None):
    """Transformer encoder iteration (BERT-like, as in the evaluation of Sec. 6.1): per layer
    40 fwd kernels (8 GEMM-like) with one fork/join group of 8 aux-stream
    kernels joined back through events, 80 bwd kernels (16 GEMM-like) and
    n_wu element-wise weight-update kernels.  With comm=True, one all-reduce
    per gradient bucket is issued on its own channel after the last backward
    kernel of its bucket; the first weight-update kernel waits for all of
    them (Sec. 4.2.1 communication tasks)."""
    b = _Builder(4)
    _, mc = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)
    ks = []
    for j in range(5):
        _, k = b.launch(CPU, S0, K_EMB, -1)
        if j == 0:
            b.edge(mc, k)
    fwd = {}
    for l in range(n_layers):
        fwd[l] = []
        for j in range(40):
            kind = K_GEMM if j % 5 == 0 else K_ELEM
            _, k = b.launch(CPU, S0, kind, l)
            fwd[l].append(k)
            if j == 19:                    # fork: aux stream waits on this kernel
                fork_src = k
                for a in range(8):
                    _, ka = b.launch(CPU, AUX_S, K_AUX, l)
                    if a == 0:
                        b.edge(fork_src, ka)
                join_src = ka
            if j == 29:                    # join: this kernel waits on the aux group
                b.edge(join_src, k)
    for j in range(8):
        b.launch(CPU, S0, K_EMB, -1)       # loss
    _, dl = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)   # D2H loss copy
    b.sync(CPU, [MEMCPY_S], -1)
    last_bwd = {}
    bwd = {}
    for l in reversed(range(n_layers)):
        bwd[l] = []
        for j in range(80):
            kind = K_GEMM if j % 5 == 0 else K_ELEM
            _, k = b.launch(CPU, S0, kind, l)
            b.edge(fwd[l][j % 40], k)       # saved activation (same stream: dominated)
            bwd[l].append(k)
        last_bwd[l] = k
    comm_nodes = []
    if comm:
        # gradient buckets: the byte stream of layer gradients in backward
        # order cut every bucket_bytes (PyTorch DDP grouping); a bucket's
        # all-reduce follows the last backward kernel among its layers
        lg = layer_grad_bytes
        total = n_layers * lg
        buckets = []
        for i in range((total + bucket_bytes - 1) // bucket_bytes):
            hi = min((i + 1) * bucket_bytes, total)
            r_last = (hi - 1) // lg                 # backward position of the last member
            buckets.append((n_layers - 1 - r_last, hi - i * bucket_bytes))
        for bi, (lay, nbytes) in enumerate(buckets):
            ar = b.task(4 + bi, K_COMM, -1, cls_override=bi)
            b.edge(last_bwd[lay], ar)
            comm_nodes.append((ar, nbytes))
        b.n_threads = 4 + len(buckets)
    first_wu = None
    for l in range(n_layers):
        for j in range(n_wu):
            _, k = b.launch(CPU, S0, K_WU, l)
            if first_wu is None:
                first_wu = k
                for ar, _ in comm_nodes:
                    b.edge(ar, k)
            b.edge(bwd[l][j % 80], k)       # gradient producer (same stream: dominated)
    b.sync(CPU, [S0, AUX_S], -1)
    t = _template(b, n_layers)
    return t, comm_nodes


def _seq2seq_iteration(n_enc=8, n_dec=8, steps=50):
    """Recurrent seq2seq: encoder and decoder stacks unrolled over timesteps,
    6 small forward kernels per cell, 12 backward per cell, one optimizer
    kernel per layer, an H2D memcpy and an end-of-iteration sync."""
    b = _Builder(3)
    _, mc = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)
    L = n_enc + n_dec
    first = True
    for t_ in range(steps):
        for l in range(L):
            for j in range(6):
                _, k = b.launch(CPU, S0, K_ELEM if j % 3 else K_GEMM, l)
                if first:
                    b.edge(mc, k)
                    first = False
    for t_ in reversed(range(steps)):
        for l in reversed(range(L)):
            for j in range(12):
                b.launch(CPU, S0, K_ELEM if j % 3 else K_GEMM, l)
    for l in range(L):
        b.launch(CPU, S0, K_OPT, l)
    b.sync(CPU, [S0, MEMCPY_S], -1)
    return _template(b, L)


# ---------------------------------------------------------------------------
# variant tables
def _identity_scale(C: int, V: int) -> np.ndarray:
    s = np.ones((C, V, 2), np.int32)
    return s


def _cls_of(layer: int, kind: int, n_layers: int) -> int:
    return (layer if layer >= 0 else n_layers) * N_KINDS + kind


def _removal_bits(rng, N: int, V: int, kernels: np.ndarray, launches: np.ndarray,
                  density: np.ndarray, chunk: int = 1 << 15) -> np.ndarray:
    """Bernoulli(density[v]) removal of each removable kernel together with
    its launch call, packed [N][ceil(V/32)]."""
    W = (V + 31) // 32
    out = np.zeros((N, W), np.uint32)
    thr = np.minimum(np.rint(density * 65536.0), 65536).astype(np.uint32)
    for s in range(0, kernels.shape[0], chunk):
        kk = kernels[s:s + chunk]
        u = rng.integers(0, 65536, size=(kk.shape[0], V), dtype=np.uint16)
        words = pack_bits(u.astype(np.uint32) < thr[None, :])
        out[kk] = words
        ll = launches[s:s + chunk]
        ok = ll >= 0
        out[ll[ok]] = words[ok]
    return out


def _random_pq(rng, qs, pmax_factor=2, pmin=0):
    q = int(rng.choice(qs))
    p = int(rng.integers(pmin, pmax_factor * q + 1))
    return p, q


# ---------------------------------------------------------------------------
def config(k: int, seed: Optional[int] = None, variants: Optional[int] = None,
           iters: Optional[int] = None) -> Tuple[TaskGraph, VariantSet]:
    """The five workloads.  `variants`/`iters` shrink a workload for tests."""
    rng = np.random.default_rng(SEED_BASE + k if seed is None else seed)
    if k == 1:
        t = _cnn_iteration()
        g = _tile(t, iters or 4, rng, _KERNEL_MEDIAN_NS, (500_000, 2_000_000), "cnn")
        V = variants or 8
        g, vs = _cnn_recipes(rng, g, t.n_layers, V)
    elif k in (2, 5):
        t, _ = _transformer_iteration()
        it = iters or (1 if k == 2 else 32)
        g = _tile(t, it, rng, _KERNEL_MEDIAN_NS, (100_000, 400_000),
                  "transformer" if k == 2 else "transformer-x%d" % it)
        V = variants or (256 if k == 2 else 2048)
        if k == 2:
            g, vs = _transformer_recipes(rng, g, t.n_layers, V)
        else:
            vs = _transformer_variants(rng, g, t.n_layers, V, qs=(1, 2, 4, 8))
    elif k == 3:
        hidden = 1024
        layer_grad = 12 * hidden * hidden * 4 + 13 * hidden * 4   # fp32 grads per layer
        t, comm = _transformer_iteration(comm=True, layer_grad_bytes=layer_grad)
        # base all-reduce duration: bytes at 10 GB/s (1 GB/s = 1 byte/ns)
        comm_ns = np.array([nb // 10 for _, nb in comm], np.int64)
        g = _tile(t, iters or 1, rng, _KERNEL_MEDIAN_NS, (100_000, 400_000),
                  "transformer+allreduce", comm_ns=comm_ns)
        V = variants or 1024
        # order edges between all-reduce channels live in classes 1..4
        g, vs = _comm_recipes(rng, g, t, [ar for ar, _ in comm], V)
    elif k == 4:
        t = _seq2seq_iteration()
        g = _tile(t, iters or 9, rng, {K_GEMM: 15_000, K_ELEM: 15_000, K_OPT: 15_000},
                  (100_000, 400_000), "seq2seq")
        V = variants or 64
        g, vs = _seq2seq_recipes(rng, g, t.n_layers, V)
    else:
        raise ValueError("config must be 1..5")
    return g, vs


# ---------------------------------------------------------------------------
# variant sweeps written as what-if recipes (recipes.py)
def _cnn_recipes(rng, g: TaskGraph, L: int, V: int):
    """CNN sweep: baseline, AMP, restructured batchnorm, both, free launch
    calls, a 2x faster GPU, and layer substitutions (scale or remove)."""
    from . import recipes as R
    sweep = []
    for v in range(V):
        kind = v % 8
        if kind == 0:
            r = []
        elif kind == 1:
            r = [R.AMP()]
        elif kind == 2:
            r = [R.RestructureBatchnorm()]
        elif kind == 3:
            r = [R.AMP(), R.RestructureBatchnorm()]
        elif kind == 4:
            r = [R.ScaleLaunch(0, 1)]
        elif kind == 5:
            r = [R.ScaleKernels(1, 2)]
        elif kind == 6:
            layers = [l for l in range(L) if rng.random() < 0.5]
            p, q = _random_pq(rng, (2, 4, 8), 2, 1)
            r = [R.ScaleLayers(layers, p, q)]
        else:
            layers = [int(x) for x in rng.choice(L, size=2, replace=False)]
            r = [R.RemoveLayers(layers), R.AMP()]
        sweep.append(r)
    return R.compile_sweep(g, sweep)


def _transformer_recipes(rng, g: TaskGraph, L: int, V: int):
    """Transformer sweep: random combinations of element-wise kernel fusion,
    a fused optimizer, AMP and layer scaling (variant 0 is the baseline)."""
    from . import recipes as R
    sweep = [[]]
    for v in range(1, V):
        r = []
        fused_adam = rng.random() < 0.5
        if rng.random() < 0.7:
            kinds = (K_ELEM, K_AUX) if fused_adam else (K_ELEM, K_AUX, K_WU)
            r.append(R.FuseElementwise(float(rng.uniform(0.1, 0.5)), int(rng.integers(1 << 30)),
                                       kinds))
        if fused_adam:
            r.append(R.FusedAdam())
        if rng.random() < 0.5:
            r.append(R.AMP())
        if rng.random() < 0.5:
            layers = [l for l in range(L) if rng.random() < 0.5]
            p, q = _random_pq(rng, (1, 2, 3, 4, 8), 2, 0)
            r.append(R.ScaleLayers(layers, p, q))
        sweep.append(r)
    return R.compile_sweep(g, sweep)


def _comm_recipes(rng, g: TaskGraph, t: _Template, ars: List[int], V: int):
    """Data-parallel sweep: four orders of the all-reduce channel (edge
    classes 1..4) x link bandwidth 10, 25, 100 GB/s x gradient compression
    of random buckets, some with AMP."""
    from . import recipes as R
    g = _with_channel_orders(rng, g, t, ars)
    B = len(ars)
    per = V // 4
    sweep = []
    for gi in range(4):
        n_g = V - 3 * per if gi == 3 else per
        for j in range(n_g):
            r = [R.EdgeClasses(on=1 << (1 + gi)), R.Distributed([10, 25, 100][j % 3])]
            if j >= 3:
                r.append(R.CompressGradients(1, 4, [b for b in range(B) if rng.random() < 0.5]))
            if j >= 6 and rng.random() < 0.5:
                r.append(R.AMP())
            sweep.append(r)
    return R.compile_sweep(g, sweep, base_edge_mask=1)


def _seq2seq_recipes(rng, g: TaskGraph, L: int, V: int):
    """Seq2seq sweep: CPU launch cost x {1, 0, 1/4, 1/2, 2} with element-wise
    fusion of U[0.1, 0.5] of the kernels (variant 0 is the baseline)."""
    from . import recipes as R
    lscales = [(1, 1), (0, 1), (1, 4), (1, 2), (2, 1)]
    sweep = []
    for v in range(V):
        r = [R.ScaleLaunch(*lscales[v % 5])]
        if v:
            r.append(R.FuseElementwise(float(rng.uniform(0.1, 0.5)), int(rng.integers(1 << 30)),
                                       (K_ELEM,)))
        sweep.append(r)
    return R.compile_sweep(g, sweep)


def _removable(g: TaskGraph, kinds) -> Tuple[np.ndarray, np.ndarray]:
    k = np.nonzero(np.isin(g.kind, kinds))[0]
    return k.astype(np.int64), g.launch_of[k].astype(np.int64)


def _transformer_variants(rng, g: TaskGraph, L: int, V: int, qs) -> VariantSet:
    """Stress sweep of the large transformer workload: every (layer, kind)
    class draws its own ratio p/q (q in `qs`, p in [0, 2q]) with probability
    1/2 per variant, and each variant removes element-wise, auxiliary and
    weight-update kernels (with their launch calls) at a density drawn from
    U[0.1, 0.5].  Variant 0 is the baseline."""
    C = g.n_node_cls
    s = _identity_scale(C, V)
    kinds = (K_GEMM, K_ELEM, K_AUX, K_WU, K_LAUNCH)
    for v in range(1, V):
        for l in range(L):
            for kd in kinds:
                if rng.random() < 0.5:
                    s[_cls_of(l, kd, L), v] = _random_pq(rng, qs, 2, 0)
    dens = rng.uniform(0.1, 0.5, size=V)
    dens[0] = 0.0
    kern, lau = _removable(g, (K_ELEM, K_WU, K_AUX))
    rb = _removal_bits(rng, g.n, V, kern, lau, dens)
    eo = np.ones((V, 1), np.uint64)
    return VariantSet(V, s, rb, eo, [(0, V, 1)])


def _with_channel_orders(rng, g: TaskGraph, t: _Template, ars: List[int]) -> TaskGraph:
    """The all-reduce channel's four orders (ready order, reverse, interleaved
    priority, seeded permutation) as order edges of classes 1..4."""
    n1 = t.thread.shape[0]
    iters = g.n // n1
    B = len(ars)
    orders = [list(range(B)), list(reversed(range(B))),
              list(range(0, B, 2)) + list(range(1, B, 2)),      # interleaved priority
              [int(x) for x in rng.permutation(B)]]
    extra_src, extra_dst, extra_cls = [], [], []
    for it in range(iters):
        base = it * n1
        for gi, od in enumerate(orders):
            for a, bq in zip(od[:-1], od[1:]):
                extra_src.append(base + ars[a])
                extra_dst.append(base + ars[bq])
                extra_cls.append(1 + gi)
    # rebuild CSR with the extra edges
    dst_old = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.in_ptr))
    src = np.concatenate([g.in_src.astype(np.int64), np.array(extra_src, np.int64)])
    dst = np.concatenate([dst_old, np.array(extra_dst, np.int64)])
    cls = np.concatenate([g.edge_cls, np.array(extra_cls, np.uint8)])
    o = np.argsort(dst, kind="stable")
    src, dst, cls = src[o], dst[o], cls[o]
    in_ptr = np.zeros(g.n + 1, np.int64)
    np.add.at(in_ptr, dst + 1, 1)
    in_ptr = np.cumsum(in_ptr)
    return dataclasses.replace(g, in_ptr=in_ptr, in_src=src.astype(np.int32),
                               edge_cls=cls.astype(np.uint8), n_edge_cls=5)


# ---------------------------------------------------------------------------
# parameter-server training with sliced gradient pushes and pulls (the P3
# what-if of Sec. 5.1 and the appendix: every layer's gradient is cut into
# slices; each slice is pushed after the backward kernel that produced it and
# pulled back before the next iteration's forward kernel of that layer)
SEND, RECV = 3, 4


def vgg19_layer_params() -> Tuple[List[int], List[bool]]:
    """Parameter counts of VGG-19's 19 weight layers (16 3x3 convolutions,
    then three fully connected layers), from its layer shapes."""
    chans = [64, 64, 128, 128, 256, 256, 256, 256, 512, 512, 512, 512, 512, 512, 512, 512]
    params, fc = [], []
    cin = 3
    for c in chans:
        params.append(9 * cin * c + c)
        fc.append(False)
        cin = c
    for a, b in ((512 * 7 * 7, 4096), (4096, 4096), (4096, 1000)):
        params.append(a * b + b)
        fc.append(True)
    return params, fc


def _p3_iteration(params, fc, slice_bytes, servers):
    """One iteration: forward (a convolution or GEMM and an element-wise
    kernel per layer), loss, backward (data-gradient and weight-gradient
    kernels per layer, in reverse), and for every layer's gradient its
    slices: push on the send channel after the weight-gradient kernel, then
    pull (on the send channel for slices kept by the first server, on the
    receive channel otherwise).  Returns the template, the pull ids of each
    layer, the first forward kernel of each layer and the slice sizes."""
    L = len(params)
    b = _Builder(5)
    _, mc = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)
    ff_first = []
    for l in range(L):
        _, k = b.launch(CPU, S0, K_GEMM if fc[l] else K_CONV, l,
                        op=OP_OTHER if fc[l] else OP_CONV)
        if l == 0:
            b.edge(mc, k)
        ff_first.append(k)
        b.launch(CPU, S0, K_ELEM, l, op=OP_RELU)
    b.launch(CPU, S0, K_ELEM, -1)                                   # loss
    pulls = [[] for _ in range(L)]
    sizes = []
    n_slice = 0
    for l in reversed(range(L)):
        kind = K_GEMM if fc[l] else K_CONV
        b.launch(CPU, S0, kind, l, op=OP_OTHER if fc[l] else OP_CONV)   # data gradient
        _, u = b.launch(CPU, S0, kind, l, op=OP_OTHER if fc[l] else OP_CONV)   # weight gradient
        left = 4 * params[l]
        while left > 0:
            sz = min(left, slice_bytes)
            push = b.task(SEND, K_COMM, l)
            pull = b.task(SEND if n_slice % servers == 0 else RECV, K_COMM, l)
            b.edge(u, push)
            b.edge(push, pull)
            pulls[l].append(pull)
            sizes += [sz, sz]
            left -= sz
            n_slice += 1
    b.sync(CPU, [S0], -1)
    return _template(b, L), pulls, ff_first, np.array(sizes, np.int64)


def p3_workload(iters: int = 8, slice_bytes: int = 4 << 20, servers: int = 4, gbps: int = 10,
                variants: int = 1024, seed: Optional[int] = None):
    """VGG-19 data-parallel training on a parameter server with P3's sliced
    pushes and pulls: `iters` chained iterations; the two channels (threads
    SEND and RECV) hold the slices with no recorded order, so a schedule rule
    orders them.  Slice durations are bytes at `gbps` Gbit/s; kernels are
    lognormal (convolutions median 3 ms, GEMMs 1 ms, element-wise 0.3 ms).
    Variants (through the recipe compiler): link bandwidth 1-40 Gbit/s, with
    or without AMP, and some with cheaper launch calls.
    Returns (graph, variants, pp, prio): pp = 1 on push/pull tasks, prio =
    minus the layer index (layers nearer the input first)."""
    from . import recipes as R
    rng = np.random.default_rng(SEED_BASE + 6 if seed is None else seed)
    params, fc = vgg19_layer_params()
    t, pulls, ff_first, sizes = _p3_iteration(params, fc, slice_bytes, servers)
    comm_ns = sizes * 8 // gbps
    medians = {K_CONV: 3_000_000, K_GEMM: 1_000_000, K_ELEM: 300_000}
    g = _tile(t, iters, rng, medians, (1_000_000, 4_000_000), "vgg19-p3", comm_ns=comm_ns)
    n1 = t.thread.shape[0]
    # the channels keep no recorded order: every slice task is a chain of its own
    g.thread_prev[np.isin(g.thread_id, (SEND, RECV))] = -1
    ch = np.isin(g.thread_id, (SEND, RECV))
    nxt = np.full(g.n, -1, np.int64)
    has = g.thread_prev >= 0
    nxt[g.thread_prev[has]] = np.nonzero(has)[0]
    assert not ch[nxt[nxt >= 0]].any()
    # a layer's pulls come before the next iteration's forward kernel of it
    xs, xd = [], []
    for it in range(iters - 1):
        for l, pl in enumerate(pulls):
            for p_ in pl:
                xs.append(it * n1 + p_)
                xd.append((it + 1) * n1 + ff_first[l])
    dst_old = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.in_ptr))
    src = np.concatenate([g.in_src.astype(np.int64), np.array(xs, np.int64)])
    dst = np.concatenate([dst_old, np.array(xd, np.int64)])
    cls = np.concatenate([g.edge_cls, np.zeros(len(xs), np.uint8)])
    o = np.argsort(dst, kind="stable")
    in_ptr = np.zeros(g.n + 1, np.int64)
    np.add.at(in_ptr, dst + 1, 1)
    g = dataclasses.replace(g, in_ptr=np.cumsum(in_ptr), in_src=src[o].astype(np.int32),
                            edge_cls=cls[o].astype(np.uint8), n_threads=5)
    pp = (g.kind == K_COMM).astype(np.uint8)
    prio = np.where(g.kind == K_COMM, -g.layer, 0).astype(np.int32)
    sweep = []
    bws = (1, 2, 5, 10, 25, 40)
    for v in range(variants):
        r = [R.Distributed(bws[v % len(bws)], base_gbps=gbps)]
        if (v // len(bws)) % 2:
            r.append(R.AMP())
        if (v // (2 * len(bws))) % 2:
            r.append(R.ScaleLaunch(1, 2))
        if v >= 4 * len(bws) and rng.random() < 0.5:
            r.append(R.ScaleKernels(int(rng.integers(1, 4)), int(rng.integers(1, 4))))
        sweep.append(r)
    g, vs = R.compile_sweep(g, sweep)
    return g, vs, pp, prio


# ---------------------------------------------------------------------------
# memory offloading (vDNN, the appendix's model): each convolution's output is
# copied to the host after the layer's forward pass and copied back before
# its backward pass; when a copy back may start is the prefetch policy
def _vdnn_iteration(n_layers=20, max_dist=3):
    """One CNN iteration with vDNN's copies: after each layer's forward
    kernels an offload copy (device to host) of its convolution output on the
    copy stream; when the backward pass starts, one prefetch copy per layer
    in backward order, each needed by the first backward kernel of its
    layer.  Edge class d (1..max_dist) holds the prefetch policy "start the
    copy back of layer l once the backward pass of layer l + d has begun"
    (vDNN's choice of prefetch layer); with no class on, copies go back as
    early as the copy stream allows."""
    b = _Builder(3)
    _, mc = b.launch(CPU, MEMCPY_S, K_MEMCPY, -1)
    fwd_ops = (OP_CONV, OP_BN, OP_RELU)
    bwd_ops = (OP_CONV, OP_CONV, OP_RELU, OP_BN, OP_OTHER, OP_OTHER)
    first = True
    for l in range(n_layers):
        for j in range(3):
            _, k = b.launch(CPU, S0, K_CONV if j == 0 else K_GPU_OTHER, l, op=fwd_ops[j])
            if first:
                b.edge(mc, k)
                first = False
            if j == 0:
                conv = k
        _, off = b.launch(CPU, MEMCPY_S, K_MEMCPY, l, op=OP_OFFLOAD)
        b.edge(conv, off)                       # the feature map leaves once written
    pf = {}
    for l in reversed(range(n_layers)):
        _, pf[l] = b.launch(CPU, MEMCPY_S, K_MEMCPY, l, op=OP_PREFETCH)
    bwd_first = {}
    for l in reversed(range(n_layers)):
        for j in range(6):
            _, k = b.launch(CPU, S0, K_CONV if bwd_ops[j] == OP_CONV else K_GPU_OTHER, l,
                            op=bwd_ops[j])
            if j == 0:
                bwd_first[l] = k
                b.edge(pf[l], k)                # the layer's backward needs its input back
    for l in range(n_layers):
        for d in range(1, max_dist + 1):
            if l + d < n_layers:
                b.edge(bwd_first[l + d], pf[l], d)
    for l in range(n_layers):
        b.launch(CPU, S0, K_OPT, l)
    b.sync(CPU, [S0, MEMCPY_S], -1)
    return _template(b, n_layers)


def vdnn_workload(iters: int = 4, variants: int = 256, seed: Optional[int] = None):
    """A 20-layer CNN trained with vDNN's offloading of convolution outputs
    (the appendix's vDNN model), `iters` chained iterations.  Kernels are
    lognormal (convolutions median 500 us, other kernels 100 us, optimizer
    50 us); each copy takes U[100, 600] us (feature map over PCIe).
    Variants (through the recipe compiler, one levelization for all: the
    union of the policy classes is acyclic): no offloading, copies back as
    early as possible, or prefetch 1, 2 or 3 layers ahead; PCIe 2x faster
    or slower; with or without AMP."""
    from . import recipes as R
    rng = np.random.default_rng(SEED_BASE + 7 if seed is None else seed)
    t = _vdnn_iteration()
    g = _tile(t, iters, rng, {K_CONV: 500_000, K_GPU_OTHER: 100_000, K_OPT: 50_000},
              (100_000, 600_000), "cnn-vdnn")
    sweep = []
    for v in range(variants):
        pol = v % 5                       # 0: no offloading, 1: eager, 2-4: distance 1-3
        r = [R.RemoveOffload()] if pol == 0 else (
            [] if pol == 1 else [R.EdgeClasses(on=1 << (pol - 1))])
        pcie = (v // 5) % 3
        if pcie == 1:
            r.append(R.ScaleCopies(1, 2))
        elif pcie == 2:
            r.append(R.ScaleCopies(2, 1))
        if (v // 15) % 2:
            r.append(R.AMP())
        sweep.append(r)
    return R.compile_sweep(g, sweep, one_batch_mask=0xF)


def task_roles(g: TaskGraph) -> np.ndarray:
    """Roles for the runtime breakdown: 1 = GPU kernel, 2 = CPU call that
    waits for GPU work (the synchronization tasks), 0 = anything else
    (launch calls, memory copies, communication)."""
    role = np.zeros(g.n, np.uint8)
    role[np.isin(g.kind, GPU_KINDS)] = 1
    role[g.kind == K_SYNC] = 2
    return role


# ---------------------------------------------------------------------------
def random_graph(rng, n: int, n_threads: int, p_edge: float = 0.3, max_dur: int = 20,
                 zero_frac: float = 0.2, n_edge_cls: int = 1,
                 same_thread_edges: bool = True) -> TaskGraph:
    """A small random DAG: tasks in id order (topological), random thread
    assignment, random forward dependency edges, durations incl. 0."""
    thread = rng.integers(0, n_threads, size=n).astype(np.int32)
    prev = np.full(n, -1, np.int32)
    last = {}
    for i in range(n):
        t = int(thread[i])
        if t in last:
            prev[i] = last[t]
        last[t] = i
    srcs, dsts, cls = [], [], []
    for j in range(n):
        for i in range(j):
            if rng.random() < p_edge and (same_thread_edges or thread[i] != thread[j]):
                srcs.append(i)
                dsts.append(j)
                cls.append(int(rng.integers(0, n_edge_cls)))
    in_ptr = np.zeros(n + 1, np.int64)
    for d in dsts:
        in_ptr[d + 1] += 1
    in_ptr = np.cumsum(in_ptr)
    dur = rng.integers(0, max_dur + 1, size=n).astype(np.int64)
    dur[rng.random(n) < zero_frac] = 0
    gap = rng.integers(0, max_dur // 2 + 1, size=n).astype(np.int64)
    gap[rng.random(n) < 0.5] = 0
    kind = np.zeros(n, np.uint8)
    return TaskGraph(n, n_threads, in_ptr, np.array(srcs, np.int32),
                     np.array(cls, np.uint8), prev, thread, dur, gap,
                     rng.integers(0, 3, size=n).astype(np.uint16), 3, n_edge_cls,
                     kind, np.full(n, -1, np.int32), np.full(n, -1, np.int64), "random")


def random_graph_sparse(rng, n: int, n_threads: int, mean_in: float = 0.3,
                        window: int = 64, n_edge_cls: int = 1, max_dur: int = 10**5,
                        n_node_cls: int = 3, run_len: int = 1) -> TaskGraph:
    """A larger random DAG built without a quadratic loop: task j gets
    Poisson(mean_in) dependency edges from tasks drawn uniformly in
    [j - window, j); tasks come in runs of `run_len` consecutive ids on one
    random thread.  Ids are topological; thread order is id order."""
    runs = (n + run_len - 1) // run_len
    thread = np.repeat(rng.integers(0, n_threads, size=runs), run_len)[:n].astype(np.int32)
    prev = np.full(n, -1, np.int32)
    last = np.full(n_threads, -1, np.int64)
    for i in range(n):           # O(n): previous task on the same thread
        t = thread[i]
        prev[i] = last[t]
        last[t] = i
    k = rng.poisson(mean_in, size=n).astype(np.int64)
    k[0] = 0
    dst = np.repeat(np.arange(n, dtype=np.int64), k)
    lo = np.maximum(dst - window, 0)
    src = lo + (rng.random(dst.shape[0]) * (dst - lo)).astype(np.int64)
    ok = src < dst
    src, dst = src[ok], dst[ok]
    in_ptr = np.zeros(n + 1, np.int64)
    np.add.at(in_ptr, dst + 1, 1)
    in_ptr = np.cumsum(in_ptr)
    dur = rng.integers(0, max_dur + 1, size=n).astype(np.int64)
    dur[rng.random(n) < 0.1] = 0
    gap = rng.integers(0, max_dur // 4 + 1, size=n).astype(np.int64)
    gap[rng.random(n) < 0.5] = 0
    cls = rng.integers(0, n_edge_cls, size=src.shape[0]).astype(np.uint8)
    return TaskGraph(n, n_threads, in_ptr, src.astype(np.int32), cls, prev, thread, dur, gap,
                     rng.integers(0, n_node_cls, size=n).astype(np.uint16), n_node_cls,
                     n_edge_cls, np.zeros(n, np.uint8), np.full(n, -1, np.int32),
                     np.full(n, -1, np.int64), "random-sparse")


def random_shared_graph(rng, n: int, n_ordered: int, n_shared: int, mean_in: float = 1.5,
                        window: int = 32, max_dur: int = 1000, zero_frac: float = 0.2,
                        n_edge_cls: int = 1, chain_frac: float = 0.3, n_node_cls: int = 3,
                        prio_range: int = 4):
    """A random DAG whose last `n_shared` threads hold tasks with no order
    among them (a schedule decides it), like the push/pull slices of a
    communication channel.  Tasks on the first `n_ordered` threads form one
    chain per thread (id order); a task on a shared thread starts a chain of
    its own, or with probability `chain_frac` continues the tail of one of
    that thread's chains.  Dependency edges: Poisson(mean_in) per task from
    the previous `window` ids.  Returns (graph, pp, prio): pp = 1 on tasks of
    shared threads (the push/pull tasks of the priority rule), prio drawn from
    [-prio_range, prio_range] so that equal priorities occur."""
    T = n_ordered + n_shared
    thread = rng.integers(0, T, size=n).astype(np.int32)
    prev = np.full(n, -1, np.int32)
    last = np.full(T, -1, np.int64)
    tails = [[] for _ in range(T)]
    for i in range(n):
        t = int(thread[i])
        if t < n_ordered:
            prev[i] = last[t]
            last[t] = i
        else:
            if tails[t] and rng.random() < chain_frac:
                k = int(rng.integers(0, len(tails[t])))
                prev[i] = tails[t][k]
                tails[t][k] = i
            else:
                tails[t].append(i)
    k = rng.poisson(mean_in, size=n).astype(np.int64)
    k[0] = 0
    dst = np.repeat(np.arange(n, dtype=np.int64), k)
    lo = np.maximum(dst - window, 0)
    src = lo + (rng.random(dst.shape[0]) * (dst - lo)).astype(np.int64)
    ok = src < dst
    src, dst = src[ok], dst[ok]
    o = np.argsort(dst, kind="stable")
    src, dst = src[o], dst[o]
    in_ptr = np.zeros(n + 1, np.int64)
    np.add.at(in_ptr, dst + 1, 1)
    in_ptr = np.cumsum(in_ptr)
    dur = rng.integers(1, max_dur + 1, size=n).astype(np.int64)
    dur[rng.random(n) < zero_frac] = 0
    gap = rng.integers(0, max_dur // 4 + 1, size=n).astype(np.int64)
    gap[rng.random(n) < 0.5] = 0
    cls = rng.integers(0, n_edge_cls, size=src.shape[0]).astype(np.uint8)
    g = TaskGraph(n, T, in_ptr, src.astype(np.int32), cls, prev, thread, dur, gap,
                  rng.integers(0, n_node_cls, size=n).astype(np.uint16), n_node_cls,
                  n_edge_cls, np.zeros(n, np.uint8), np.full(n, -1, np.int32),
                  np.full(n, -1, np.int64), "random-shared")
    pp = (thread >= n_ordered).astype(np.uint8)
    prio = rng.integers(-prio_range, prio_range + 1, size=n).astype(np.int32)
    return g, pp, prio


def random_variants(rng, g: TaskGraph, V: int, p_remove: float = 0.2,
                    qs=(1, 2, 3, 4, 5, 7, 8, 10)) -> VariantSet:
    C = g.n_node_cls
    s = np.ones((C, V, 2), np.int32)
    for v in range(1, V):
        for c in range(C):
            if rng.random() < 0.6:
                s[c, v] = _random_pq(rng, qs, 3, 0)
    bits = rng.random((g.n, V)) < p_remove
    bits[:, 0] = False
    rb = pack_bits(bits)
    K = g.n_edge_cls
    eo = np.zeros((V, 1), np.uint64)
    for v in range(V):
        m = int(rng.integers(0, 1 << K)) | 1
        eo[v, 0] = np.uint64(m)
    eo[0, 0] = np.uint64((1 << K) - 1)
    return VariantSet(V, s, rb, eo, [(0, V, (1 << K) - 1)])
