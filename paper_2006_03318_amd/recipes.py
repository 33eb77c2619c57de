"""What-if recipes compiled into variant tables.

The paper models each optimization as a short program over the task graph
(Sec. 5.1 and the what-if algorithms of its appendix): select tasks by what
they are (GPU kernel, weight-update kernel, layer, communication), then
shrink or scale their durations, remove them, or switch dependencies.  Here
a recipe is such a program over the metadata of a `workloads.TaskGraph`
(task kind, layer, operator tag, iteration, launch call), and a sweep is a
list of variants, each a list of recipes applied in order.  `compile_sweep`
turns a sweep into what the C-ABI takes:

  * one task class per distinct column of (p, q) ratios over the sweep, so
    each task's duration in variant v is floor(d * p / q) with (p, q) =
    scale[class][v] (stacked scales are multiplied as reduced rationals);
  * removal bits per (task, variant);
  * the edge classes each variant switches on, and the batches of
    consecutive variants that share them.

Host-only: it computes ratios, removal sets and masks, never a start or a
finish time.  The one recipe that needs durations (fused weight update: the
remaining kernel takes the sum of the fused ones) sums floor(d * p / q) of
the tasks it fuses, with the ratios the earlier recipes of that variant left.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import workloads as W

I32_MAX = (1 << 31) - 1


@dataclasses.dataclass
class Plan:
    """The state of one variant while its recipes run."""
    p: np.ndarray            # int64 [N] numerators
    q: np.ndarray            # int64 [N] denominators (q >= 1)
    removed: np.ndarray      # bool [N]
    edge_mask: int           # edge classes switched on


def _reduce(p: np.ndarray, q: np.ndarray):
    g = np.gcd(p, q)
    g[g == 0] = 1
    return p // g, q // g


def scale_tasks(plan: Plan, mask: np.ndarray, num: int, den: int):
    """Multiply the duration ratio of the selected tasks by num / den."""
    if num < 0 or den < 1:
        raise ValueError("a scale needs num >= 0 and den >= 1")
    p, q = _reduce(plan.p[mask] * num, plan.q[mask] * den)
    if p.size and (p.max() > I32_MAX or q.max() > I32_MAX):
        raise ValueError("a stacked scale does not fit 32-bit p/q")
    plan.p[mask], plan.q[mask] = p, q


def remove_tasks(plan: Plan, g: W.TaskGraph, mask: np.ndarray, with_launch: bool = True):
    """Remove the selected tasks (Sec. 4.4, Remove) and, for device tasks,
    the CPU launch calls that issued them."""
    plan.removed |= mask
    if with_launch:
        lo = g.launch_of[mask]
        lo = lo[lo >= 0]
        plan.removed[lo] = True


# ---------------------------------------------------------------------------
# task selections (the Select primitive)
def is_kernel(g):
    return np.isin(g.kind, W.GPU_KINDS)


def is_compute_kernel(g):
    """GEMM and convolution kernels: the ones tensor cores speed up 3x."""
    return np.isin(g.kind, (W.K_GEMM, W.K_CONV))


def is_weight_update(g):
    return np.isin(g.kind, (W.K_WU, W.K_OPT))


def is_comm(g):
    return g.kind == W.K_COMM


def is_launch(g):
    return g.kind == W.K_LAUNCH


def in_layers(g, layers):
    return np.isin(g.layer, np.asarray(list(layers), dtype=g.layer.dtype))


def with_op(g, op):
    if g.op is None:
        raise ValueError("the graph carries no operator tags")
    return g.op == op


# ---------------------------------------------------------------------------
# recipes
class Recipe:
    def apply(self, g: W.TaskGraph, plan: Plan) -> None:
        raise NotImplementedError


@dataclasses.dataclass
class AMP(Recipe):
    """Automatic mixed precision (appendix, What_If_AMP): GPU kernels run
    2x faster, compute kernels (GEMM, convolution) 3x."""
    compute_den: int = 3
    other_den: int = 2

    def apply(self, g, plan):
        k = is_kernel(g)
        c = is_compute_kernel(g)
        scale_tasks(plan, k & c, 1, self.compute_den)
        scale_tasks(plan, k & ~c, 1, self.other_den)


@dataclasses.dataclass
class FusedAdam(Recipe):
    """Fused optimizer (appendix, What_If_Fused_Adam; Sec. 5.1): in every
    iteration's weight-update phase one kernel remains, with the sum of the
    durations of all of the phase's kernels; the others are removed together
    with their launch calls (the fused optimizer launches once)."""

    def apply(self, g, plan):
        wu = is_weight_update(g) & ~plan.removed
        iters = g.iteration if g.iteration is not None else np.zeros(g.n, np.int32)
        for it in np.unique(iters[wu]):
            ids = np.nonzero(wu & (iters == it))[0]
            d = g.dur[ids].astype(object)
            cur = [int(x) * int(pp) // int(qq) for x, pp, qq in zip(d, plan.p[ids], plan.q[ids])]
            total = sum(cur)
            keep = next((int(u) for u in ids if g.dur[u] > 0), None)
            if keep is None:
                remove_tasks(plan, g, np.isin(np.arange(g.n), ids))
                continue
            if total > I32_MAX or g.dur[keep] > I32_MAX:
                raise ValueError("fused duration does not fit a 32-bit ratio")
            rest = np.isin(np.arange(g.n), ids[ids != keep])
            remove_tasks(plan, g, rest)
            # floor(d_keep * total / d_keep) = total, exactly
            dk = int(g.dur[keep])
            gg = math.gcd(total, dk)
            plan.p[keep] = total // gg
            plan.q[keep] = dk // gg


@dataclasses.dataclass
class RestructureBatchnorm(Recipe):
    """Restructured batch normalization (appendix,
    What_If_Restructuring_Batchnorm): ReLU kernels are removed (fused away)
    and batch-normalization kernels take half their time."""

    def apply(self, g, plan):
        k = is_kernel(g)
        remove_tasks(plan, g, k & with_op(g, W.OP_RELU))
        scale_tasks(plan, k & with_op(g, W.OP_BN), 1, 2)


@dataclasses.dataclass
class ScaleLayers(Recipe):
    """MetaFlow-style layer substitution, scaling half (appendix,
    What_If_MetaFlow, Scale_layer): the GPU kernels of the given layers run
    num/den as long."""
    layers: Sequence[int]
    num: int
    den: int

    def apply(self, g, plan):
        scale_tasks(plan, is_kernel(g) & in_layers(g, self.layers), self.num, self.den)


@dataclasses.dataclass
class RemoveLayers(Recipe):
    """MetaFlow-style layer substitution, removal half (Remove_layer): the
    GPU kernels of the given layers disappear, with their launch calls."""
    layers: Sequence[int]

    def apply(self, g, plan):
        remove_tasks(plan, g, is_kernel(g) & in_layers(g, self.layers))


@dataclasses.dataclass
class FuseElementwise(Recipe):
    """Kernel fusion of element-wise kernels into their producers: each
    selected kernel (kinds `kinds`) is removed, with its launch call, with
    probability `density` (seeded)."""
    density: float
    seed: int
    kinds: Tuple[int, ...] = (W.K_ELEM, W.K_AUX, W.K_WU)

    def apply(self, g, plan):
        rng = np.random.default_rng(self.seed)
        sel = np.isin(g.kind, self.kinds) & (rng.random(g.n) < self.density)
        remove_tasks(plan, g, sel)


@dataclasses.dataclass
class ScaleKernels(Recipe):
    """Every GPU kernel num/den as long (a faster or slower device)."""
    num: int
    den: int

    def apply(self, g, plan):
        scale_tasks(plan, is_kernel(g), self.num, self.den)


@dataclasses.dataclass
class ScaleLaunch(Recipe):
    """CPU launch overhead num/den as long (0 = free launches)."""
    num: int
    den: int

    def apply(self, g, plan):
        scale_tasks(plan, is_launch(g), self.num, self.den)


@dataclasses.dataclass
class Distributed(Recipe):
    """Data-parallel training (appendix, What_If_Distributed_Training): the
    graph carries one all-reduce per gradient bucket (after the bucket's last
    backward kernel, before the first weight-update kernel), with durations
    for `base_gbps`; at `gbps` they take base/gbps as long."""
    gbps: int
    base_gbps: int = 10

    def apply(self, g, plan):
        scale_tasks(plan, is_comm(g), self.base_gbps, self.gbps)


@dataclasses.dataclass
class SingleDevice(Recipe):
    """No data parallelism: every all-reduce is removed."""

    def apply(self, g, plan):
        remove_tasks(plan, g, is_comm(g), with_launch=False)


@dataclasses.dataclass
class CompressGradients(Recipe):
    """Gradient compression (Deep Gradient Compression, appendix
    What_If_DGC, its communication-scaling step): the all-reduces of the
    given buckets (indices in trace order within an iteration; None = all)
    move `ratio_num/ratio_den` of the bytes.  The inserted compression
    kernels of the recipe are not modeled."""
    ratio_num: int = 1
    ratio_den: int = 4
    buckets: Optional[Sequence[int]] = None

    def apply(self, g, plan):
        c = is_comm(g)
        if self.buckets is not None:
            iters = g.iteration if g.iteration is not None else np.zeros(g.n, np.int32)
            idx = np.full(g.n, -1, np.int64)
            for it in np.unique(iters[c]):
                ids = np.nonzero(c & (iters == it))[0]
                idx[ids] = np.arange(ids.shape[0])
            c = c & np.isin(idx, np.asarray(list(self.buckets), np.int64))
        scale_tasks(plan, c, self.ratio_num, self.ratio_den)


@dataclasses.dataclass
class ScaleCopies(Recipe):
    """The offload and prefetch copies num/den as long (a faster or slower
    host link)."""
    num: int
    den: int

    def apply(self, g, plan):
        scale_tasks(plan, (g.kind == W.K_MEMCPY) & np.isin(g.op, (W.OP_OFFLOAD, W.OP_PREFETCH)),
                    self.num, self.den)


@dataclasses.dataclass
class RemoveOffload(Recipe):
    """No memory offloading: the offload and prefetch copies are removed
    with their launch calls."""

    def apply(self, g, plan):
        remove_tasks(plan, g, (g.kind == W.K_MEMCPY) & np.isin(g.op, (W.OP_OFFLOAD,
                                                                      W.OP_PREFETCH)))


@dataclasses.dataclass
class EdgeClasses(Recipe):
    """Switch dependency classes on or off (Select plus re-route: for
    example one order of the communication channel)."""
    on: int = 0
    off: int = 0

    def apply(self, g, plan):
        plan.edge_mask = (plan.edge_mask | self.on) & ~self.off


# ---------------------------------------------------------------------------
def compile_sweep(g: W.TaskGraph, variants: List[List[Recipe]],
                  base_edge_mask: int = 1,
                  one_batch_mask: Optional[int] = None) -> Tuple[W.TaskGraph, W.VariantSet]:
    """Run each variant's recipes and pack the result.  Returns the graph
    with one task class per distinct ratio column (and n_node_cls set) and
    the variant tables; batches are the runs of consecutive variants with
    the same edge classes, or, with `one_batch_mask`, one batch levelized
    with those classes (the caller knows their union is acyclic; every
    variant's classes must lie inside it)."""
    V = len(variants)
    if V < 1:
        raise ValueError("a sweep needs at least one variant")
    N = g.n
    P = np.ones((V, N), np.int64)
    Q = np.ones((V, N), np.int64)
    R = np.zeros((V, N), bool)
    masks = []
    for v, recipes in enumerate(variants):
        plan = Plan(np.ones(N, np.int64), np.ones(N, np.int64), np.zeros(N, bool), base_edge_mask)
        for r in recipes:
            r.apply(g, plan)
        P[v], Q[v], R[v] = plan.p, plan.q, plan.removed
        masks.append(plan.edge_mask)
    cls, rep = _ratio_classes(P, Q)
    C = rep.shape[0]
    if C > 65535:
        raise ValueError("more than 65535 distinct ratio columns")
    scale = np.stack([P[:, rep].T, Q[:, rep].T], axis=2).astype(np.int32)   # [C][V][2]
    edge_on = np.array(masks, np.uint64).reshape(V, 1)
    batches = []
    if one_batch_mask is not None:
        if any(m & ~one_batch_mask for m in masks):
            raise ValueError("a variant switches on an edge class outside the batch's")
        batches.append((0, V, int(one_batch_mask)))
    else:
        v0 = 0
        for v in range(1, V + 1):
            if v == V or masks[v] != masks[v0]:
                batches.append((v0, v, int(masks[v0])))
                v0 = v
    g2 = dataclasses.replace(g, node_cls=cls.astype(np.uint16), n_node_cls=int(C))
    return g2, W.VariantSet(V, scale, W.pack_bits(np.ascontiguousarray(R.T)), edge_on, batches)


def _ratio_classes(P: np.ndarray, Q: np.ndarray):
    """Group tasks by their column of ratios over the sweep.  P, Q: [V][N].
    Returns (class of each task, one representative task per class), classes
    numbered in order of their first task.  Columns are hashed, then every
    task is compared with its class representative, so a hash collision can
    only cost time (the exact row sort below), never a wrong grouping."""
    V, N = P.shape
    if N == 0:
        return np.zeros(0, np.int64), np.zeros(1, np.int64)
    h = np.zeros(N, np.uint64)
    with np.errstate(over="ignore"):
        for v in range(V):
            h = h * np.uint64(0x9E3779B97F4A7C15) + P[v].astype(np.uint64) * np.uint64(
                0xC2B2AE3D27D4EB4F) + Q[v].astype(np.uint64)
            h ^= h >> np.uint64(29)
    _, first, inv = np.unique(h, return_index=True, return_inverse=True)
    inv = inv.reshape(-1)
    if not (np.array_equal(P, P[:, first[inv]]) and np.array_equal(Q, Q[:, first[inv]])):
        key = np.concatenate([P, Q], axis=0).T
        _, first, inv = np.unique(key, axis=0, return_index=True, return_inverse=True)
        inv = inv.reshape(-1)
    order = np.argsort(first, kind="stable")          # classes by first task
    rank = np.empty_like(order)
    rank[order] = np.arange(order.shape[0])
    return rank[inv], first[order]


def task_ratios(vs: W.VariantSet, g: W.TaskGraph, v: int):
    """(p, q) of every task in variant v (for inspection and tests)."""
    return vs.scale[g.node_cls, v, 0].astype(np.int64), vs.scale[g.node_cls, v, 1].astype(np.int64)
