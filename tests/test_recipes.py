"""The what-if recipe compiler against hand-derived tables.

A 23-task graph of two training iterations carries every task kind the
recipes select.  For each recipe combination the expected duration ratio
(p, q) and removal of every task is written out by hand from the recipe's
definition (AMP, fused optimizer, restructured batchnorm, layer scaling and
removal, data-parallel bandwidth, gradient compression, launch cost), and
the compiled tables must reproduce it exactly.  A second check runs the
oracle on the compiled tables and on graphs edited by hand (durations
replaced, removed tasks zeroed), which must agree task by task.
"""
import numpy as np
import pytest

from paper_2006_03318_amd import recipes as R
from paper_2006_03318_amd import workloads as W
from tests import helpers as H

CPU, GPU, NET = 0, 1, 2

# (thread, kind, layer, op, dur, launch_of, iteration)
TASKS = [
    (CPU, W.K_LAUNCH, 0, W.OP_NONE, 10, -1, 0),      # 0
    (GPU, W.K_CONV, 0, W.OP_CONV, 300, 0, 0),        # 1
    (CPU, W.K_LAUNCH, 0, W.OP_NONE, 10, -1, 0),      # 2
    (GPU, W.K_GPU_OTHER, 0, W.OP_BN, 100, 2, 0),     # 3
    (CPU, W.K_LAUNCH, 0, W.OP_NONE, 10, -1, 0),      # 4
    (GPU, W.K_ELEM, 0, W.OP_RELU, 50, 4, 0),         # 5
    (CPU, W.K_LAUNCH, 1, W.OP_NONE, 10, -1, 0),      # 6
    (GPU, W.K_GEMM, 1, W.OP_NONE, 90, 6, 0),         # 7
    (CPU, W.K_LAUNCH, -1, W.OP_NONE, 10, -1, 0),     # 8
    (GPU, W.K_WU, -1, W.OP_NONE, 7, 8, 0),           # 9
    (CPU, W.K_LAUNCH, -1, W.OP_NONE, 10, -1, 0),     # 10
    (GPU, W.K_OPT, -1, W.OP_NONE, 11, 10, 0),        # 11
    (NET, W.K_COMM, -1, W.OP_NONE, 1000, -1, 0),     # 12  bucket 0
    (NET, W.K_COMM, -1, W.OP_NONE, 400, -1, 0),      # 13  bucket 1
    (GPU, W.K_MEMCPY, -1, W.OP_NONE, 200, -1, 0),    # 14
    (CPU, W.K_SYNC, -1, W.OP_NONE, 5, -1, 0),        # 15
    (CPU, W.K_LAUNCH, -1, W.OP_NONE, 10, -1, 1),     # 16
    (GPU, W.K_WU, -1, W.OP_NONE, 0, 16, 1),          # 17  zero-length kernel
    (CPU, W.K_LAUNCH, -1, W.OP_NONE, 10, -1, 1),     # 18
    (GPU, W.K_WU, -1, W.OP_NONE, 30, 18, 1),         # 19
    (CPU, W.K_LAUNCH, -1, W.OP_NONE, 10, -1, 1),     # 20
    (GPU, W.K_OPT, -1, W.OP_NONE, 13, 20, 1),        # 21
    (NET, W.K_COMM, -1, W.OP_NONE, 600, -1, 1),      # 22  bucket 0 of iteration 1
]
EDGES = [(0, 1), (2, 3), (4, 5), (6, 7), (8, 9), (10, 11), (7, 12), (7, 13), (12, 9),
         (13, 9), (14, 15), (13, 15), (16, 17), (18, 19), (20, 21), (19, 22), (11, 16)]
LAUNCHES = [0, 2, 4, 6, 8, 10, 16, 18, 20]


def toy_graph():
    th, kind, layer, op, dur, lo, it = zip(*TASKS)
    g = H.graph(3, list(th), EDGES, list(dur), [0] * len(TASKS))
    g.kind = np.array(kind, np.uint8)
    g.layer = np.array(layer, np.int32)
    g.op = np.array(op, np.uint8)
    g.launch_of = np.array(lo, np.int64)
    g.iteration = np.array(it, np.int32)
    return g


SWEEP = [
    [],
    [R.AMP()],
    [R.RestructureBatchnorm()],
    [R.AMP(), R.FusedAdam()],
    [R.FusedAdam(), R.AMP()],
    [R.Distributed(25), R.CompressGradients(1, 4, [1])],
    [R.EdgeClasses(on=4)],
    [R.EdgeClasses(on=4), R.ScaleLaunch(0, 1), R.RemoveLayers([0]), R.ScaleLayers([1], 3, 2),
     R.SingleDevice()],
]

AMP_RATIO = {1: (1, 3), 3: (1, 2), 5: (1, 2), 7: (1, 3), 9: (1, 2), 11: (1, 2), 17: (1, 2),
             19: (1, 2), 21: (1, 2)}

# per variant: {task: (p, q)} for tasks that are not 1/1, and the removed set
EXPECTED = [
    ({}, set()),
    (AMP_RATIO, set()),
    ({3: (1, 2)}, {4, 5}),
    # AMP first: iteration 0 fuses floor(7/2) + floor(11/2) = 8 into task 9;
    # iteration 1 keeps task 19 (task 17 has zero length): 0 + 15 + 6 = 21
    ({**AMP_RATIO, 9: (8, 7), 19: (7, 10)}, {10, 11, 16, 17, 20, 21}),
    # fused first: 7 + 11 = 18 then halved -> 9/7; 0 + 30 + 13 = 43 then halved
    ({**AMP_RATIO, 9: (9, 7), 19: (43, 60)}, {10, 11, 16, 17, 20, 21}),
    # 10 GB/s -> 25 GB/s is 2/5; bucket 1 also moves 1/4 of the bytes
    ({12: (2, 5), 13: (1, 10), 22: (2, 5)}, set()),
    ({}, set()),
    ({**{u: (0, 1) for u in LAUNCHES}, 7: (3, 2)}, {0, 1, 2, 3, 4, 5, 12, 13, 22}),
]
EXPECTED_MASKS = [1, 1, 1, 1, 1, 1, 5, 5]


def _hand_tables(n):
    V = len(EXPECTED)
    P = np.ones((n, V), np.int64)
    Q = np.ones((n, V), np.int64)
    Rm = np.zeros((n, V), bool)
    for v, (ratios, removed) in enumerate(EXPECTED):
        for u, (p, q) in ratios.items():
            P[u, v], Q[u, v] = p, q
        for u in removed:
            Rm[u, v] = True
    return P, Q, Rm


def test_hand_table():
    g = toy_graph()
    g2, vs = R.compile_sweep(g, SWEEP)
    P, Q, Rm = _hand_tables(g.n)
    for v in range(len(SWEEP)):
        p, q = R.task_ratios(vs, g2, v)
        assert (p == P[:, v]).all() and (q == Q[:, v]).all(), v
    assert (W.unpack_bits(vs.remove_bits, vs.n_variants) == Rm).all()
    assert vs.edge_on[:, 0].tolist() == EXPECTED_MASKS
    assert vs.batches == [(0, 6, 1), (6, 8, 5)]


def test_classes_are_distinct_columns():
    """One class per distinct ratio column, numbered by first task."""
    g = toy_graph()
    g2, vs = R.compile_sweep(g, SWEEP)
    P, Q, _ = _hand_tables(g.n)
    cols = [tuple(P[u]) + tuple(Q[u]) for u in range(g.n)]
    first = {}
    for u, c in enumerate(cols):
        first.setdefault(c, len(first))
    assert g2.n_node_cls == len(first) == vs.scale.shape[0]
    assert [int(c) for c in g2.node_cls] == [first[c] for c in cols]


def test_fused_durations_are_exact_sums():
    g = toy_graph()
    g2, vs = R.compile_sweep(g, SWEEP)
    d = lambda u, v: int(g.dur[u]) * int(R.task_ratios(vs, g2, v)[0][u]) // int(
        R.task_ratios(vs, g2, v)[1][u])
    assert d(9, 3) == 7 // 2 + 11 // 2 and d(19, 3) == 0 + 30 // 2 + 13 // 2
    assert d(9, 4) == (7 + 11) // 2 and d(19, 4) == (0 + 30 + 13) // 2


def _hand_edited(g, v):
    """The graph of variant v written out directly: durations from the hand
    table, removed tasks with zero duration and gap."""
    P, Q, Rm = _hand_tables(g.n)
    g2 = W.TaskGraph(**{**g.__dict__})
    g2.dur = np.where(Rm[:, v], 0, g.dur * P[:, v] // Q[:, v])
    g2.gap = np.where(Rm[:, v], 0, g.gap)
    return g2


def test_oracle_on_compiled_tables_matches_hand_edited_graphs(oracle_mod):
    g = toy_graph()
    g.gap = np.array([3 if t == CPU else 0 for t, *_ in TASKS], np.int64)
    g2, vs = R.compile_sweep(g, SWEEP)
    S, F, M, _ = oracle_mod.run(g2, vs)
    for v in range(len(SWEEP)):
        ge = _hand_edited(g, v)
        ident = H.variants(ge, V=1, edge_on=[EXPECTED_MASKS[v]])
        s, f, m, _ = oracle_mod.run(ge, ident)
        assert (S[v] == s[0]).all() and (F[v] == f[0]).all() and M[v] == m[0], v


def test_identity_sweep_has_one_class():
    g = toy_graph()
    g2, vs = R.compile_sweep(g, [[], [R.ScaleKernels(3, 3)], [R.Distributed(10)]])
    assert g2.n_node_cls == 1 and (vs.scale == 1).all()
    assert not W.unpack_bits(vs.remove_bits, 3).any()


def test_stacking_reduces_and_guards_overflow():
    g = toy_graph()
    g2, vs = R.compile_sweep(g, [[R.ScaleKernels(6, 4), R.ScaleKernels(2, 3)]])
    p, q = R.task_ratios(vs, g2, 0)
    assert (p[1], q[1]) == (1, 1) and (p[0], q[0]) == (1, 1)
    with pytest.raises(ValueError):
        R.compile_sweep(g, [[R.ScaleKernels(1, 1 << 20), R.ScaleKernels(1, 1 << 12)]])
    with pytest.raises(ValueError):
        R.compile_sweep(g, [[R.ScaleKernels(-1, 1)]])
    with pytest.raises(ValueError):
        R.compile_sweep(g, [])


def test_batchnorm_needs_operator_tags():
    g = toy_graph()
    g.op = None
    with pytest.raises(ValueError):
        R.compile_sweep(g, [[R.RestructureBatchnorm()]])


def _random_sweep(rng, g, V, L):
    out = []
    for _ in range(V):
        r = []
        for _ in range(int(rng.integers(0, 4))):
            k = int(rng.integers(0, 9))
            if k == 0:
                r.append(R.AMP())
            elif k == 1:
                r.append(R.FusedAdam())
            elif k == 2:
                r.append(R.ScaleLayers([int(x) for x in rng.choice(L, 3)],
                                       int(rng.integers(0, 9)), int(rng.integers(1, 9))))
            elif k == 3:
                r.append(R.RemoveLayers([int(rng.integers(0, L))]))
            elif k == 4:
                r.append(R.FuseElementwise(float(rng.uniform(0, 0.5)), int(rng.integers(1000))))
            elif k == 5:
                r.append(R.ScaleLaunch(int(rng.integers(0, 3)), int(rng.integers(1, 5))))
            elif k == 6:
                r.append(R.ScaleKernels(int(rng.integers(1, 4)), int(rng.integers(1, 4))))
            elif k == 7:
                r.append(R.EdgeClasses(on=int(rng.integers(0, 4))))
            else:
                r.append(R.RestructureBatchnorm())
        out.append(r)
    return out


@pytest.mark.parametrize("seed", range(4))
def test_packing_matches_each_variant_alone(seed):
    """Compiling a sweep packs each variant's ratios and removals the same
    way compiling that variant on its own does."""
    rng = np.random.default_rng(900 + seed)
    g, _ = W.config(1, variants=1)
    sweep = _random_sweep(rng, g, 12, 20)
    g2, vs = R.compile_sweep(g, sweep)
    bits = W.unpack_bits(vs.remove_bits, vs.n_variants)
    for v, r in enumerate(sweep):
        g1, v1 = R.compile_sweep(g, [r])
        p, q = R.task_ratios(vs, g2, v)
        p1, q1 = R.task_ratios(v1, g1, 0)
        assert (p == p1).all() and (q == q1).all()
        assert (bits[:, v] == W.unpack_bits(v1.remove_bits, 1)[:, 0]).all()
        assert vs.edge_on[v, 0] == v1.edge_on[0, 0]
    for v0, v1_, m in vs.batches:
        assert (vs.edge_on[v0:v1_, 0] == np.uint64(m)).all()


def test_class_grouping_against_row_sort():
    rng = np.random.default_rng(5)
    for N, V in ((1, 1), (50, 3), (2000, 17)):
        base = rng.integers(0, 4, size=(7, 2 * V))
        rows = base[rng.integers(0, 7, size=N)]
        P, Q = rows[:, :V].T.copy(), rows[:, V:].T.copy() + 1
        cls, rep = R._ratio_classes(P, Q)
        _, inv = np.unique(rows, axis=0, return_inverse=True)
        inv = inv.reshape(-1)
        # same partition: equal rows <=> equal class
        assert all((cls == cls[u]).tolist() == (inv == inv[u]).tolist() for u in range(min(N, 50)))
        assert (P[:, rep[cls]] == P).all() and (Q[:, rep[cls]] == Q).all()
        assert cls[0] == 0 and (np.diff(np.maximum.accumulate(cls)) <= 1).all()


# --------------------------------------------------------------------------
# memory offloading (vDNN)
def test_vdnn_tables_and_structure():
    g, vs = W.vdnn_workload(iters=2, variants=30)
    copies = (g.kind == W.K_MEMCPY) & np.isin(g.op, (W.OP_OFFLOAD, W.OP_PREFETCH))
    assert copies.sum() == 2 * 20 * 2                   # one out, one back per layer and iteration
    bits = W.unpack_bits(vs.remove_bits, vs.n_variants)
    launches = g.launch_of[copies]
    for v in range(vs.n_variants):
        p, q = R.task_ratios(vs, g, v)
        if v % 5 == 0:                                  # no offloading: copies and launches gone
            assert bits[copies, v].all() and bits[launches, v].all()
            assert bits[:, v].sum() == 2 * copies.sum()
        else:
            assert not bits[:, v].any()
        pcie = (v // 5) % 3
        want = {0: (1, 1), 1: (1, 2), 2: (2, 1)}[pcie]
        assert (p[copies] == want[0]).all() and (q[copies] == want[1]).all()
        other = (g.kind == W.K_MEMCPY) & ~copies        # the input batch's copy keeps its time
        assert (p[other] == 1).all() and (q[other] == 1).all()
        pol = v % 5
        assert int(vs.edge_on[v, 0]) == (1 | (1 << (pol - 1)) if pol >= 2 else 1)
    assert vs.batches == [(0, 30, 0xF)]
    # policy edges: class d goes from the backward pass of layer l + d to the copy back of l
    dst = np.repeat(np.arange(g.n), np.diff(g.in_ptr))
    for d in (1, 2, 3):
        e = g.edge_cls == d
        assert e.sum() == (20 - d) * 2
        assert (g.op[dst[e]] == W.OP_PREFETCH).all()
        assert (g.layer[g.in_src[e]] == g.layer[dst[e]] + d).all()
    with pytest.raises(ValueError):
        R.compile_sweep(g, [[R.EdgeClasses(on=1 << 5)]], one_batch_mask=0xF)


def test_vdnn_policies_order(oracle_mod):
    """Prefetching further ahead never lengthens the iteration: the copy back
    of layer l waits for the backward pass of layer l + d, which starts no
    later for larger d; eager copies wait for nothing, and no offloading
    removes the copies altogether."""
    g, vs = W.vdnn_workload(iters=2, variants=30)
    _, _, M, _ = oracle_mod.run(g, vs, want_start=False, want_finish=False)
    for base in range(0, 30, 5):
        none, eager, d1, d2, d3 = M[base:base + 5]
        assert none <= eager <= d3 <= d2 <= d1
    assert M[2] > M[0]              # offloading costs something here
