"""Pins of the oracle against what the paper and the mathematics fix.

The oracle runs the event-driven simulation of Sec. 4.1 (Algorithm 1).  It
is checked here against things that are not the oracle:
  * brute force over every path of tiny random graphs (the start of a task is
    the latest release over all chains of parents; Algorithm 1 adds
    duration + gap along every dependency it follows);
  * closed forms (one thread; a CPU thread launching onto one stream);
  * the hand-worked rounding table for the shrink/scale primitive (Sec. 4.4);
  * invariants (serialization lower bound, monotonicity, 1-Lipschitz);
  * agreement of two readings of Remove (Sec. 4.4) and of three tie rules of
    schedule(), which the per-thread trace order makes irrelevant
    (Sec. 4.2.2: the order on a thread does not change between executions).
"""
import os

import numpy as np
import pytest

from paper_2006_03318_amd import workloads as W
from tests import helpers as H

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# independent brute force (pure Python, tiny graphs)
def _active_parents(g, vs, v, u):
    ps = []
    for e in range(int(g.in_ptr[u]), int(g.in_ptr[u + 1])):
        c = int(g.edge_cls[e])
        if (int(vs.edge_on[v, c // 64]) >> (c % 64)) & 1:
            ps.append(int(g.in_src[e]))
    if g.thread_prev[u] >= 0:
        ps.append(int(g.thread_prev[u]))
    return ps


def _weights(g, vs, v):
    rm = W.unpack_bits(vs.remove_bits, vs.n_variants)[:, v]
    d = np.zeros(g.n, dtype=object)
    gg = np.zeros(g.n, dtype=object)
    for u in range(g.n):
        p, q = (int(x) for x in vs.scale[g.node_cls[u], v])
        d[u] = 0 if rm[u] else (int(g.dur[u]) * p) // q
        gg[u] = 0 if rm[u] else int(g.gap[u])
    return rm, d, gg


def _paths_to(parents, u):
    ps = parents[u]
    if not ps:
        yield [u]
        return
    yield [u]
    for p in ps:
        for path in _paths_to(parents, p):
            yield path + [u]


def brute_force(g, vs, v):
    """Every start = max over all parent chains of the summed
    duration + gap of the tasks on the chain (removed tasks weigh 0)."""
    rm, d, gg = _weights(g, vs, v)
    parents = {u: _active_parents(g, vs, v, u) for u in range(g.n)}
    S = []
    for u in range(g.n):
        best = 0
        for path in _paths_to(parents, u):
            best = max(best, sum(d[x] + gg[x] for x in path[:-1]))
        S.append(best)
    F = [S[u] + d[u] for u in range(g.n)]
    ms = max([F[u] for u in range(g.n) if not rm[u]], default=0)
    return S, F, ms


def brute_force_contracted(g, vs, v):
    """Remove = unlink: delete removed tasks and link every predecessor to
    every successor, then brute-force the smaller graph."""
    rm, d, gg = _weights(g, vs, v)
    raw = {u: _active_parents(g, vs, v, u) for u in range(g.n)}

    def eff(u, seen=None):
        out = set()
        for p in raw[u]:
            if rm[p]:
                out |= eff(p)
            else:
                out.add(p)
        return out
    parents = {u: sorted(eff(u)) for u in range(g.n)}
    kept = [u for u in range(g.n) if not rm[u]]
    S = {}
    for u in kept:
        best = 0
        for path in _paths_to({k: parents[k] for k in range(g.n)}, u):
            best = max(best, sum(d[x] + gg[x] for x in path[:-1]))
        S[u] = best
    for u in range(g.n):
        if rm[u]:
            S[u] = max([S[p] + d[p] + gg[p] for p in parents[u]], default=0)
    F = [S[u] + d[u] for u in range(g.n)]
    ms = max([F[u] for u in kept], default=0)
    return [S[u] for u in range(g.n)], F, ms


def _random_case(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 10))
    T = int(rng.integers(1, 4))
    K = int(rng.integers(1, 3))
    g = W.random_graph(rng, n, T, p_edge=float(rng.uniform(0.1, 0.5)), n_edge_cls=K)
    vs = W.random_variants(rng, g, int(rng.integers(1, 5)), p_remove=0.25)
    return g, vs


# P1 ------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(150))
def test_oracle_equals_brute_force(oracle_mod, seed):
    g, vs = _random_case(seed)
    S, F, ms, _ = oracle_mod.run(g, vs)
    for v in range(vs.n_variants):
        bS, bF, bms = brute_force(g, vs, v)
        assert list(S[v]) == bS
        assert list(F[v]) == bF
        assert ms[v] == bms


@pytest.mark.parametrize("seed", range(40))
def test_oracle_equals_brute_force_wide_variant_sets(oracle_mod, seed):
    """Variant counts past one and two 32-bit removal words (33, 64, 65, 97)
    and three or four edge classes: the removal bit of (task u, variant v)
    sits in word v // 32 of a row of ceil(V / 32) words, and each variant
    switches its own subset of edge classes on.  The brute force unpacks the
    bits with the input module's own routine, not the oracle's indexing."""
    rng = np.random.default_rng(50_000 + seed)
    n = int(rng.integers(2, 9))
    T = int(rng.integers(1, 4))
    K = int(rng.integers(3, 5))
    g = W.random_graph(rng, n, T, p_edge=float(rng.uniform(0.2, 0.6)), n_edge_cls=K)
    V = int(rng.choice([33, 64, 65, 97]))
    vs = W.random_variants(rng, g, V, p_remove=0.3)
    S, F, ms, _ = oracle_mod.run(g, vs)
    # each variant is also run on its own, alone in a set of one variant
    for v in range(V):
        bS, bF, bms = brute_force(g, vs, v)
        assert list(S[v]) == bS, (v, V)
        assert list(F[v]) == bF, (v, V)
        assert ms[v] == bms, (v, V)
    for v in (V - 1, 32, 31):
        one = vs.subset(v, v + 1)
        S1, F1, ms1, _ = oracle_mod.run(g, one)
        assert list(S1[0]) == list(S[v]) and ms1[0] == ms[v]


@pytest.mark.parametrize("seed", range(150, 230))
def test_unlink_reading_equals_contracted_brute_force(oracle_mod, seed):
    g, vs = _random_case(seed)
    S1, F1, ms1, _ = oracle_mod.run(g, vs, mode=1)
    S0, F0, ms0, _ = oracle_mod.run(g, vs, mode=0)
    for v in range(vs.n_variants):
        bS, bF, bms = brute_force_contracted(g, vs, v)
        assert list(S1[v]) == bS
        assert ms1[v] == bms
    # P7: the two readings of Remove agree
    assert (S0 == S1).all() and (F0 == F1).all() and (ms0 == ms1).all()


# P2 ------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(10))
def test_single_thread_closed_form(oracle_mod, seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 50))
    d = rng.integers(0, 10**6, n)
    gp = rng.integers(0, 10**4, n)
    g = H.graph(1, [0] * n, [], d, gp)
    vs = H.variants(g, V=1)
    _, _, ms, _ = oracle_mod.run(g, vs)
    # the last task starts after every earlier task and its gap
    assert ms[0] == int(d[:-1].sum() + gp[:-1].sum() + d[-1])


# P3 ------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(10))
def test_launch_pipeline_closed_form(oracle_mod, seed):
    """CPU thread issues n launches; launch i triggers kernel i on one stream.
    Two-stage flow shop: makespan = max_j [sum_{i<=j}(dL_i+gL_i) + sum_{i>=j} dK_i]."""
    rng = np.random.default_rng(2000 + seed)
    n = int(rng.integers(1, 40))
    dL = rng.integers(5000, 15001, n)
    gL = rng.integers(0, 3001, n)
    dK = rng.integers(1, 60000, n)
    thread, dur, gap, edges = [], [], [], []
    for i in range(n):
        thread += [0, 1]
        dur += [int(dL[i]), int(dK[i])]
        gap += [int(gL[i]), 0]
        edges.append((2 * i, 2 * i + 1))
    g = H.graph(2, thread, edges, dur, gap)
    vs = H.variants(g, V=1)
    _, _, ms, _ = oracle_mod.run(g, vs)
    cum = np.cumsum(dL + gL)
    tail = np.cumsum(dK[::-1])[::-1]
    assert ms[0] == int(max(cum[j] + tail[j] for j in range(n)))


# P9 ------------------------------------------------------------------------
def _floor_rows():
    rows = []
    with open(os.path.join(GOLDEN, "floor_table.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(int(x) for x in line.split()))
    return rows


@pytest.mark.parametrize("d,p,q,expected", _floor_rows())
def test_scale_rounding_table(oracle_mod, d, p, q, expected):
    g = H.graph(1, [0], [], [d], [0])
    vs = H.variants(g, scales=[{0: (p, q)}])
    _, F, ms, _ = oracle_mod.run(g, vs)
    assert ms[0] == expected and F[0][0] == expected


# P4 ------------------------------------------------------------------------
def _replay_in_trace_order(g):
    """Replay the untransformed trace task by task in emission order (the
    order the trace was recorded in): a task begins once its thread is free
    and every task it depends on has released (end + gap)."""
    n = g.n
    rel = np.zeros(n, np.int64)
    start = np.zeros(n, np.int64)
    free = {}
    for u in range(n):
        t = int(g.thread_id[u])
        s = free.get(t, 0)
        for e in range(int(g.in_ptr[u]), int(g.in_ptr[u + 1])):
            s = max(s, int(rel[g.in_src[e]]))
        start[u] = s
        rel[u] = s + int(g.dur[u]) + int(g.gap[u])
        free[t] = int(rel[u])
    end = start + g.dur
    return start, int(end.max()) if n else 0


@pytest.mark.parametrize("k,iters", [(1, 4), (2, 1), (4, 1), (3, 1)])
def test_identity_reproduces_trace(oracle_mod, k, iters):
    g, vs = W.config(k, iters=iters, variants=4 if k != 3 else 8)
    start, it_time = _replay_in_trace_order(g)
    v0 = 0
    S, F, ms, nb = oracle_mod.run(g, vs, variants=[v0])
    assert (S[0] == start).all()
    assert ms[0] == it_time
    assert nb[0] == 0      # the thread order never had to hold a task back


# P5, P6 ---------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(20))
def test_serialization_bound_and_monotone(oracle_mod, seed):
    rng = np.random.default_rng(3000 + seed)
    g = W.random_graph(rng, int(rng.integers(5, 60)), int(rng.integers(1, 5)), p_edge=0.1,
                       max_dur=1000)
    vs = W.random_variants(rng, g, 4, p_remove=0.2)
    S, F, ms, _ = oracle_mod.run(g, vs)
    rm = W.unpack_bits(vs.remove_bits, vs.n_variants)
    for v in range(vs.n_variants):
        d = (g.dur * vs.scale[g.node_cls, v, 0]) // vs.scale[g.node_cls, v, 1]
        d = np.where(rm[:, v], 0, d)
        for t in range(g.n_threads):
            assert ms[v] >= d[g.thread_id == t].sum()
    # raising one duration or gap by delta moves the makespan by [0, delta]
    ident = H.variants(g, V=1)
    base = oracle_mod.run(g, ident)[2][0]
    for _ in range(10):
        u = int(rng.integers(0, g.n))
        delta = int(rng.integers(1, 5000))
        for field in ("dur", "gap"):
            g2 = W.TaskGraph(**{**g.__dict__})
            arr = getattr(g, field).copy()
            arr[u] += delta
            setattr(g2, field, arr)
            m2 = oracle_mod.run(g2, ident)[2][0]
            assert base <= m2 <= base + delta
        # removal never lengthens the iteration
        rmv = H.variants(g, removed=[[u]])
        assert oracle_mod.run(g, rmv)[2][0] <= base


def test_unit_scale_is_identity(oracle_mod):
    g, vs = W.config(1)
    ident = H.variants(g, V=1)
    ones = H.variants(g, scales=[{c: (7, 7) for c in range(g.n_node_cls)}])
    assert (oracle_mod.run(g, ident)[0] == oracle_mod.run(g, ones)[0]).all()


# P8 ------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 2])
def test_schedule_tie_rules_agree(oracle_mod, k):
    g, vs = W.config(k, variants=8)
    outs = [oracle_mod.run(g, vs, tie=t) for t in (0, 1, 2)]
    for o in outs[1:]:
        assert (o[0] == outs[0][0]).all() and (o[2] == outs[0][2]).all()
    assert (outs[0][3] == 0).all()


@pytest.mark.parametrize("seed", range(40))
def test_tie_rules_agree_random(oracle_mod, seed):
    g, vs = _random_case(500 + seed)
    outs = [oracle_mod.run(g, vs, tie=t) for t in (0, 1, 2)]
    for o in outs[1:]:
        assert (o[0] == outs[0][0]).all()


# errors ---------------------------------------------------------------------
def test_cycle_is_reported(oracle_mod):
    g = H.graph(2, [0, 1], [(0, 1), (1, 0)], [1, 1], [0, 0])
    with pytest.raises(oracle_mod.OracleError) as ei:
        oracle_mod.run(g, H.variants(g, V=1))
    assert ei.value.code == oracle_mod.ECYCLE


def test_inactive_edge_breaks_cycle(oracle_mod):
    g = H.graph(2, [0, 1], [(0, 1), (1, 0)], [5, 7], [0, 0], edge_cls=[0, 1], n_edge_cls=2)
    vs = H.variants(g, edge_on=[0b01, 0b10])
    S, F, ms, _ = oracle_mod.run(g, vs)
    assert list(S[0]) == [0, 5] and list(S[1]) == [7, 0]


def test_empty_graph(oracle_mod):
    g = H.graph(1, [], [], [], [])
    vs = H.variants(g, V=3)
    S, F, ms, _ = oracle_mod.run(g, vs)
    assert list(ms) == [0, 0, 0]


def test_all_removed_makespan_zero(oracle_mod):
    g = H.graph(2, [0, 1, 0], [(0, 1)], [5, 6, 7], [1, 1, 1])
    vs = H.variants(g, removed=[[0, 1, 2]])
    S, F, ms, _ = oracle_mod.run(g, vs)
    assert ms[0] == 0 and (S[0] == 0).all()


# levelization ---------------------------------------------------------------
def _brute_steps(g, mask):
    par = {}
    for u in range(g.n):
        ps = []
        for e in range(int(g.in_ptr[u]), int(g.in_ptr[u + 1])):
            if (mask >> int(g.edge_cls[e])) & 1:
                s = int(g.in_src[e])
                ps.append((s, 1 if g.thread_id[s] != g.thread_id[u] else 0))
        if g.thread_prev[u] >= 0:
            ps.append((int(g.thread_prev[u]), 0))
        par[u] = ps

    def walk(u):
        # all paths ending at u: (edges, cross edges)
        if not par[u]:
            yield (0, 0)
        for p, w in par[u]:
            for a, b in walk(p):
                yield (a + 1, b + w)
    lv, ph = [], []
    for u in range(g.n):
        paths = list(walk(u))
        lv.append(max(a for a, _ in paths))
        ph.append(max(b for _, b in paths))
    return lv, ph


@pytest.mark.parametrize("seed", range(80))
def test_levels_and_phases_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(7000 + seed)
    g = W.random_graph(rng, int(rng.integers(1, 10)), int(rng.integers(1, 4)),
                       p_edge=float(rng.uniform(0.1, 0.5)), n_edge_cls=2)
    mask = int(rng.integers(1, 4))
    lv, ph = oracle_mod.steps(g, mask)
    blv, bph = _brute_steps(g, mask)
    assert list(lv) == blv and list(ph) == bph


def test_steps_cycle(oracle_mod):
    g = H.graph(2, [0, 1], [(0, 1), (1, 0)], [1, 1], [0, 0])
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.steps(g)
