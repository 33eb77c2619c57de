"""Pins of the oracle's simulation under an overridden schedule() (Sec. 4.4,
"Schedule"; the appendix's P3 priority rule).

* a hand-worked P3 example (tests/golden/p3_toy.txt) under both rules;
* on graphs where every thread is one chain the schedule cannot change the
  result, so both rules must reproduce the default simulation exactly;
* closed forms: a channel whose tasks are all ready at time 0 runs them back
  to back in priority order (trace order for the default rule);
* properties of any valid run on random graphs with shared threads: no two
  tasks of one thread overlap, every task starts after its parents release
  it, a thread never idles while one of its tasks is ready, and of two
  channel tasks ready when the first starts, the first has the higher
  priority (the earlier id for the default rule or equal priorities).
"""
import os

import numpy as np
import pytest

from paper_2006_03318_amd import workloads as W
from tests import helpers as H

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "p3_toy.txt")


def load_p3_toy():
    tasks, edges, exp = [], [], {}
    for line in open(GOLD):
        f = line.split("#")[0].split()
        if not f:
            continue
        if f[0] == "task":
            tasks.append([int(x) for x in f[1:8]])
        elif f[0] == "edge":
            edges.append((int(f[1]), int(f[2])))
        else:
            exp[f[0]] = [int(x) for x in f[1:]]
    tasks.sort()
    n = len(tasks)
    thread = [t[1] for t in tasks]
    g = H.graph(2, thread, edges, [t[3] for t in tasks], [t[4] for t in tasks],
                thread_order=[])
    g.thread_prev = np.array([t[2] for t in tasks], np.int32)
    pp = np.array([t[5] for t in tasks], np.uint8)
    prio = np.array([t[6] for t in tasks], np.int32)
    assert n == 9
    return g, pp, prio, exp


@pytest.mark.parametrize("policy", [0, 1])
def test_p3_hand_example(oracle_mod, policy):
    g, pp, prio, exp = load_p3_toy()
    S, F, M = oracle_mod.run_policy(g, H.variants(g, V=1), policy, pp, prio)
    assert S[0].tolist() == exp["start%d" % policy]
    assert M[0] == exp["makespan%d" % policy][0]
    assert (F[0] == S[0] + g.dur).all()


def _chain_case(seed):
    rng = np.random.default_rng(7100 + seed)
    n = int(rng.integers(1, 80))
    g = W.random_graph(rng, n, int(rng.integers(1, 5)), p_edge=float(rng.uniform(0.02, 0.3)),
                       n_edge_cls=int(rng.integers(1, 4)), max_dur=int(rng.choice([5, 1000])))
    vs = W.random_variants(rng, g, int(rng.integers(1, 40)), p_remove=0.3)
    pp = (rng.random(n) < 0.5).astype(np.uint8)
    prio = rng.integers(-3, 4, size=n).astype(np.int32)
    return g, vs, pp, prio


@pytest.mark.parametrize("seed", range(30))
def test_chains_make_the_rule_irrelevant(oracle_mod, seed):
    g, vs, pp, prio = _chain_case(seed)
    S, F, M, _ = oracle_mod.run(g, vs)
    for policy in (0, 1):
        s, f, m = oracle_mod.run_policy(g, vs, policy, pp, prio)
        assert (s == S).all() and (f == F).all() and (m == M).all()


def test_workload_rule_irrelevant(oracle_mod):
    g, vs = W.config(1, variants=8)
    S, F, M, _ = oracle_mod.run(g, vs)
    pp = np.ones(g.n, np.uint8)
    prio = (np.arange(g.n) % 7).astype(np.int32)
    s, f, m = oracle_mod.run_policy(g, vs, 1, pp, prio)
    assert (s == S).all() and (m == M).all()


@pytest.mark.parametrize("seed", range(10))
def test_all_ready_channel_closed_form(oracle_mod, seed):
    rng = np.random.default_rng(7300 + seed)
    n = int(rng.integers(1, 40))
    dur = rng.integers(0, 100, size=n)
    gap = rng.integers(0, 10, size=n)
    g = H.graph(1, [0] * n, [], dur, gap, thread_order=[])
    g.thread_prev = np.full(n, -1, np.int32)
    prio = rng.integers(-2, 3, size=n).astype(np.int32)
    pp = np.ones(n, np.uint8)
    for policy, order in ((0, list(range(n))),
                          (1, sorted(range(n), key=lambda u: (-int(prio[u]), u)))):
        S, F, M = oracle_mod.run_policy(g, H.variants(g, V=1), policy, pp, prio)
        t = 0
        for u in order:
            assert S[0][u] == t
            t += int(dur[u]) + int(gap[u])
        ends = [int(S[0][u] + dur[u]) for u in range(n)]
        assert M[0] == max(ends)


def _shared_case(seed, zero_frac=0.0):
    rng = np.random.default_rng(7500 + seed)
    n = int(rng.integers(5, 300))
    g, pp, prio = W.random_shared_graph(rng, n, int(rng.integers(1, 4)), int(rng.integers(1, 3)),
                                        mean_in=float(rng.uniform(0.5, 2.5)),
                                        zero_frac=zero_frac,
                                        n_edge_cls=int(rng.integers(1, 3)))
    vs = W.random_variants(rng, g, int(rng.integers(1, 6)), p_remove=0.0, qs=(1,))
    vs.scale[:] = 1
    return g, vs, pp, prio


def _check_valid_run(g, vs, v, S, pp, prio, policy):
    """The properties above, for one variant with positive durations."""
    R = S + g.dur + g.gap
    mask = int(vs.edge_on[v, 0])
    est = np.zeros(g.n, np.int64)
    for u in range(g.n):
        ps = [int(g.in_src[e]) for e in range(g.in_ptr[u], g.in_ptr[u + 1])
              if (mask >> int(g.edge_cls[e])) & 1]
        if g.thread_prev[u] >= 0:
            ps.append(int(g.thread_prev[u]))
        est[u] = max([int(R[p]) for p in ps], default=0)
        assert S[u] >= est[u]
    for t in range(g.n_threads):
        ids = np.nonzero(g.thread_id == t)[0]
        o = ids[np.argsort(S[ids], kind="stable")]
        for a, b in zip(o[:-1], o[1:]):
            assert S[b] >= R[a]                      # one task at a time per thread
        rel = set(int(R[a]) for a in ids)
        for u in ids:                                # never idle while u is ready
            assert S[u] == est[u] or int(S[u]) in rel
        if not pp[ids].all():
            continue
        for x in ids:
            for y in ids:
                if S[x] < S[y] and est[y] <= S[x]:
                    if policy == 1:
                        assert prio[x] > prio[y] or (prio[x] == prio[y] and x < y)
                    else:
                        assert x < y


@pytest.mark.parametrize("seed", range(25))
@pytest.mark.parametrize("policy", [0, 1])
def test_shared_threads_valid_runs(oracle_mod, seed, policy):
    g, vs, pp, prio = _shared_case(seed)
    S, F, M = oracle_mod.run_policy(g, vs, policy, pp, prio)
    for v in range(vs.n_variants):
        _check_valid_run(g, vs, v, S[v], pp, prio, policy)
        assert M[v] == (S[v] + g.dur).max()


def test_priority_rule_changes_some_runs(oracle_mod):
    """The rule is not vacuous: on shared threads the two rules disagree on
    some of these inputs."""
    diffs = 0
    for seed in range(10):
        g, vs, pp, prio = _shared_case(seed)
        a = oracle_mod.run_policy(g, vs, 0, pp, prio)[0]
        b = oracle_mod.run_policy(g, vs, 1, pp, prio)[0]
        diffs += not np.array_equal(a, b)
    assert diffs >= 3


def test_policy_errors(oracle_mod):
    g, pp, prio, _ = load_p3_toy()
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.run_policy(g, H.variants(g, V=1), 2, pp, prio)
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.run_policy(g, H.variants(g, V=1), 1, None, None)
