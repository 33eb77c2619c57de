"""Parity of kernel paths that the workloads alone do not reach, through
the C-ABI against the oracle (start, finish and makespan bit-exact):

* graphs with more than 64 threads, whose run heads take the previous task
  of their thread as an ordinary gather (from HBM when it ended two or more
  rounds earlier, from LDS when it ended in the previous round), in phases
  of many rounds;
* scale tables too large for LDS (task classes x variants per workgroup
  above the LDS table limit), read from HBM, with non-power-of-two q;
* a task waiting on 200 tasks of 200 other threads inside a round of more
  than 64 positions (the wide fan-in loop).
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests import helpers as H
from tests.gpu_common import assert_equal_arrays, gpu_run, require_gpu, say

pytestmark = pytest.mark.gpu


def _check(g, vs, mode=B.DD_PHASES, label="", variants_per_wg=0, want_start=True):
    say("coverage", label, "n=%d threads=%d V=%d mode=%d vs=%d start=%d"
        % (g.n, g.n_threads, vs.n_variants, mode, variants_per_wg, want_start))
    S, F, M = gpu_run(g, vs, mode=mode, variants_per_wg=variants_per_wg, want_start=want_start)
    oS, oF, oM, _ = O.run(g, vs, want_start=want_start)
    assert_equal_arrays(label + " makespan", M, oM)
    assert_equal_arrays(label + " finish", F, oF)
    if want_start:
        assert_equal_arrays(label + " start", S, oS)


# (tasks, threads, mean in-degree, tasks per burst on one thread); phases of
# these graphs hold up to 23,000 positions (tens of rounds)
MANY_THREADS = [(24000, 150, 0.08, 8), (30000, 2000, 0.02, 16), (20000, 100, 0.3, 4),
                (26000, 700, 0.05, 32)]


def _many_threads_case(i, V):
    n, T, mi, rl = MANY_THREADS[i]
    rng = np.random.default_rng(60_000 + i)
    g = W.random_graph_sparse(rng, n, T, mean_in=mi, window=2000, n_edge_cls=2, run_len=rl)
    vs = W.random_variants(rng, g, V, p_remove=0.25)
    return g, vs


@pytest.mark.parametrize("i", range(len(MANY_THREADS)))
def test_many_threads_multi_round(i):
    require_gpu()
    g, vs = _many_threads_case(i, 16 + 17 * (i % 2))
    assert g.n_threads > 64
    _check(g, vs, B.DD_PHASES, "many-threads%d" % i)


@pytest.mark.parametrize("vs_width", [1, 4, 16])
def test_many_threads_every_width(vs_width):
    require_gpu()
    g, vs = _many_threads_case(0, 37)
    _check(g, vs, B.DD_PHASES, "many-threads-w%d" % vs_width, vs_width)


def test_many_threads_levels_mode():
    require_gpu()
    g, vs = _many_threads_case(2, 16)
    _check(g, vs, B.DD_LEVELS, "many-threads-levels")


def _big_table_case(V, seed, qs):
    rng = np.random.default_rng(70_000 + seed)
    g = W.random_graph_sparse(rng, 3000, 3, mean_in=0.4, window=200, n_edge_cls=2,
                              n_node_cls=600, run_len=40)
    vs = W.random_variants(rng, g, V, p_remove=0.2, qs=qs)
    return g, vs


@pytest.mark.parametrize("vs_width", [8, 16])
@pytest.mark.parametrize("V", [37, 38])
@pytest.mark.parametrize("want_start", [True, False])
def test_scale_table_in_hbm(vs_width, V, want_start):
    """600 task classes x 8 or 16 variants per workgroup exceed the 4,096
    entries kept in LDS: the kernels that read the scale table from HBM."""
    require_gpu()
    g, vs = _big_table_case(V, vs_width + V, qs=(1, 2, 3, 5, 7, 8, 10))
    _check(g, vs, B.DD_PHASES, "table-hbm", vs_width, want_start)


def test_scale_table_in_hbm_power_of_two():
    require_gpu()
    g, vs = _big_table_case(38, 5, qs=(1, 2, 4, 8))
    _check(g, vs, B.DD_PHASES, "table-hbm-pow2", 16)


def _fan_in_graph(rng, T=220, width=200, per=10):
    """Phase 0: a run of `per` tasks on each of T threads.  Phase 1: task X
    on thread 0 waits on the last phase-0 task of threads 1..width, and
    every other thread runs 5 more tasks whose first waits on a phase-0 task
    of the next thread, so phase 1 spans well over 64 positions."""
    thread, edges = [], []
    last = {}
    for t in range(T):
        for _ in range(per):
            thread.append(t)
        last[t] = len(thread) - 1
    x = len(thread)
    thread.append(0)
    for t in range(1, width + 1):
        edges.append((last[t], x))
    for t in range(1, T):
        first = len(thread)
        for _ in range(5):
            thread.append(t)
        edges.append((last[(t % (T - 1)) + 1] - 3, first))
    y = len(thread)              # after X on thread 0 (phase 1, same run)
    thread.append(0)
    n = len(thread)
    dur = rng.integers(0, 10**5, n)
    gap = rng.integers(0, 3000, n) * (rng.random(n) < 0.5)
    g = H.graph(T, thread, edges, dur, gap)
    return g, x, y


def test_wide_fan_in_inside_big_round():
    require_gpu()
    rng = np.random.default_rng(80_000)
    g, x, _ = _fan_in_graph(rng)
    assert int(g.in_ptr[x + 1] - g.in_ptr[x]) == 200
    lv, ph = O.steps(g)
    assert (ph == ph[x]).sum() > 64      # X sits in a big round
    V = 24
    removed = [[] for _ in range(V)]
    for v in range(1, V):
        removed[v] = [int(u) for u in rng.choice(g.n, size=g.n // 4, replace=False)]
    vs = H.variants(g, removed=removed, V=V)
    _check(g, vs, B.DD_PHASES, "fan-in-200")
    for w in (1, 16):
        _check(g, vs, B.DD_PHASES, "fan-in-200-w%d" % w, w)


def _multi_fan_in(rng, T=160, per=8, n_x=6, width=(70, 180), n_cls=3):
    """Phase 0: runs of `per` tasks on T threads (several rounds, so a later
    gather's source is in the previous round or older).  Phase 1: n_x tasks,
    each on its own thread right after that thread's run, each waiting on
    70-180 random phase-0 tasks through edges of random classes; the other
    threads run two more tasks, so phase 1 has well over 64 positions and
    several wide positions share a wave."""
    thread, edges, ecls = [], [], []
    for t in range(T):
        thread += [t] * per
    p0 = len(thread)
    xs = []
    for i in range(n_x):
        x = len(thread)
        thread.append(1 + i * 3)
        xs.append(x)
        k = int(rng.integers(width[0], width[1]))
        for s in rng.choice(p0, size=k, replace=False):
            if thread[int(s)] != thread[x]:
                edges.append((int(s), x))
                ecls.append(int(rng.integers(0, n_cls)))
    for t in range(T):
        if t % 3 == 1 and (t - 1) // 3 < n_x:
            continue
        a = len(thread)
        thread += [t, t]
        edges.append((int(rng.integers(0, p0)), a))
        ecls.append(0)
    n = len(thread)
    g = H.graph(T, thread, edges, rng.integers(0, 10**6, n), rng.integers(0, 3000, n),
                edge_cls=ecls, n_edge_cls=n_cls)
    return g, xs


@pytest.mark.parametrize("V", [37, 40])
def test_several_wide_fan_ins_with_edge_classes(V):
    """Wide positions (more than two gathers) several to a wave, sources
    both in the previous round and older, edge classes switched per variant,
    removals: every variants-per-workgroup width."""
    require_gpu()
    rng = np.random.default_rng(81_000 + V)
    g, xs = _multi_fan_in(rng)
    lv, ph = O.steps(g)
    assert len(set(ph[xs].tolist())) == 1 and (ph == ph[xs[0]]).sum() > 64
    assert min(int(g.in_ptr[x + 1] - g.in_ptr[x]) for x in xs) > 40
    removed = [[int(u) for u in rng.choice(g.n, size=g.n // 5, replace=False)] if v else []
               for v in range(V)]
    masks = [1 | int(rng.integers(0, 8)) for _ in range(V)]
    vs = H.variants(g, removed=removed, edge_on=masks, V=V)
    vs.batches = [(0, V, 7)]
    for w in (0, 1, 2, 4, 8, 16):
        _check(g, vs, B.DD_PHASES, "multi-fan-in-V%d-w%d" % (V, w), w)
