"""GPU levelization (Kahn levels and phases) against the oracle's plain
Kahn's algorithm; graph-load error handling through the C-ABI."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests import helpers as H
from tests.gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu


def _steps_gpu(g, mask, mode):
    import torch
    vs = H.variants(g, V=1)
    di = BT.to_device(g, vs)
    gh = BT.load_graph(di)
    try:
        sch, nsteps = B.dd_levelize(gh, mask, mode)
        try:
            out = np.zeros(max(g.n, 1), np.int32)
            B.dd_sched_task_steps(sch, out)
            info = B.dd_sched_info(sch)
        finally:
            B.dd_sched_free(sch)
    finally:
        B.dd_graph_free(gh)
    torch.cuda.synchronize()
    return out[:g.n], nsteps, info


@pytest.mark.parametrize("seed", range(30))
def test_random_steps(seed):
    require_gpu()
    rng = np.random.default_rng(40_000 + seed)
    g = W.random_graph(rng, int(rng.integers(1, 80)), int(rng.integers(1, 6)),
                       p_edge=float(rng.uniform(0.02, 0.3)), n_edge_cls=3)
    mask = int(rng.integers(1, 8))
    say("steps", seed, g.n, mask)
    lv, ph = O.steps(g, mask)
    gl, nl, _ = _steps_gpu(g, mask, B.DD_LEVELS)
    gp, np_, info = _steps_gpu(g, mask, B.DD_PHASES)
    assert np.array_equal(gl, lv)
    assert np.array_equal(gp, ph)
    assert nl == (int(lv.max()) + 1 if g.n else 0)
    assert np_ == (int(ph.max()) + 1 if g.n else 0)


@pytest.mark.parametrize("n", [63, 64, 65, 66, 127, 128, 129, 130])
def test_ping_pong_round_counts(n):
    """Two threads that hand over at every task: one Kahn round per task, so
    the round count crosses the 64-row batches in which the rounds' fronts
    are written (a last batch that is full, one row short, one row over)."""
    require_gpu()
    thread = [i % 2 for i in range(n)]
    edges = [(i - 1, i) for i in range(1, n)]
    g = H.graph(2, thread, edges, [3 + i % 5 for i in range(n)], [i % 2 for i in range(n)])
    lv, ph = O.steps(g, 1)
    gp, nph, _ = _steps_gpu(g, 1, B.DD_PHASES)
    say("ping-pong", n, "phases", nph)
    assert nph == int(ph.max()) + 1
    assert np.array_equal(gp, ph)


@pytest.mark.parametrize("seed", [0, 1])
def test_many_threads_chain_ranks(seed):
    """Thousands of threads spread over the task ids: more tile exits than
    one workgroup ranks, so graph load falls back to plain pointer jumping;
    the schedule still matches the oracle's."""
    require_gpu()
    rng = np.random.default_rng(50_000 + seed)
    n, T = 30000, 3000
    thread = rng.integers(0, T, n)
    thread[:T] = np.arange(T)                       # every thread has a task
    a = rng.integers(0, n - 1, 3000)
    b = np.minimum(a + rng.integers(1, 500, 3000), n - 1)
    edges = [(int(x), int(y)) for x, y in zip(a, b) if x < y]
    g = H.graph(T, thread, edges, rng.integers(0, 100, n), rng.integers(0, 10, n))
    lv, ph = O.steps(g, 1)
    gp, nph, _ = _steps_gpu(g, 1, B.DD_PHASES)
    say("many threads", seed, "phases", nph)
    assert np.array_equal(gp, ph)


@pytest.mark.parametrize("T", [17, 33, 64, 65, 129, 255, 256, 257, 513, 1025, 2048, 2049])
def test_kahn_rounds_thread_counts(T):
    """Phases of graphs with more threads than the windowed rounds take: every
    lane-group width of the probe (32 lanes per thread down to 1, and
    several passes past 1,024 threads), packed candidate entries (up to 255
    threads) and not, round state in LDS (up to 2,048 threads) and not;
    tasks with parents on one, two and three or more other threads."""
    require_gpu()
    rng = np.random.default_rng(45_000 + T)
    n = max(6000, 6 * T)
    g = W.random_graph_sparse(rng, n, T, mean_in=0.9, window=400, n_edge_cls=2,
                              run_len=int(rng.integers(1, 12)))
    for mask in (1, 3):
        lv, ph = O.steps(g, mask)
        gp, nph, _ = _steps_gpu(g, mask, B.DD_PHASES)
        say("kahn threads", T, "mask", mask, "phases", nph)
        assert nph == int(ph.max()) + 1
        assert np.array_equal(gp, ph)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_config_steps(k):
    require_gpu()
    g, vs = W.config(k, variants=8)
    mask = vs.batches[0][2]
    lv, ph = O.steps(g, mask)
    gp, nph, info = _steps_gpu(g, mask, B.DD_PHASES)
    say("config", k, "phases", nph, info)
    assert np.array_equal(gp, ph)
    if k in (1, 2):
        gl, nl, info = _steps_gpu(g, mask, B.DD_LEVELS)
        say("config", k, "levels", nl, info)
        assert np.array_equal(gl, lv)


def _load(g):
    di = BT.to_device(g, H.variants(g, V=1))
    return BT.load_graph(di)


def _expect(code, fn):
    with pytest.raises(B.DDError) as ei:
        fn()
    assert ei.value.code == code, str(ei.value)


def test_load_errors():
    require_gpu()
    good = H.graph(2, [0, 1, 0], [(0, 1)], [1, 2, 3], [0, 0, 0])
    B.dd_graph_free(_load(good))
    # source out of range
    g = H.graph(2, [0, 1, 0], [(0, 1)], [1, 2, 3], [0, 0, 0])
    g.in_src[0] = 7
    _expect(B.DD_EINVAL, lambda: _load(g))
    # self loop
    g = H.graph(2, [0, 1, 0], [(1, 1)], [1, 2, 3], [0, 0, 0])
    _expect(B.DD_ECYCLE, lambda: _load(g))
    # negative duration
    g = H.graph(2, [0, 1, 0], [(0, 1)], [1, -2, 3], [0, 0, 0])
    _expect(B.DD_EINVAL, lambda: _load(g))
    # duration beyond the 2^62 bound
    g = H.graph(2, [0, 1, 0], [(0, 1)], [1, 2**62, 3], [0, 0, 0])
    _expect(B.DD_ERANGE, lambda: _load(g))
    # thread order names a task of another thread
    g = H.graph(2, [0, 1, 0], [], [1, 2, 3], [0, 0, 0])
    g.thread_prev[2] = 1
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # two first tasks on one thread
    g = H.graph(2, [0, 1, 0], [], [1, 2, 3], [0, 0, 0])
    g.thread_prev[2] = -1
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # two tasks name the same previous task (the thread order forks)
    g = H.graph(1, [0, 0, 0], [], [1, 2, 3], [0, 0, 0])
    g.thread_prev[2] = 0
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # the same fork deep inside a long thread
    g = H.graph(1, [0] * 3000, [], [1] * 3000, [0] * 3000)
    g.thread_prev[2500] = 1700
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # thread order loops across tiles of consecutive tasks, away from the
    # thread's head (the loop is found among the tile exits)
    n = 3000
    g = H.graph(1, [0] * n, [], [1] * n, [0] * n)
    g.thread_prev[2000] = n - 1
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # thread order loops (plus a proper head elsewhere)
    g = H.graph(1, [0, 0, 0], [], [1, 2, 3], [0, 0, 0], thread_order=[[0]])
    g.thread_prev[1] = 2
    g.thread_prev[2] = 1
    _expect(B.DD_ECHAIN, lambda: _load(g))
    # dependency backwards along one thread
    g = H.graph(1, [0, 0], [(1, 0)], [1, 2], [0, 0])
    _expect(B.DD_ECYCLE, lambda: _load(g))
    # thread id out of range
    g = H.graph(2, [0, 1, 0], [], [1, 2, 3], [0, 0, 0])
    g.thread_id[1] = 5
    g.thread_prev[1] = -1
    _expect(B.DD_EINVAL, lambda: _load(g))


def test_cycle_at_levelize_and_mismatch():
    require_gpu()
    import torch
    g = H.graph(2, [0, 1], [(0, 1), (1, 0)], [5, 7], [0, 0], edge_cls=[0, 1], n_edge_cls=2)
    gh = _load(g)
    try:
        _expect(B.DD_ECYCLE, lambda: B.dd_levelize(gh, 0b11, B.DD_PHASES))
        sch, n = B.dd_levelize(gh, 0b01, B.DD_PHASES)
        eon = torch.tensor([1, 3], dtype=torch.uint64, device="cuda")
        var = B.dd_apply_transforms(gh, 2, 1, None, None, eon)
        fin = torch.zeros((2, 2), dtype=torch.int64, device="cuda")
        ms = torch.zeros(2, dtype=torch.int64, device="cuda")
        # variant 1 switches on class 1, which this schedule does not cover
        _expect(B.DD_EMISMATCH, lambda: B.dd_simulate_batch(gh, sch, var, fin, None, ms))
        _expect(B.DD_EINVAL, lambda: B.dd_simulate_batch(gh, sch, var, None, None, ms))
        B.dd_variants_free(var)
        # scale entries must have p >= 0 and q >= 1
        bad = np.array([[[1, 0], [1, 1]]], np.int32)
        _expect(B.DD_EINVAL, lambda: B.dd_apply_transforms(gh, 2, 1, bad, None, None))
        # scaled durations that could overflow
        big = np.array([[[2**30, 1], [1, 1]]], np.int32)
        g2 = H.graph(1, [0], [], [2**40], [0])
        gh2 = _load(g2)
        _expect(B.DD_ERANGE, lambda: B.dd_apply_transforms(gh2, 2, 1, big, None, None))
        # handles of different graphs
        var2 = B.dd_apply_transforms(gh2, 1, 1, None, None, None)
        _expect(B.DD_EMISMATCH, lambda: B.dd_simulate_batch(gh, sch, var2, fin, None, ms))
        B.dd_variants_free(var2)
        B.dd_graph_free(gh2)
        B.dd_sched_free(sch)
    finally:
        B.dd_graph_free(gh)
