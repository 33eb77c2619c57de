"""Parity of the HIP path (through the C-ABI) with the oracle: bit-exact
start, finish and makespan on the same seeded inputs (all times int64 ns)."""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests import helpers as H
from tests.gpu_common import assert_equal_arrays, gpu_run, require_gpu, say

pytestmark = pytest.mark.gpu


def _check(g, vs, mode=B.DD_PHASES, label="", variants_per_wg=0):
    say("parity", label, "n=%d V=%d mode=%d vs=%d" % (g.n, vs.n_variants, mode, variants_per_wg))
    S, F, M = gpu_run(g, vs, mode=mode, variants_per_wg=variants_per_wg)
    oS, oF, oM, _ = O.run(g, vs)
    assert_equal_arrays(label + " makespan", M, oM)
    assert_equal_arrays(label + " finish", F, oF)
    assert_equal_arrays(label + " start", S, oS)


def _random(seed, nmax=60, vmax=40):
    rng = np.random.default_rng(10_000 + seed)
    n = int(rng.integers(1, nmax))
    T = int(rng.integers(1, 5))
    K = int(rng.integers(1, 4))
    g = W.random_graph(rng, n, T, p_edge=float(rng.uniform(0.02, 0.3)), n_edge_cls=K,
                       max_dur=int(rng.choice([5, 1000, 10**6])))
    vs = W.random_variants(rng, g, int(rng.integers(1, vmax)), p_remove=float(rng.uniform(0, 0.5)))
    return g, vs


@pytest.mark.parametrize("seed", range(40))
@pytest.mark.parametrize("mode", [B.DD_PHASES, B.DD_LEVELS])
def test_random_graphs(seed, mode):
    require_gpu()
    g, vs = _random(seed)
    _check(g, vs, mode, "random%d" % seed)


@pytest.mark.parametrize("seed", range(6))
def test_random_larger_graphs(seed):
    """Several rounds of several hundred positions, ragged tails."""
    require_gpu()
    rng = np.random.default_rng(20_000 + seed)
    n = int(rng.integers(3000, 9000))
    g = W.random_graph(rng, n, int(rng.integers(2, 6)), p_edge=3.0 / n, n_edge_cls=2,
                       max_dur=10**5)
    vs = W.random_variants(rng, g, int(rng.integers(20, 70)), p_remove=0.2)
    _check(g, vs, B.DD_PHASES, "larger%d" % seed)


@pytest.mark.parametrize("k,iters,variants", [(1, None, None), (2, None, None), (3, None, None),
                                              (4, None, None)])
def test_configs(k, iters, variants):
    require_gpu()
    g, vs = W.config(k, iters=iters, variants=variants)
    _check(g, vs, B.DD_PHASES, "config%d" % k)


@pytest.mark.parametrize("k", [1, 2])
def test_configs_levels_mode(k):
    require_gpu()
    g, vs = W.config(k, variants=16)
    _check(g, vs, B.DD_LEVELS, "config%d-levels" % k)


@pytest.mark.parametrize("vs_width", [1, 2, 4, 8, 16])
def test_every_variant_width(vs_width):
    """Each compiled variants-per-workgroup width gives the same answer,
    including a last workgroup that is only partly used."""
    require_gpu()
    g, vs = W.config(1, variants=37)
    _check(g, vs, B.DD_PHASES, "width%d" % vs_width, vs_width)
    rng = np.random.default_rng(33)
    g = W.random_graph(rng, 500, 3, p_edge=0.01, n_edge_cls=2, max_dur=1000)
    vs = W.random_variants(rng, g, 19, p_remove=0.3)
    _check(g, vs, B.DD_PHASES, "width%d-random" % vs_width, vs_width)


@pytest.mark.parametrize("vs_width", [1, 2, 4, 8, 16])
def test_outputs_prefilled_with_sentinel(vs_width):
    """Output buffers start full of a huge sentinel: a read of finish before
    its task is written, or any stale read, shows up as a wrong value.  Odd
    and even variant counts cover both lane layouts of every width."""
    import torch
    require_gpu()
    sent = 1 << 61
    for V in (37, 38):
        g, vs = W.config(1, variants=V)
        di = BT.to_device(g, vs)
        outs = [(torch.full((g.n, v1 - v0), sent, dtype=torch.int64, device="cuda"),
                 torch.full((g.n, v1 - v0), sent, dtype=torch.int64, device="cuda"),
                 torch.full((v1 - v0,), sent, dtype=torch.int64, device="cuda"))
                for (v0, v1, *_r) in di.batches]
        say("parity sentinel width%d V=%d" % (vs_width, V))
        res = BT.simulate(di, want_start=True, outputs=outs, variants_per_wg=vs_width)
        torch.cuda.synchronize()
        oS, oF, oM, _ = O.run(g, vs)
        for v0, v1, f, s_, m in res:
            assert_equal_arrays("sentinel makespan", m.cpu().numpy(), oM[v0:v1])
            assert_equal_arrays("sentinel finish", f.cpu().numpy().T, oF[v0:v1])
            assert_equal_arrays("sentinel start", s_.cpu().numpy().T, oS[v0:v1])


def test_empty_graph():
    require_gpu()
    g = H.graph(1, [], [], [], [])
    vs = H.variants(g, V=5)
    _check(g, vs, B.DD_PHASES, "empty")


def test_single_task_and_all_removed():
    require_gpu()
    g = H.graph(1, [0], [], [123], [7])
    _check(g, H.variants(g, V=3), B.DD_PHASES, "single")
    g = H.graph(2, [0, 1, 0, 1], [(0, 1), (2, 3)], [5, 6, 7, 8], [1, 0, 1, 0])
    vs = H.variants(g, removed=[[0, 1, 2, 3], [], [1, 2]])
    _check(g, vs, B.DD_PHASES, "all-removed")


def test_extreme_scales():
    """p = 0, q up to 2^31-1, non-power-of-two q, large durations near the bound."""
    require_gpu()
    rng = np.random.default_rng(5)
    n = 300
    g = W.random_graph(rng, n, 3, p_edge=0.02, max_dur=10)
    g.dur[:] = rng.integers(0, 2**40, n)
    g.node_cls[:] = rng.integers(0, 3, n).astype(np.uint16)
    qs = [1, 2, 3, 5, 7, 10, 1000003, 2**31 - 1, 2**30, 6]
    scales = []
    for v in range(len(qs)):
        q = qs[v]
        scales.append({0: (0, 1), 1: (int(rng.integers(0, 4096)), q), 2: (7, 7)})
    vs = H.variants(g, scales=scales)
    _check(g, vs, B.DD_PHASES, "extreme")


def test_high_in_degree():
    """One task waits for many tasks on many threads (a sync after many
    all-reduce channels)."""
    require_gpu()
    T = 70
    thread = list(range(T)) + [0]
    edges = [(i, T) for i in range(1, T)]
    rng = np.random.default_rng(9)
    g = H.graph(T, thread, edges, rng.integers(0, 10**6, T + 1), rng.integers(0, 10, T + 1))
    vs = H.variants(g, removed=[[], [5, 6], list(range(1, T))], V=3)
    _check(g, vs, B.DD_PHASES, "fan-in")


def test_deterministic_repeat():
    require_gpu()
    g, vs = W.config(2, variants=64)
    a = gpu_run(g, vs)
    b = gpu_run(g, vs)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
