"""Pins of the oracle's runtime breakdown (Sec. 6.2, Fig. 6: CPU-only,
GPU-only and CPU+GPU-parallel runtime) against what does not come from the
oracle:
  * a hand-worked trace (tests/golden/breakdown_toy.txt);
  * brute force over unit time steps on small random traces: the start and
    finish of every task from the all-paths brute force of the simulation
    pins, then GPU busy time and CPU blocked time counted step by step;
  * invariants: the three parts add up to the iteration time; with every
    kernel removed the whole iteration is CPU-only.
The paper prints no numbers for the breakdown (the figure is missing from
the text), so the readings are ours: GPU kernel time is the sum of kernel
durations (one stream serialises them), and a waiting call's GPU-only time
runs from the moment its thread reaches it to its start."""
import os

import numpy as np
import pytest

from paper_2006_03318_amd import workloads as W
from tests import helpers as H
from tests.test_oracle_pins import brute_force

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "breakdown_toy.txt")


def _read_toy():
    f = {}
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            k, *v = line.split()
            f[k] = v
    edges = [tuple(int(x) for x in e.split(">")) for e in f["edges"]]
    g = H.graph(int(f["threads"][0]), [int(x) for x in f["thread"]], edges,
                [int(x) for x in f["dur"]], [int(x) for x in f["gap"]])
    return g, np.array([int(x) for x in f["role"]], np.uint8), [int(x) for x in f["expect"]]


def test_hand_worked_trace(oracle_mod):
    g, role, expect = _read_toy()
    out = oracle_mod.breakdown(g, H.variants(g, V=1), role)
    assert list(out[0]) == expect


def _trace(rng, n_launch, p_sync=0.3, two_cpu=False):
    """CPU thread 0 launches kernels onto GPU stream 1 and sometimes waits
    for the latest kernel (a synchronization call); optionally a second CPU
    thread 2 with its own calls and occasional waits."""
    thread, dur, gap, edges, role = [], [], [], [], []
    last_kernel = -1
    for i in range(n_launch):
        cpu = 2 if (two_cpu and rng.random() < 0.3) else 0
        thread.append(cpu); dur.append(int(rng.integers(0, 6))); gap.append(int(rng.integers(0, 3)))
        role.append(0)
        lid = len(thread) - 1
        thread.append(1); dur.append(int(rng.integers(0, 12))); gap.append(0); role.append(1)
        last_kernel = len(thread) - 1
        edges.append((lid, last_kernel))
        if rng.random() < p_sync:
            thread.append(cpu); dur.append(int(rng.integers(0, 4))); gap.append(int(rng.integers(0, 2)))
            role.append(2)
            edges.append((last_kernel, len(thread) - 1))
    g = H.graph(3 if two_cpu else 2, thread, edges, dur, gap)
    g.node_cls[:] = np.array([0 if t != 1 else 1 for t in thread], np.uint16)
    g.n_node_cls = 2
    return g, np.array(role, np.uint8)


def _stepwise(g, vs, v, role):
    """Breakdown by unit time steps from the brute-force schedule."""
    S, F, T = brute_force(g, vs, v)
    rm = W.unpack_bits(vs.remove_bits, vs.n_variants)[:, v]
    gpu_busy = 0
    for t in range(T):
        if any(role[u] == 1 and not rm[u] and S[u] <= t < F[u] for u in range(g.n)):
            gpu_busy += 1
    blocked = 0
    for u in range(g.n):
        if role[u] != 2:
            continue
        p = int(g.thread_prev[u])
        if p >= 0:
            p_gap = 0 if rm[p] else int(g.gap[p])
            reached = F[p] + p_gap
        else:
            reached = 0
        blocked += sum(1 for t in range(reached, S[u]))
    cpu_only = T - gpu_busy
    return [T, cpu_only, blocked, T - cpu_only - blocked]


@pytest.mark.parametrize("seed", range(60))
def test_stepwise_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(170_000 + seed)
    g, role = _trace(rng, int(rng.integers(1, 6)), two_cpu=seed % 2 == 1)
    V = 4
    scales = [{}] + [{c: (int(rng.integers(0, 5)), int(rng.choice([1, 2, 3]))) for c in (0, 1)}
                     for _ in range(V - 1)]
    removed = [[]] + [[u for u in range(g.n) if rng.random() < 0.2] for _ in range(V - 1)]
    vs = H.variants(g, scales=scales, removed=removed, V=V)
    out = oracle_mod.breakdown(g, vs, role)
    for v in range(V):
        assert list(out[v]) == _stepwise(g, vs, v, role), v


@pytest.mark.parametrize("seed", range(10))
def test_invariants(oracle_mod, seed):
    rng = np.random.default_rng(180_000 + seed)
    g, role = _trace(rng, 30, two_cpu=False)
    vs = H.variants(g, removed=[[], [u for u in range(g.n) if role[u] == 1]], V=2)
    out = oracle_mod.breakdown(g, vs, role)
    _, _, ms, _ = oracle_mod.run(g, vs)
    assert (out[:, 0] == ms).all()
    assert (out[:, 1] + out[:, 2] + out[:, 3] == out[:, 0]).all()
    assert (out[:, 2] >= 0).all()
    # every kernel removed: no GPU time, and the one CPU thread never waits
    # (a removed kernel passes on its launch's release, which the thread has
    # already passed)
    assert out[1, 1] == out[1, 0] and out[1, 2] == 0
