"""Parity of the HIP path with the oracle on variant tables built by the
what-if recipe compiler (bit-exact start, finish and makespan)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import recipes as R
from paper_2006_03318_amd import workloads as W
from tests.gpu_common import assert_equal_arrays, gpu_run, require_gpu, say
from tests.test_recipes import SWEEP, _random_sweep, toy_graph

pytestmark = pytest.mark.gpu


def _check(g, vs, label):
    say("recipes", label, "n=%d V=%d classes=%d" % (g.n, vs.n_variants, g.n_node_cls))
    S, F, M = gpu_run(g, vs)
    oS, oF, oM, _ = O.run(g, vs)
    assert_equal_arrays(label + " makespan", M, oM)
    assert_equal_arrays(label + " finish", F, oF)
    assert_equal_arrays(label + " start", S, oS)


def test_hand_sweep():
    require_gpu()
    g, vs = R.compile_sweep(toy_graph(), SWEEP)
    _check(g, vs, "hand")


@pytest.mark.parametrize("k,V", [(1, 40), (2, 64), (3, 96), (4, 16)])
def test_config_sweeps(k, V):
    """The recipe sweeps of the four trace-shaped workloads, shortened in
    variants (config 3 keeps all four channel-order batches)."""
    require_gpu()
    g, vs = W.config(k, variants=V)
    _check(g, vs, "config%d" % k)


@pytest.mark.parametrize("seed", range(3))
def test_random_recipe_mixes(seed):
    """Random recipe stacks on the CNN and transformer graphs, including
    edge-class switches that split the sweep into several batches."""
    require_gpu()
    rng = np.random.default_rng(4200 + seed)
    for k, L in ((1, 20), (2, 24)):
        g, _ = W.config(k, variants=1)
        sweep = _random_sweep(rng, g, 70, L)
        g2, vs = R.compile_sweep(g, sweep)
        _check(g2, vs, "mix%d-config%d" % (seed, k))


def test_vdnn_sweep():
    """Memory offloading with the prefetch policies as edge classes, all in
    one levelization."""
    require_gpu()
    g, vs = W.vdnn_workload(iters=3, variants=60)
    _check(g, vs, "vdnn")
